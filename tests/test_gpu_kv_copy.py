"""GPU tier, bit-exact: KV append and gather through the C ABI against the oracle.

The whole pool is compared after the append, so a stray write anywhere (including the NaN
canaries in stale slots and unowned blocks) fails the test."""
import numpy as np
import pytest

import oracle
import workloads as W
from tests.gpu_util import DevBatch, dev_pools, say, to_host_bits

pytestmark = pytest.mark.gpu

SMALL = [
    W.TINY,
    W.LLAMA3_8B_PREFILL.scaled(prefill=12),
    W.LLAMA3_8B_DECODE.scaled(decode=40),
    W.MIXED_70B.scaled(prefill=4, decode=24),
    W.LONG_DOC_SHARED_PROMPT.scaled(prefill=4),
]


@pytest.mark.parametrize("spec", SMALL, ids=lambda s: s.name)
def test_append_then_gather_bit_exact(gpu_lib, spec):
    import torch
    lib = gpu_lib
    say(f"[append/gather] {spec.name}")
    case = W.make_case(spec)
    pk, pv = dev_pools(case)
    ref_k, ref_v = case.pool_k, case.pool_v
    for b in case.batches:
        db = DevBatch(b)
        lib.pkv_kv_append(pk, pv, db.k_new, db.v_new, db.tables, db.cached, db.cu, db.max_new)
        ref_k, ref_v = oracle.kv_append(ref_k, ref_v, b.block_tables, b.prefix_lens,
                                        b.cu_new_lens, b.k_new, b.v_new, spec.block_size)
    torch.cuda.synchronize()
    got_k, got_v = to_host_bits(pk), to_host_bits(pv)
    assert np.array_equal(got_k, ref_k), f"K pool differs in {np.sum(got_k != ref_k)} elements"
    assert np.array_equal(got_v, ref_v), f"V pool differs in {np.sum(got_v != ref_v)} elements"

    for b in case.batches:
        db = DevBatch(b)
        lens = b.prefix_lens + b.new_lens
        cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
        tot = int(cu[-1])
        ko = torch.empty((tot, case.hkv, case.d), dtype=torch.bfloat16, device="cuda")
        vo = torch.empty_like(ko)
        from tests.gpu_util import i32
        lib.pkv_gather_kv(pk, pv, db.tables, i32(lens), i32(cu), int(lens.max()), ko, vo)
        torch.cuda.synchronize()
        ek, ev = oracle.gather_kv(ref_k, ref_v, b.block_tables, lens, spec.block_size)
        assert np.array_equal(to_host_bits(ko), ek)
        assert np.array_equal(to_host_bits(vo), ev)


def test_append_partial_blocks_and_empty_sequences(gpu_lib):
    """Prefixes ending mid-block, sequences with no new tokens, a new range that starts and ends
    inside one block, and sequences spanning many blocks, in one call."""
    import torch
    lib = gpu_lib
    say("[append] partial blocks / empty sequences")
    prefixes = [0, 5, 16, 17, 31, 40, 100, 7]
    news = [3, 0, 16, 1, 40, 0, 77, 9]
    spec = W.WorkloadSpec("append_edges", 90, 4, 2, 128,
                          (W.BatchSpec("prefill", len(prefixes), W.Dist.const(1),
                                       W.Dist.const(1)),), ("scale", 1.5))
    case = W.make_case(spec, prefix_override=[prefixes], new_override=[news])
    b = case.batches[0]
    pk, pv = dev_pools(case)
    db = DevBatch(b)
    lib.pkv_kv_append(pk, pv, db.k_new, db.v_new, db.tables, db.cached, db.cu, db.max_new)
    torch.cuda.synchronize()
    ref_k, ref_v = oracle.kv_append(case.pool_k, case.pool_v, b.block_tables, b.prefix_lens,
                                    b.cu_new_lens, b.k_new, b.v_new, 16)
    assert np.array_equal(to_host_bits(pk), ref_k)
    assert np.array_equal(to_host_bits(pv), ref_v)


def test_append_head_dim_64_many_heads(gpu_lib):
    import torch
    lib = gpu_lib
    say("[append] head_dim 64, 8 kv heads")
    spec = W.WorkloadSpec("append_d64", 91, 8, 8, 64,
                          (W.BatchSpec("prefill", 6, W.Dist.uniform(0, 70),
                                       W.Dist.uniform(1, 50)),), ("scale", 1.3))
    case = W.make_case(spec)
    b = case.batches[0]
    pk, pv = dev_pools(case)
    db = DevBatch(b)
    lib.pkv_kv_append(pk, pv, db.k_new, db.v_new, db.tables, db.cached, db.cu, db.max_new)
    torch.cuda.synchronize()
    ref_k, ref_v = oracle.kv_append(case.pool_k, case.pool_v, b.block_tables, b.prefix_lens,
                                    b.cu_new_lens, b.k_new, b.v_new, 16)
    assert np.array_equal(to_host_bits(pk), ref_k)
    assert np.array_equal(to_host_bits(pv), ref_v)


@pytest.mark.parametrize("hq,hkv,d", [(32, 8, 128), (8, 2, 64)])
def test_append_one_token_per_sequence(gpu_lib, hq, hkv, d):
    """A decode step's append (max_new_len == 1, its own launch shape): every slot position in
    a block, sequences with no token, bit-exact over the whole pool (stale NaN canaries
    included)."""
    import torch
    lib = gpu_lib
    say(f"[append] one token per sequence hq={hq} hkv={hkv} d={d}")
    prefixes = [0, 1, 7, 8, 9, 15, 16, 17, 31, 100, 255, 256, 5, 40]
    news = [1] * 12 + [0, 1]
    spec = W.WorkloadSpec(f"append_token_{d}", 95 + d, hq, hkv, d,
                          (W.BatchSpec("prefill", len(prefixes), W.Dist.const(1),
                                       W.Dist.const(1)),), ("scale", 1.5))
    case = W.make_case(spec, prefix_override=[prefixes], new_override=[news])
    b = case.batches[0]
    pk, pv = dev_pools(case)
    db = DevBatch(b)
    assert db.max_new == 1
    lib.pkv_kv_append(pk, pv, db.k_new, db.v_new, db.tables, db.cached, db.cu, db.max_new)
    torch.cuda.synchronize()
    ref_k, ref_v = oracle.kv_append(case.pool_k, case.pool_v, b.block_tables, b.prefix_lens,
                                    b.cu_new_lens, b.k_new, b.v_new, 16)
    assert np.array_equal(to_host_bits(pk), ref_k)
    assert np.array_equal(to_host_bits(pv), ref_v)
