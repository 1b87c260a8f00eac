"""GPU tier: a seeded sweep of random small shapes through the C ABI.

Each case draws a kv-head count, a query/kv head ratio (1 to 16), a head dim (64 or 128), a
batch size, per-sequence prefix and suffix lengths (prefixes ending anywhere in a block,
empty prefixes included) and a random block placement. The append is checked bit for bit
over the whole pool (every byte outside the new slots unchanged, NaN canaries included),
prefill and decode against the fp64 oracle at the same bar as the other GPU tests; a sweep of
small batches of long sequences runs the prefill with its plan (key split, order).
PKV_RANDOM_SCALE=n runs n times as many cases (the default sweep is 12 + 12 + 8)."""
import os

import numpy as np
import pytest

import oracle
import workloads as W
from tests.gpu_util import DevBatch, dev_pools, say, to_host_bits
from tests.test_gpu_decode import check as check_decode
from tests.test_gpu_decode import oracle_decode, run_decode
from tests.test_gpu_prefill import check as check_prefill
from tests.test_gpu_prefill import oracle_prefill, run_prefill

pytestmark = pytest.mark.gpu

SEED = 260723815 + 900
SCALE = max(1, int(os.environ.get("PKV_RANDOM_SCALE", "1")))


def _heads(rng):
    hkv = int(rng.choice([1, 2, 4, 8]))
    g = int(rng.choice([1, 2, 4, 8, 16]))
    while hkv * g > 32:  # keeps the fp64 oracle within seconds
        g //= 2
    return hkv * g, hkv, int(rng.choice([64, 128]))


def _prefill_case(k):
    rng = np.random.default_rng(SEED + k)
    hq, hkv, d = _heads(rng)
    b = int(rng.integers(1, 7))
    prefixes = rng.integers(0, 600, b)
    prefixes[rng.random(b) < 0.2] = 0
    news = rng.integers(1, 200, b)
    spec = W.WorkloadSpec(f"random_prefill_{k}", 900 + k, hq, hkv, d,
                          (W.BatchSpec("prefill", b, W.Dist.const(1), W.Dist.const(1)),),
                          ("scale", float(rng.choice([1.0, 1.5, 3.0]))))
    return W.make_case(spec, prefix_override=[prefixes.tolist()],
                       new_override=[news.tolist()])


def _decode_case(k):
    rng = np.random.default_rng(SEED + 100 + k)
    hq, hkv, d = _heads(rng)
    b = int(rng.integers(1, 30))
    ctx = rng.integers(0, 2200, b)  # up to 138 blocks: past a 64-entry table chunk
    spec = W.WorkloadSpec(f"random_decode_{k}", 1000 + k, hq, hkv, d,
                          (W.BatchSpec("decode", b, W.Dist.const(1), W.Dist.const(1)),),
                          ("scale", float(rng.choice([1.0, 1.25, 2.0]))))
    return W.make_case(spec, prefix_override=[ctx.tolist()])


@pytest.mark.parametrize("k", range(12 * SCALE))
def test_random_prefill_and_append(gpu_lib, k):
    case = _prefill_case(k)
    b = case.batches[0]
    say(f"[random] prefill {k}: hq={case.hq} hkv={case.hkv} d={case.d} "
        f"prefix={b.prefix_lens.tolist()} new={b.new_lens.tolist()}")
    pk, pv = dev_pools(case)
    db = DevBatch(b)
    gpu_lib.pkv_kv_append(pk, pv, db.k_new, db.v_new, db.tables, db.cached, db.cu, db.max_new)
    ref_k, ref_v = oracle.kv_append(case.pool_k, case.pool_v, b.block_tables, b.prefix_lens,
                                    b.cu_new_lens, b.k_new, b.v_new, case.bs)
    assert np.array_equal(to_host_bits(pk), ref_k)
    assert np.array_equal(to_host_bits(pv), ref_v)
    # the prefill appends again (the same bits) and attends over prefix + suffix
    check_prefill(f"random_prefill_{k}", case, run_prefill(gpu_lib, case, pools=(pk, pv)),
                  oracle_prefill(case))


@pytest.mark.parametrize("k", range(12 * SCALE))
def test_random_decode(gpu_lib, k):
    case = _decode_case(k)
    b = case.batches[0]
    say(f"[random] decode {k}: hq={case.hq} hkv={case.hkv} d={case.d} seqs={b.n_seqs} "
        f"max context={int(b.prefix_lens.max())}")
    check_decode(f"random_decode_{k}", run_decode(gpu_lib, case), oracle_decode(case))


def _plan_case(k):
    """A small batch of long sequences: the prefill's plan splits its keys (and, when several
    sequences reach 8192 keys, orders them longest first)."""
    rng = np.random.default_rng(SEED + 200 + k)
    hq, hkv, d = _heads(rng)
    b = int(rng.integers(1, 4))
    prefixes = rng.integers(2100, 12000, b)
    news = rng.integers(1, 160, b)
    spec = W.WorkloadSpec(f"random_plan_{k}", 1100 + k, hq, hkv, d,
                          (W.BatchSpec("prefill", b, W.Dist.const(1), W.Dist.const(1)),),
                          ("scale", 1.25))
    return W.make_case(spec, prefix_override=[prefixes.tolist()],
                       new_override=[news.tolist()])


@pytest.mark.parametrize("k", range(8 * SCALE))
def test_random_prefill_with_plan(gpu_lib, k):
    """Random small batches of long sequences through the prefill with the plan's workspace
    (key split, longest-first order) against the oracle."""
    import torch
    from tests.gpu_util import scale_for
    case = _plan_case(k)
    b = case.batches[0]
    db = DevBatch(b)
    nbytes = gpu_lib.pkv_prefill_workspace_bytes(b.n_seqs, b.total_new, case.hq, case.hkv,
                                                 case.d, db.max_new, db.max_total)
    say(f"[random] plan {k}: hq={case.hq} hkv={case.hkv} d={case.d} "
        f"prefix={b.prefix_lens.tolist()} new={b.new_lens.tolist()} workspace={nbytes}")
    assert nbytes > 0, "the case was meant to split"
    pk, pv = dev_pools(case)
    ws = gpu_lib.alloc_workspace(nbytes)
    out = torch.empty((b.total_new, case.hq, case.d), dtype=torch.bfloat16, device="cuda")
    lse = torch.empty((b.total_new, case.hq), dtype=torch.float32, device="cuda")
    gpu_lib.pkv_kv_append(pk, pv, db.k_new, db.v_new, db.tables, db.cached, db.cu, db.max_new)
    gpu_lib.pkv_prefill_attention(pk, pv, db.q, db.tables, db.cached, db.cu, db.max_new,
                                  db.max_total, scale_for(case.d), out, lse=lse, workspace=ws)
    torch.cuda.synchronize()
    check_prefill(f"random_plan_{k}", case,
                  (to_host_bits(out), lse.cpu().numpy().astype(np.float64)),
                  oracle_prefill(case))
