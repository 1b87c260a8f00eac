"""GPU tier: prefix-reuse paged prefill attention through the C ABI against the fp64 oracle.

Bar: max-abs <= 2e-2 and mean-abs <= 2e-3 over every output element (bf16 inputs, fp32
accumulation, bf16 output), LSE within LSE_MAX / LSE_MEAN below. Cases span several key tiles, ragged query
tails, prefixes ending mid-block, no prefix at all, single new tokens, head ratios 1..8, head
dims 64 and 128, the shared-prompt layout, and stale NaN slots in every block tail."""
import numpy as np
import pytest

import oracle
import workloads as W
from tests.gpu_util import (DevBatch, bf16_to_f64, compare, dev_pools, say, scale_for,
                            to_host_bits)

pytestmark = pytest.mark.gpu

# LSE = m + ln(sum of the fp32 weights): bf16 rounding never touches it (the rounded weights
# only feed the value product). Its error is that of fp32 arithmetic: a score is an fp32 sum
# of D exact bf16 products, off by at most (D - 1) u scale sum_d |q_d k_d| to first order
# (u = 2^-24; ~8.8e-5 at D = 128 for the largest such sum among N(0,1) rows), the LSE is a
# weighted mean of score errors, so bounded by the same; the fp32 sums of the weights add at
# most ~(adds in sequence) u ~ 1.5e-5 at 16k keys, exp2 and log2 an ulp each. Measured:
# ~2e-6 max. Bounds: twice the first-order worst case for the max, 1e-5 for the mean.
LSE_MAX = 2e-4
LSE_MEAN = 1e-5


def run_prefill(lib, case, bi=0, pools=None):
    """Append the batch's new tokens, then prefill attention; returns (out bits, lse)."""
    import torch
    b = case.batches[bi]
    pk, pv = pools if pools is not None else dev_pools(case)
    db = DevBatch(b)
    out = torch.empty((b.total_new, case.hq, case.d), dtype=torch.bfloat16, device="cuda")
    lse = torch.empty((b.total_new, case.hq), dtype=torch.float32, device="cuda")
    lib.pkv_kv_append(pk, pv, db.k_new, db.v_new, db.tables, db.cached, db.cu, db.max_new)
    lib.pkv_prefill_attention(pk, pv, db.q, db.tables, db.cached, db.cu, db.max_new,
                              db.max_total, scale_for(case.d), out, lse=lse)
    torch.cuda.synchronize()
    return to_host_bits(out), lse.cpu().numpy().astype(np.float64)


def oracle_prefill(case, bi=0):
    b = case.batches[bi]
    return oracle.prefill_attention(case.pool_k, case.pool_v, b.block_tables, b.prefix_lens,
                                    b.cu_new_lens, b.q, b.k_new, b.v_new, scale_for(case.d),
                                    case.bs)


def check(name, case, got, ref):
    out_bits, lse = got
    o_ref, lse_ref = ref
    compare(name + " out", bf16_to_f64(out_bits), o_ref)
    compare(name + " lse", lse, lse_ref, atol_max=LSE_MAX, atol_mean=LSE_MEAN)


WORKLOADS = [
    W.TINY,
    W.LLAMA3_8B_PREFILL.scaled(prefill=8),
    W.MIXED_70B.scaled(prefill=3, decode=0),
    W.LONG_DOC_SHARED_PROMPT.scaled(prefill=3),
]


@pytest.mark.parametrize("spec", WORKLOADS, ids=lambda s: s.name)
def test_prefill_matches_oracle(gpu_lib, spec):
    say(f"[prefill] {spec.name}")
    case = W.make_case(spec)
    check(spec.name, case, run_prefill(gpu_lib, case), oracle_prefill(case))


def _edge_spec(name, idx, hq, hkv, d, nseq=6):
    return W.WorkloadSpec(name, idx, hq, hkv, d,
                          (W.BatchSpec("prefill", nseq, W.Dist.const(1), W.Dist.const(1)),),
                          ("scale", 1.5))


EDGES = [
    # (name, hq, hkv, d, prefixes, news)
    ("mha_d128", 4, 4, 128, [0, 1, 15, 16, 17, 63], [1, 2, 33, 64, 65, 130]),
    ("gqa2_d64", 8, 4, 64, [0, 5, 64, 100, 128, 33], [1, 31, 32, 97, 1, 200]),
    ("gqa4_d128", 32, 8, 128, [0, 1, 16, 255, 256, 257], [64, 1, 17, 33, 128, 3]),
    ("gqa8_d128", 64, 8, 128, [0, 31, 512, 47, 2, 700], [5, 16, 100, 130, 256, 1]),
    ("gqa8_d64", 16, 2, 64, [0, 200, 3, 64, 1, 9], [300, 7, 16, 1, 64, 40]),
    # one kv head for 16 query heads (8 tokens per query tile); a prefix of 132 blocks, past
    # the 64-entry block-table chunk each wave keeps in registers
    ("mqa16_d128", 16, 1, 128, [0, 100, 1000, 3, 16, 2100], [1, 40, 9, 300, 16, 2]),
    # sequences with no new tokens between others: no output rows, nothing launched for them
    ("empty_rows", 32, 8, 128, [5, 0, 300, 17, 1024, 0], [0, 3, 0, 50, 0, 1]),
    # a group of 7 query heads (28/4): tokens straddle the 32-column waves and the output
    # rows of one store instruction belong to different tokens
    ("gqa7_d128", 28, 4, 128, [0, 77, 16, 500, 1, 260], [1, 45, 64, 9, 130, 33]),
    # a group of 32 (one token per wave), head dim 64 (8 output rows per store instruction)
    ("mqa32_d64", 32, 1, 64, [3, 0, 129, 640, 48, 2], [17, 70, 1, 5, 40, 128]),
]


@pytest.mark.parametrize("edge", EDGES, ids=lambda e: e[0])
def test_prefill_edge_shapes(gpu_lib, edge):
    name, hq, hkv, d, prefixes, news = edge
    say(f"[prefill] edge {name}")
    spec = _edge_spec(name, 100 + EDGES.index(edge), hq, hkv, d, len(prefixes))
    case = W.make_case(spec, prefix_override=[prefixes], new_override=[news])
    check(name, case, run_prefill(gpu_lib, case), oracle_prefill(case))


def test_prefill_host_maxima_are_upper_bounds(gpu_lib):
    """max_new_len and max_total_len only size the launch: larger values give the same bits
    (the extra query tiles are empty)."""
    import torch
    say("[prefill] inflated host maxima")
    case = W.make_case(W.LLAMA3_8B_PREFILL.scaled(prefill=4))
    b = case.batches[0]
    pk, pv = dev_pools(case)
    db = DevBatch(b)
    gpu_lib.pkv_kv_append(pk, pv, db.k_new, db.v_new, db.tables, db.cached, db.cu, db.max_new)
    outs = []
    wide = int(b.block_tables.shape[1]) * case.bs  # the most the table can describe
    for mn, mt in ((db.max_new, db.max_total), (3 * db.max_new, wide)):
        out = torch.empty((b.total_new, case.hq, case.d), dtype=torch.bfloat16, device="cuda")
        gpu_lib.pkv_prefill_attention(pk, pv, db.q, db.tables, db.cached, db.cu, mn, mt,
                                      scale_for(case.d), out)
        torch.cuda.synchronize()
        outs.append(to_host_bits(out))
    assert np.array_equal(outs[0], outs[1])


def test_prefill_is_deterministic_and_placement_invariant(gpu_lib):
    """Same inputs -> identical bits; the same logical data under another block placement
    -> identical bits (the kernel's arithmetic depends on key positions only)."""
    say("[prefill] determinism / placement invariance")
    spec = W.LLAMA3_8B_PREFILL.scaled(prefill=5)
    a = W.make_case(spec)
    out1, lse1 = run_prefill(gpu_lib, a)
    out2, lse2 = run_prefill(gpu_lib, W.make_case(spec))
    assert np.array_equal(out1, out2) and np.array_equal(lse1, lse2)
    # re-place every sequence's blocks with a different permutation, carrying the data along
    b = a.batches[0]
    rng = np.random.default_rng(5)
    perm = rng.permutation(a.num_blocks).astype(np.int32)  # old block id -> new block id
    moved = W.plan_case(spec)
    moved.pool_k = np.empty_like(a.pool_k)
    moved.pool_v = np.empty_like(a.pool_v)
    moved.pool_k[perm] = a.pool_k
    moved.pool_v[perm] = a.pool_v
    mb = moved.batches[0]
    mb.block_tables = np.where(b.block_tables >= 0, perm[np.maximum(b.block_tables, 0)], -1)
    mb.block_tables = mb.block_tables.astype(np.int32)
    mb.q, mb.k_new, mb.v_new = b.q, b.k_new, b.v_new
    out3, lse3 = run_prefill(gpu_lib, moved)
    assert np.array_equal(out1, out3) and np.array_equal(lse1, lse3)


@pytest.mark.parametrize("prefixes,news,probes", [
    ([40, 77, 0], [50, 90, 33], ((0, 7), (1, 63), (2, 20))),
    # long cached prefixes: the boundary sits past the first 64-entry table chunk, in the
    # 65th and later key tiles, and (8191 + 32) in the last slot of a block
    ([4096, 5000, 8191], [40, 90, 34], ((0, 0), (1, 63), (2, 32))),
], ids=["short", "long"])
def test_prefill_spike_probes_mask_boundary(gpu_lib, prefixes, news, probes):
    """Plant a key parallel to query (j, h) at position P + j (visible: output ~ its value)
    and at P + j + 1 (hidden: output unaffected). The tolerance alone is blind to a one-key
    mask error at long context; these probes are not."""
    say(f"[prefill] spike probes, prefixes {prefixes}")
    spec = _edge_spec("spike", 130, 8, 2, 128, 3)
    for offset in (0, 1):
        case = W.make_case(spec, prefix_override=[prefixes], new_override=[news])
        b = case.batches[0]
        probes = []
        for i, j in probes:
            h = 5
            row = int(b.cu_new_lens[i]) + j
            qv = bf16_to_f64(b.q[row, h])
            spike = (qv * (320.0 / np.linalg.norm(qv))).astype(np.float32)
            kj = j + offset  # new-token index of the planted key
            krow = int(b.cu_new_lens[i]) + kj
            b.k_new[krow, h // 4] = (spike.view(np.uint32) >> 16).astype(np.uint16)
            b.v_new[krow, h // 4] = np.uint16(0x4120)  # 10.0
            probes.append((row, h))
        out_bits, _ = run_prefill(gpu_lib, case)
        o = bf16_to_f64(out_bits)
        ref, _ = oracle_prefill(case)
        for row, h in probes:
            if offset == 0:
                assert np.max(np.abs(o[row, h] - 10.0)) < 0.1
            else:
                assert np.max(np.abs(o[row, h] - 10.0)) > 4.0
            assert np.max(np.abs(o[row, h] - ref[row, h])) < 2e-2


def test_prefill_constant_values(gpu_lib):
    """V = 1 everywhere a key is visible -> every output element is 1 (up to bf16 rounding of
    the weights, which the normalisation removes)."""
    say("[prefill] constant V")
    spec = W.LLAMA3_8B_PREFILL.scaled(prefill=3)
    case = W.make_case(spec)
    one = np.uint16(0x3F80)
    case.pool_v = np.where(case.pool_v == W.BF16_NAN, case.pool_v, one).astype(np.uint16)
    case.batches[0].v_new = np.full_like(case.batches[0].v_new, one)
    out_bits, _ = run_prefill(gpu_lib, case)
    assert np.max(np.abs(bf16_to_f64(out_bits) - 1.0)) <= 2.0 ** -7
