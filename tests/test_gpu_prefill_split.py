"""GPU tier: the prefill's plan (key split, longest-first order), through the C ABI, against
the fp64 oracle.

A batch whose work items cannot fill the chip (few sequences, few new tokens) and whose keys
are long runs with its keys cut at multiples of a split size when the caller passes the
workspace pkv_prefill_workspace_bytes asks for: rows whose keys all fall in the first split
finish there, every other row is merged from one partial result per split it reaches. Same
bar as the unsplit prefill (max-abs 2e-2, mean-abs 2e-3, LSE bound of test_gpu_prefill);
cases cover rows ending in the first split next to merged rows, prefixes ending exactly at
and around split boundaries, head ratios 1, 4 and 8, both head dims, and spike keys planted
on both sides of a split boundary (the tolerance alone is blind to a one-key error)."""
import numpy as np
import pytest

import workloads as W
from tests.gpu_util import DevBatch, bf16_to_f64, dev_pools, say, scale_for, to_host_bits
from tests.test_gpu_prefill import _edge_spec, check, oracle_prefill

pytestmark = pytest.mark.gpu


def nsplit_of(case, nbytes):
    """The number of splits a workspace size stands for."""
    b = case.batches[0]
    return nbytes // (b.total_new * case.hq * (case.d + 2) * 4)


def split_bytes(lib, case):
    b = case.batches[0]
    return lib.pkv_prefill_workspace_bytes(b.n_seqs, b.total_new, case.hq, case.hkv, case.d,
                                           int(b.new_lens.max()),
                                           int((b.prefix_lens + b.new_lens).max()))


def run(lib, case, split=True):
    """Append, then prefill with the split's workspace (split=True) or none; returns (out bits,
    lse, workspace bytes)."""
    import torch
    b = case.batches[0]
    pk, pv = dev_pools(case)
    db = DevBatch(b)
    nbytes = split_bytes(lib, case)
    ws = lib.alloc_workspace(nbytes) if split and nbytes else None
    out = torch.empty((b.total_new, case.hq, case.d), dtype=torch.bfloat16, device="cuda")
    lse = torch.empty((b.total_new, case.hq), dtype=torch.float32, device="cuda")
    lib.pkv_kv_append(pk, pv, db.k_new, db.v_new, db.tables, db.cached, db.cu, db.max_new)
    lib.pkv_prefill_attention(pk, pv, db.q, db.tables, db.cached, db.cu, db.max_new,
                              db.max_total, scale_for(case.d), out, lse=lse, workspace=ws)
    torch.cuda.synchronize()
    return to_host_bits(out), lse.cpu().numpy().astype(np.float64), nbytes


SPLIT_CASES = [
    # (name, hq, hkv, d, prefixes, news)
    # every row merged from 10 splits of 1024 keys
    ("two_long_gqa4", 32, 8, 128, [5000, 9100], [37, 150]),
    # split size 2048: tokens j < 1948 end in the first split, the rest are merged
    ("rows_end_in_split0", 32, 8, 128, [100], [3000]),
    # one query head per kv head, head dim 64: prefixes ending at (2047), just past (1024 + 1)
    # and well past a boundary; a single new token
    ("mha_d64", 4, 4, 64, [2047, 1025, 6000], [1, 64, 200]),
    # 8 query heads per kv head, split size 1024: the first token of one sequence ends in the
    # first split (its last key is 1023), the next one does not
    ("gqa8_ragged", 64, 8, 128, [1023, 4100], [17, 260]),
    # sequences without new tokens (no rows, no work items) between split ones, and keys past
    # 8192 (so the plan also orders the sequences, the empty ones last)
    ("empty_rows_ordered", 32, 8, 128, [5000, 0, 9000, 3000, 64], [0, 40, 100, 0, 7]),
]


@pytest.mark.parametrize("c", SPLIT_CASES, ids=lambda c: c[0])
def test_split_prefill_matches_oracle(gpu_lib, c):
    name, hq, hkv, d, prefixes, news = c
    say(f"[prefill split] {name}")
    spec = _edge_spec(name, 160 + SPLIT_CASES.index(c), hq, hkv, d, len(prefixes))
    case = W.make_case(spec, prefix_override=[prefixes], new_override=[news])
    out, lse, nbytes = run(gpu_lib, case)
    assert nbytes > 0, "the case was meant to split"
    check(name, case, (out, lse), oracle_prefill(case))


def test_split_is_deterministic_and_agrees_with_unsplit(gpu_lib):
    """Two split runs give identical bits; the unsplit launch (no workspace) of the same batch
    meets the same bar against the oracle."""
    say("[prefill split] determinism, unsplit agreement")
    spec = _edge_spec("split_det", 170, 32, 8, 128, 2)
    case = W.make_case(spec, prefix_override=[[3000, 7000]], new_override=[[100, 41]])
    a = run(gpu_lib, case)
    b = run(gpu_lib, W.make_case(spec, prefix_override=[[3000, 7000]],
                                 new_override=[[100, 41]]))
    assert a[2] > 0
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])
    u = run(gpu_lib, case, split=False)
    ref = oracle_prefill(case)
    check("unsplit", case, u[:2], ref)
    check("split", case, a[:2], ref)


# (sequence, query token j, token index of the planted key, visible?) with 8 query / 2 kv
# heads, three sequences of P = 100 cached and N = 3000 new tokens: 564 work items, so the
# keys are cut into 4 splits of 1024, and key positions 1023 | 1024 (token indices
# 923 | 924) sit on both sides of the first boundary.
SPIKES = [
    (0, 923, 923, True),      # a row ending in the first split sees its last key (1023)
    (0, 923, 924, False),     # ... and not the first key of the next split
    (1, 924, 924, True),      # a merged row sees the first key of its second split
    (1, 924, 925, False),
    (2, 2500, 923, True),     # a merged row sees a key at the end of its first split
    (2, 2500, 2501, False),
]


@pytest.mark.parametrize("probe", SPIKES, ids=lambda p: f"s{p[0]}_j{p[1]}_k{p[2]}")
def test_split_spike_probes_at_boundary(gpu_lib, probe):
    """A key parallel to query (j, h), planted at token index kj: the output is ~ its value
    when the key is visible to the query and unaffected when it is not."""
    i, j, kj, visible = probe
    say(f"[prefill split] spike seq {i} query {j} key {kj}")
    spec = _edge_spec("split_spike", 180, 8, 2, 128, 3)
    case = W.make_case(spec, prefix_override=[[100, 100, 100]],
                       new_override=[[3000, 3000, 3000]])
    b = case.batches[0]
    h = 5
    row = int(b.cu_new_lens[i]) + j
    qv = bf16_to_f64(b.q[row, h])
    spike = (qv * (320.0 / np.linalg.norm(qv))).astype(np.float32)
    krow = int(b.cu_new_lens[i]) + kj
    b.k_new[krow, h // 4] = (spike.view(np.uint32) >> 16).astype(np.uint16)
    b.v_new[krow, h // 4] = np.uint16(0x4120)  # 10.0
    out, lse, nbytes = run(gpu_lib, case)
    assert nsplit_of(case, nbytes) == 4
    o = bf16_to_f64(out)
    ref, _ = oracle_prefill(case)
    if visible:
        assert np.max(np.abs(o[row, h] - 10.0)) < 0.1
    else:
        assert np.max(np.abs(o[row, h] - 10.0)) > 4.0
    assert np.max(np.abs(o[row, h] - ref[row, h])) < 2e-2


def test_split_long_prefix_few_tuples_full_size(gpu_lib):
    """The workload the split is for, at full size (4 tuples of 24-32k cached tokens, short
    suffixes: 224 work items, so 8 splits of 4096 keys), against the oracle."""
    say("[prefill split] long_prefix_few_tuples, full size")
    case = W.make_case(W.LONG_PREFIX_FEW_TUPLES)
    out, lse, nbytes = run(gpu_lib, case)
    assert nsplit_of(case, nbytes) == 8
    check("long_prefix_few_tuples", case, (out, lse), oracle_prefill(case))


def test_ordered_prefill_is_bit_identical(gpu_lib):
    """With a workspace, a batch whose keys reach 8192 takes its sequences longest first (2048
    work items here, so no split): the order moves work items, not arithmetic, so the output is
    bit-identical to the launch without a workspace, and meets the bar against the oracle."""
    say("[prefill plan] longest-first order")
    prefixes = [300, 9000, 40, 5000, 1200, 7000, 16, 2500, 600, 8100, 64, 3000, 90, 4000, 128, 6000]
    news = [512, 17, 300, 128, 64, 512, 1, 200, 480, 33, 256, 100, 512, 7, 150, 90]
    spec = _edge_spec("order", 190, 32, 8, 128, len(prefixes))
    case = W.make_case(spec, prefix_override=[prefixes], new_override=[news])
    a = run(gpu_lib, case)
    assert a[2] == 256, "ordered, not split"
    u = run(gpu_lib, W.make_case(spec, prefix_override=[prefixes], new_override=[news]),
            split=False)
    assert np.array_equal(a[0], u[0]) and np.array_equal(a[1], u[1])
    check("ordered", case, a[:2], oracle_prefill(case))
