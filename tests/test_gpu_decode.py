"""GPU tier: paged split-K decode attention through the C ABI against the fp64 oracle.

Each case appends the step's token (position C_i) and then attends over all C_i + 1 keys.
Lengths straddle every split and block boundary; the bar is the prefill bar."""
import numpy as np
import pytest

import oracle
import workloads as W
from tests.gpu_util import (DevBatch, bf16_to_f64, compare, dev_pools, i32, say, scale_for,
                            to_host_bits)
from tests.test_gpu_prefill import LSE_MAX, LSE_MEAN

pytestmark = pytest.mark.gpu


def run_decode(lib, case, bi=0, pools=None):
    import torch
    b = case.batches[bi]
    pk, pv = pools if pools is not None else dev_pools(case)
    db = DevBatch(b)
    nseq = b.n_seqs
    seq_lens = b.prefix_lens + 1
    max_len = int(seq_lens.max())
    out = torch.empty((nseq, case.hq, case.d), dtype=torch.bfloat16, device="cuda")
    lse = torch.empty((nseq, case.hq), dtype=torch.float32, device="cuda")
    ws = lib.alloc_workspace(lib.pkv_decode_workspace_bytes(nseq, case.hq, case.hkv, case.d,
                                                            max_len))
    lib.pkv_kv_append(pk, pv, db.k_new, db.v_new, db.tables, db.cached, db.cu, 1)
    lib.pkv_decode_attention(pk, pv, db.q, db.tables, i32(seq_lens), max_len,
                             scale_for(case.d), out, lse=lse, workspace=ws)
    torch.cuda.synchronize()
    return to_host_bits(out), lse.cpu().numpy().astype(np.float64)


def oracle_decode(case, bi=0):
    b = case.batches[bi]
    return oracle.decode_attention(case.pool_k, case.pool_v, b.block_tables, b.prefix_lens,
                                   b.q, b.k_new, b.v_new, scale_for(case.d), case.bs)


def check(name, got, ref):
    compare(name + " out", bf16_to_f64(got[0]), ref[0])
    compare(name + " lse", got[1], ref[1], atol_max=LSE_MAX, atol_mean=LSE_MEAN)


@pytest.mark.parametrize("spec", [W.LLAMA3_8B_DECODE.scaled(decode=48),
                                  W.MIXED_70B.scaled(prefill=0, decode=24)],
                         ids=lambda s: s.name)
def test_decode_matches_oracle(gpu_lib, spec):
    say(f"[decode] {spec.name}")
    case = W.make_case(spec)
    bi = [k for k, b in enumerate(case.batches) if b.kind == "decode"][0]
    check(spec.name, run_decode(gpu_lib, case, bi), oracle_decode(case, bi))


CONTEXTS = [0, 1, 14, 15, 16, 17, 30, 31, 32, 33, 63, 64, 127, 255, 256, 257, 511, 512, 1000,
            2047, 2048, 4095]


@pytest.mark.parametrize("hq,hkv,d", [(32, 8, 128), (64, 8, 128), (4, 2, 64), (16, 1, 128),
                                      (28, 4, 128)])
def test_decode_split_and_block_boundaries(gpu_lib, hq, hkv, d):
    say(f"[decode] boundaries hq={hq} hkv={hkv} d={d}")
    spec = W.WorkloadSpec(f"decode_edges_{hq}_{hkv}_{d}", 140 + hq + d, hq, hkv, d,
                          (W.BatchSpec("decode", len(CONTEXTS), W.Dist.const(1),
                                       W.Dist.const(1)),), ("scale", 1.25))
    case = W.make_case(spec, prefix_override=[CONTEXTS])
    check(spec.name, run_decode(gpu_lib, case), oracle_decode(case))


def test_decode_long_contexts_in_long_splits(gpu_lib):
    """Many sequences keep the grid full, so the split stays long and a split spans several
    64-block chunks of the block table; a few long contexts cross chunk and split
    boundaries."""
    say("[decode] long contexts, long splits")
    longs = [1023, 1024, 1025, 2049, 4096, 4097, 16383, 16384]
    ctx = longs + [1 + (7 * j) % 40 for j in range(310)]
    spec = W.WorkloadSpec("decode_long_splits", 151, 32, 8, 128,
                          (W.BatchSpec("decode", len(ctx), W.Dist.const(1), W.Dist.const(1)),),
                          ("scale", 1.25))
    case = W.make_case(spec, prefix_override=[ctx])
    check(spec.name, run_decode(gpu_lib, case), oracle_decode(case))


def test_decode_small_batch_uses_short_splits(gpu_lib):
    """Few sequences -> the split shrinks to keep the grid full; results must not change
    beyond rounding."""
    say("[decode] small batch")
    spec = W.WorkloadSpec("decode_small", 150, 32, 8, 128,
                          (W.BatchSpec("decode", 2, W.Dist.const(1), W.Dist.const(1)),),
                          ("scale", 1.25))
    case = W.make_case(spec, prefix_override=[[3000, 77]])
    check(spec.name, run_decode(gpu_lib, case), oracle_decode(case))


def test_decode_is_deterministic(gpu_lib):
    say("[decode] determinism")
    spec = W.LLAMA3_8B_DECODE.scaled(decode=16)
    a = run_decode(gpu_lib, W.make_case(spec))
    b = run_decode(gpu_lib, W.make_case(spec))
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])


def test_decode_equals_single_token_prefill(gpu_lib):
    """One decode step == a prefill of one new token over the same cache (both within the
    tolerance of the oracle, and of each other)."""
    from tests.test_gpu_prefill import run_prefill
    say("[decode] == prefill N=1")
    spec = W.LLAMA3_8B_DECODE.scaled(decode=12)
    case = W.make_case(spec)
    d_out, _ = run_decode(gpu_lib, case)
    case2 = W.make_case(spec)
    case2.batches[0].kind = "prefill"
    p_out, _ = run_prefill(gpu_lib, case2)
    compare("decode vs prefill", bf16_to_f64(d_out), bf16_to_f64(p_out))


def _oracle_first_keys(case, b, seq_lens_cut, scale):
    """Decode of each sequence's query over its first seq_lens_cut[i] cached keys (no append)."""
    g = case.hq // case.hkv
    out = np.zeros((b.n_seqs, case.hq, case.d))
    lse = np.zeros((b.n_seqs, case.hq))
    for i in range(b.n_seqs):
        L = int(seq_lens_cut[i])
        kc, vc = oracle.gather_seq(case.pool_k, case.pool_v, b.block_tables[i], L, case.bs)
        kf, vf = oracle.bf16_bits_to_f64(kc), oracle.bf16_bits_to_f64(vc)
        qi = oracle.bf16_bits_to_f64(b.q[i])
        for h in range(case.hq):
            o, l = oracle.softmax_attention(qi[h][None], kf[:, h // g], vf[:, h // g], [L], scale)
            out[i, h], lse[i, h] = o[0], l[0]
    return out, lse


@pytest.mark.parametrize("hq,hkv,d,ctx,max_len,cut", [
    # one split per sequence planned (grid of 2048 waves): the over-long row is cut to 4096
    (16, 8, 64, [4200] + [20] * 255, 4096, 4096),
    # five 64-key splits planned: the over-long row is cut to 5 x 64 keys
    (32, 8, 128, [1000, 50, 60, 70], 300, 320),
])
def test_decode_over_long_length_is_cut_to_the_planned_splits(gpu_lib, hq, hkv, d, ctx, max_len,
                                                              cut):
    """A sequence longer than the host's max_seq_len (a broken caller contract) is cut to the
    splits the launch planned: the call stays inside its workspace (no split beyond the
    planned ones, no partial result without a workspace slot) and attends over that many
    keys; every other row is unaffected."""
    import torch
    say(f"[decode] over-long length hq={hq} hkv={hkv} d={d} B={len(ctx)} max_seq_len={max_len}")
    spec = W.WorkloadSpec(f"decode_overlong_{hq}_{d}", 160 + d, hq, hkv, d,
                          (W.BatchSpec("decode", len(ctx), W.Dist.const(1),
                                       W.Dist.const(1)),), ("scale", 1.25))
    case = W.make_case(spec, prefix_override=[ctx])
    b = case.batches[0]
    pk, pv = dev_pools(case)
    db = DevBatch(b)
    lens = np.asarray(ctx, dtype=np.int32)   # every key cached: no append in this test
    out = torch.empty((b.n_seqs, hq, d), dtype=torch.bfloat16, device="cuda")
    lse = torch.empty((b.n_seqs, hq), dtype=torch.float32, device="cuda")
    ws = gpu_lib.alloc_workspace(gpu_lib.pkv_decode_workspace_bytes(b.n_seqs, hq, hkv, d,
                                                                    max_len))
    assert b.block_tables.shape[1] * 16 >= max_len
    gpu_lib.pkv_decode_attention(pk, pv, db.q, db.tables, i32(lens), max_len, scale_for(d), out,
                                 lse=lse, workspace=ws)
    torch.cuda.synchronize()
    ref = _oracle_first_keys(case, b, np.minimum(lens, cut), scale_for(d))
    check(spec.name, (to_host_bits(out), lse.cpu().numpy().astype(np.float64)), ref)


def test_decode_spike_probes_at_long_context(gpu_lib):
    """Spike keys (parallel to the query, large norm, value 10) decide the output alone when
    visible: one in the middle of a long context (inside one split of several), one at the
    step's own appended token (position C), each ~10 after the merge. A spike in the stale
    slot C + 1 of the last block (never appended) must stay invisible."""
    import torch
    say("[decode] spike probes at long context")
    ctx = [4100, 6000, 9000, 5005]
    spec = W.WorkloadSpec("decode_spikes", 161, 16, 4, 128,
                          (W.BatchSpec("decode", len(ctx), W.Dist.const(1), W.Dist.const(1)),),
                          ("scale", 1.25))
    case = W.make_case(spec, prefix_override=[ctx])
    b = case.batches[0]
    g = case.hq // case.hkv
    h = 5
    ten = np.uint16(0x4120)

    def spike_bits(i):
        qv = bf16_to_f64(b.q[i, h])
        sp = (qv * (320.0 / np.linalg.norm(qv))).astype(np.float32)
        return (sp.view(np.uint32) >> 16).astype(np.uint16)

    def plant(i, t):
        blk, slot = int(b.block_tables[i, t // 16]), t % 16
        kb = spike_bits(i)
        case.pool_k[blk, h // g, :, slot, :] = kb.reshape(-1, 8)
        case.pool_v[blk, h // g, :, slot] = ten

    plant(0, 2049)                      # mid-context, cached
    b.k_new[1, h // g] = spike_bits(1)  # the appended token itself (position C)
    b.v_new[1, h // g] = ten
    plant(2, 7777)                      # mid-context, cached
    assert ctx[3] % 16 <= 13
    plant(3, ctx[3] + 1)                # stale slot after the appended token: hidden
    got = run_decode(gpu_lib, case)
    ref = oracle_decode(case)
    o = bf16_to_f64(got[0])
    for i in range(3):
        assert np.max(np.abs(o[i, h] - 10.0)) < 0.1, (i, o[i, h][:4])
    assert np.max(np.abs(o[3, h] - 10.0)) > 4.0
    check("decode spikes", got, ref)
