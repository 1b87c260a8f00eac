"""GPU tier: serving steps captured in a HIP graph and replayed.

The library's append and attention calls launch on the caller's stream and make no host
synchronisation, allocation or memset on the way (with the opt-in PKV_DEBUG_VALIDATE checks
off), so a caller can capture a whole step (here with
torch.cuda.CUDAGraph, whose capture stream is the current stream the bindings pass on):
  * the decode step: the one-token append, then the allocation-free decode (its workspace is
    the library's fixed per-GPU array, so the graph holds no allocation of its own);
  * the mixed-layer step: the suffix append, the decode-token append, then the fused mixed
    launch with a workspace allocated before the capture;
  * the suffix append and the prefill with its plan (ordering, key-split and merge kernels).
Each graph is replayed three times with fresh inputs copied into its static buffers in
between (eager copies and a synchronisation between replays). Every replay must equal, bit for
bit, the same calls made eagerly on a copy of the pool, pools included, and meet the oracle's
bar."""
import numpy as np
import pytest

import oracle
import workloads as W
from tests.gpu_util import (DevBatch, bf16_to_f64, compare, dev_pools, i32, say, scale_for,
                            to_host_bits)
from tests.test_gpu_prefill import LSE_MAX, LSE_MEAN

pytestmark = pytest.mark.gpu

REPLAYS = 3


def _fresh(gen, like):
    """New N(0,1) bf16 values with the shape of `like` (a device tensor)."""
    import torch
    return torch.randn(like.shape, generator=gen, device="cuda").to(torch.bfloat16)


def _bits_equal(a, b):
    import torch
    return bool(torch.equal(a.view(torch.int16) if a.dtype == torch.bfloat16 else
                            a.view(torch.int32),
                            b.view(torch.int16) if b.dtype == torch.bfloat16 else
                            b.view(torch.int32)))


def test_decode_step_graph_replays(gpu_lib):
    import torch
    lib = gpu_lib
    spec = W.WorkloadSpec("graph_decode", 240, 32, 8, 128,
                          (W.BatchSpec("decode", 40, W.Dist.uniform(100, 6000),
                                       W.Dist.const(1)),), ("scale", 1.25))
    case = W.make_case(spec)
    b = case.batches[0]
    say(f"[graph] decode step: {b.n_seqs} sequences, contexts up to {int(b.prefix_lens.max())}")
    pk, pv = dev_pools(case)
    pk_e, pv_e = pk.clone(), pv.clone()
    db = DevBatch(b)
    seq_lens = i32(b.prefix_lens + 1)
    max_len = int(b.prefix_lens.max()) + 1
    scale = scale_for(case.d)
    # static buffers of the graph, and the eager run's own
    q_s, kn_s, vn_s = db.q.clone(), db.k_new.clone(), db.v_new.clone()
    out_s = torch.empty((b.n_seqs, case.hq, case.d), dtype=torch.bfloat16, device="cuda")
    lse_s = torch.empty((b.n_seqs, case.hq), dtype=torch.float32, device="cuda")
    out_e, lse_e = torch.empty_like(out_s), torch.empty_like(lse_s)

    def step(pool_k, pool_v, q, kn, vn, out, lse):
        lib.pkv_kv_append(pool_k, pool_v, kn, vn, db.tables, db.cached, db.cu, 1)
        lib.pkv_decode_attention_noalloc(pool_k, pool_v, q, db.tables, seq_lens, max_len, scale,
                                         out, lse=lse)

    # one eager call first on the graph's pool (the library takes the scratch array's device
    # address on its first call on a device)
    step(pk, pv, q_s, kn_s, vn_s, out_s, lse_s)
    step(pk_e, pv_e, q_s, kn_s, vn_s, out_e, lse_e)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step(pk, pv, q_s, kn_s, vn_s, out_s, lse_s)
    gen = torch.Generator(device="cuda")
    gen.manual_seed(2607)
    for r in range(REPLAYS):
        q, kn, vn = _fresh(gen, q_s), _fresh(gen, kn_s), _fresh(gen, vn_s)
        q_s.copy_(q)
        kn_s.copy_(kn)
        vn_s.copy_(vn)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        step(pk_e, pv_e, q, kn, vn, out_e, lse_e)
        torch.cuda.synchronize()
        say(f"  replay {r + 1}")
        assert _bits_equal(out_s, out_e), f"replay {r + 1}: output differs from the eager calls"
        assert _bits_equal(lse_s, lse_e), f"replay {r + 1}: lse differs from the eager calls"
        assert _bits_equal(pk, pk_e) and _bits_equal(pv, pv_e), f"replay {r + 1}: pools differ"
        o, l = oracle.decode_attention(case.pool_k, case.pool_v, b.block_tables, b.prefix_lens,
                                       to_host_bits(q), to_host_bits(kn), to_host_bits(vn),
                                       scale, case.bs)
        compare(f"replay {r + 1} vs oracle", bf16_to_f64(to_host_bits(out_s)), o)
        compare(f"replay {r + 1} lse vs oracle", lse_s.cpu().numpy().astype(np.float64), l,
                atol_max=LSE_MAX, atol_mean=LSE_MEAN)


def test_mixed_step_graph_replays(gpu_lib):
    import torch
    lib = gpu_lib
    spec = W.MIXED_70B.scaled(prefill=4, decode=24)
    case = W.make_case(spec)
    bp, bd = case.batches
    say(f"[graph] mixed step: {bp.n_seqs} prefill tuples ({bp.total_new} new tokens), "
        f"{bd.n_seqs} decoding tuples")
    pk, pv = dev_pools(case)
    pk_e, pv_e = pk.clone(), pv.clone()
    dp, dd = DevBatch(bp), DevBatch(bd)
    d_lens = i32(bd.prefix_lens + 1)
    d_max = int(bd.prefix_lens.max()) + 1
    scale = scale_for(case.d)
    ws = lib.alloc_workspace(lib.pkv_decode_workspace_bytes(bd.n_seqs, case.hq, case.hkv,
                                                            case.d, d_max))
    ws_e = lib.alloc_workspace(lib.pkv_decode_workspace_bytes(bd.n_seqs, case.hq, case.hkv,
                                                              case.d, d_max))
    ins_s = [dp.q.clone(), dp.k_new.clone(), dp.v_new.clone(), dd.q.clone(), dd.k_new.clone(),
             dd.v_new.clone()]

    def outs():
        return [torch.empty((bp.total_new, case.hq, case.d), dtype=torch.bfloat16, device="cuda"),
                torch.empty((bp.total_new, case.hq), dtype=torch.float32, device="cuda"),
                torch.empty((bd.n_seqs, case.hq, case.d), dtype=torch.bfloat16, device="cuda"),
                torch.empty((bd.n_seqs, case.hq), dtype=torch.float32, device="cuda")]

    out_s, out_e = outs(), outs()

    def step(pool_k, pool_v, ins, o, w):
        pq, pkn, pvn, dq, dkn, dvn = ins
        lib.pkv_kv_append(pool_k, pool_v, pkn, pvn, dp.tables, dp.cached, dp.cu, dp.max_new)
        lib.pkv_kv_append(pool_k, pool_v, dkn, dvn, dd.tables, dd.cached, dd.cu, 1)
        lib.pkv_mixed_attention(pool_k, pool_v, scale, pq, dp.tables, dp.cached, dp.cu,
                                dp.max_new, dp.max_total, o[0], dq, dd.tables, d_lens, d_max,
                                o[2], lse=o[1], d_lse=o[3], workspace=w)

    step(pk, pv, ins_s, out_s, ws)
    step(pk_e, pv_e, ins_s, out_e, ws_e)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step(pk, pv, ins_s, out_s, ws)
    gen = torch.Generator(device="cuda")
    gen.manual_seed(2608)
    for r in range(REPLAYS):
        ins = [_fresh(gen, t) for t in ins_s]
        for dst, src in zip(ins_s, ins):
            dst.copy_(src)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        step(pk_e, pv_e, ins, out_e, ws_e)
        torch.cuda.synchronize()
        say(f"  replay {r + 1}")
        for k, name in enumerate(["prefill out", "prefill lse", "decode out", "decode lse"]):
            assert _bits_equal(out_s[k], out_e[k]), f"replay {r + 1}: {name} differs"
        assert _bits_equal(pk, pk_e) and _bits_equal(pv, pv_e), f"replay {r + 1}: pools differ"
        if r == 0:
            h = [to_host_bits(t) for t in ins]
            ro, rl = oracle.prefill_attention(case.pool_k, case.pool_v, bp.block_tables,
                                              bp.prefix_lens, bp.cu_new_lens, h[0], h[1], h[2],
                                              scale, case.bs)
            compare("replay 1 prefill vs oracle", bf16_to_f64(to_host_bits(out_s[0])), ro)
            compare("replay 1 prefill lse vs oracle", out_s[1].cpu().numpy().astype(np.float64),
                    rl, atol_max=LSE_MAX, atol_mean=LSE_MEAN)
            do, dl = oracle.decode_attention(case.pool_k, case.pool_v, bd.block_tables,
                                             bd.prefix_lens, h[3], h[4], h[5], scale, case.bs)
            compare("replay 1 decode vs oracle", bf16_to_f64(to_host_bits(out_s[2])), do)
            compare("replay 1 decode lse vs oracle", out_s[3].cpu().numpy().astype(np.float64),
                    dl, atol_max=LSE_MAX, atol_mean=LSE_MEAN)


def test_prefill_plan_graph_replays(gpu_lib):
    """The prefill with its plan (key split and merge, longest-first order; three launches)
    after the suffix append, captured and replayed."""
    import torch
    from tests.test_gpu_prefill import _edge_spec
    lib = gpu_lib
    spec = _edge_spec("graph_plan", 241, 32, 8, 128, 3)
    case = W.make_case(spec, prefix_override=[[9000, 5100, 2600]], new_override=[[37, 150, 90]])
    b = case.batches[0]
    pk, pv = dev_pools(case)
    pk_e, pv_e = pk.clone(), pv.clone()
    db = DevBatch(b)
    scale = scale_for(case.d)
    nbytes = lib.pkv_prefill_workspace_bytes(b.n_seqs, b.total_new, case.hq, case.hkv, case.d,
                                             db.max_new, db.max_total)
    say(f"[graph] prefill with its plan: {b.n_seqs} tuples, workspace {nbytes} B")
    assert nbytes > 256, "the case was meant to split its keys"
    ws, ws_e = lib.alloc_workspace(nbytes), lib.alloc_workspace(nbytes)
    ins_s = [db.q.clone(), db.k_new.clone(), db.v_new.clone()]
    out_s = [torch.empty((b.total_new, case.hq, case.d), dtype=torch.bfloat16, device="cuda"),
             torch.empty((b.total_new, case.hq), dtype=torch.float32, device="cuda")]
    out_e = [torch.empty_like(t) for t in out_s]

    def step(pool_k, pool_v, ins, o, w):
        q, kn, vn = ins
        lib.pkv_kv_append(pool_k, pool_v, kn, vn, db.tables, db.cached, db.cu, db.max_new)
        lib.pkv_prefill_attention(pool_k, pool_v, q, db.tables, db.cached, db.cu, db.max_new,
                                  db.max_total, scale, o[0], lse=o[1], workspace=w)

    step(pk, pv, ins_s, out_s, ws)
    step(pk_e, pv_e, ins_s, out_e, ws_e)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step(pk, pv, ins_s, out_s, ws)
    gen = torch.Generator(device="cuda")
    gen.manual_seed(2609)
    for r in range(REPLAYS):
        ins = [_fresh(gen, t) for t in ins_s]
        for dst, src in zip(ins_s, ins):
            dst.copy_(src)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        step(pk_e, pv_e, ins, out_e, ws_e)
        torch.cuda.synchronize()
        say(f"  replay {r + 1}")
        assert _bits_equal(out_s[0], out_e[0]), f"replay {r + 1}: output differs"
        assert _bits_equal(out_s[1], out_e[1]), f"replay {r + 1}: lse differs"
        assert _bits_equal(pk, pk_e) and _bits_equal(pv, pv_e), f"replay {r + 1}: pools differ"
        if r == 0:
            h = [to_host_bits(t) for t in ins]
            ro, rl = oracle.prefill_attention(case.pool_k, case.pool_v, b.block_tables,
                                              b.prefix_lens, b.cu_new_lens, h[0], h[1], h[2],
                                              scale, case.bs)
            compare("replay 1 vs oracle", bf16_to_f64(to_host_bits(out_s[0])), ro)
            compare("replay 1 lse vs oracle", out_s[1].cpu().numpy().astype(np.float64), rl,
                    atol_max=LSE_MAX, atol_mean=LSE_MEAN)
