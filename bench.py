#!/usr/bin/env python3
"""Benchmark of the paged prefix-reuse attention hot path on one MI355X.

One step = one serving step of a mixed pipelined batch on a 70B-shaped attention layer (64
query / 8 kv heads, head_dim 128, block size 16), the largest configuration that fits one GPU:
128 downstream-operator prefills (cached prefix U[512,2048], new tokens U[128,512]) and 384
decodes (context U[256,4096]) on one pool with random block placement:
    kv_append (the prefill suffixes) -> kv_append (one token per decoding sequence)
    -> mixed attention (the prefill and decode batches fused in one launch)
Block tables come from the library's allocator (checked equal to the generator's placement)
and every input is resident in HBM before the timed region starts. Each timed step is bracketed
by HIP events on the stream the library launches on, and 768 MiB of an unrelated buffer are
read between steps (outside the events) so that no step reads what the previous one left in
the memory-side cache; figures are medians over the steps (p10 / p90 beside them).

Prints ONE JSON line: value = sequences (tuples) per second per attention layer for the
whole step, per-kernel figures, the roofline of the dominant kernel (the fused launch: bf16
matrix cores), the CPU oracle timed on a bounded sample of the same batch, and secondary
workloads (the tiny case in microseconds, the Llama-3-8B prefix-reuse step, the 512-sequence
paged decode, long documents with a shared prompt, reuse vs recompute, achievable peaks, the
scheduler's pipelines). A compact per-workload summary goes to stderr at the end.

    python bench.py [--steps K] [--warmup W] [--no-secondary] [--no-cpu-baseline]
    python bench.py --profile-kernel {prefill,decode,append,mixed,copy} [--workload NAME]
        (launches only that kernel, for rocprofv3 kernel-trace and counter passes)
"""
import argparse
import hashlib
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2516.6   # MI355X dense bf16 matrix-core peak (256 CU x 2.4 GHz x 4096)
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E peak
METRIC = "prefill TFLOP/s (% MFMA peak) + decode HBM GB/s (% peak); tuples/s per layer"


def log(msg):
    print(msg, file=sys.stderr, flush=True)


# ---------------------------------------------------------------------------------------
# algorithmic work: the figures the measured times are divided by
# ---------------------------------------------------------------------------------------
def prefill_flops(prefix, new, hq, d):
    p = prefix.astype(np.float64)
    n = new.astype(np.float64)
    return float(4.0 * d * hq * np.sum(n * p + n * (n + 1) / 2.0))


def prefill_bytes(prefix, new, hq, hkv, d):
    keys = (prefix + new).astype(np.float64)
    kv = np.sum(keys) * hkv * d * 2 * 2
    qo = np.sum(new) * hq * d * 2 * 2
    return float(kv + qo)


def decode_bytes(seq_lens, hq, hkv, d):
    kv = np.sum(seq_lens.astype(np.float64)) * hkv * d * 2 * 2
    qo = len(seq_lens) * hq * d * 2 * 2
    return float(kv + qo)


def decode_flops(seq_lens, hq, d):
    return float(4.0 * d * hq * np.sum(seq_lens.astype(np.float64)))


def append_bytes(total_new, hkv, d):
    return float(total_new * hkv * d * 2 * 2 * 2)  # K and V, read + write


def source_hash(*names):
    h = hashlib.sha256()
    for n in names:
        with open(os.path.join(ROOT, "paper_2607_23815_amd", "csrc", n), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


KERNEL_SOURCES = {
    "prefill": ("prefill.hip", "prefill_impl.h", "device_utils.h"),
    "decode": ("decode.hip", "decode_impl.h", "device_utils.h"),
    "append": ("kv_copy.hip", "device_utils.h"),
    "mixed": ("mixed.hip", "prefill_impl.h", "decode_impl.h", "decode.hip", "device_utils.h"),
}


def traffic_from_profiles(kernel):
    """HBM bytes per launch from the committed counter summary, if it was taken on the
    current kernel source; otherwise None."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        data = json.load(f)
    ent = data.get(kernel)
    if not ent or ent.get("source_hash") != source_hash(*KERNEL_SOURCES[kernel]):
        return None
    return ent.get("hbm_bytes_per_launch")


# ---------------------------------------------------------------------------------------
# workload set-up
# ---------------------------------------------------------------------------------------
class Workload:
    """A generated workload on the device, with tables from the library's allocator."""

    def __init__(self, spec, lib, torch):
        import workloads as W
        from tests.gpu_util import i32
        t0 = time.time()
        case = W.plan_case(spec)
        W.fill_device(case, "cuda")
        self.spec, self.case = spec, case
        self.hq, self.hkv, self.d = spec.num_q_heads, spec.num_kv_heads, spec.head_dim
        self.scale = 1.0 / math.sqrt(self.d)
        # allocator: same placement order; the upstream operator's prefix is committed, the
        # downstream suffix reserved
        t_alloc = time.perf_counter()
        pool = lib.BlockPool(case.num_blocks, spec.block_size, free_order=case.free_order)
        parent = None
        if spec.shared_prompt_tokens:
            parent = pool.create()
            pool.reserve(parent, spec.shared_prompt_tokens)
            pool.commit(parent, spec.shared_prompt_tokens)
        self.batches = []
        for b in case.batches:
            sids = []
            for k in range(b.n_seqs):
                if parent is not None:
                    s = pool.fork(parent, spec.shared_prompt_tokens)
                    st = pool.reserve(s, int(b.prefix_lens[k]) - spec.shared_prompt_tokens)
                else:
                    s = pool.create()
                    st = pool.reserve(s, int(b.prefix_lens[k]))
                assert st == lib.PKV_OK
                pool.commit(s, int(b.prefix_lens[k]) - (spec.shared_prompt_tokens
                                                        if parent is not None else 0))
                assert pool.reserve(s, int(b.new_lens[k])) == lib.PKV_OK
                sids.append(s)
            tables, lens = pool.block_tables(sids, b.max_blocks)
            assert np.array_equal(tables, b.block_tables), "allocator != generator placement"
            assert np.array_equal(lens, b.prefix_lens)
            self.batches.append((b, sids))
        self.alloc_s = time.perf_counter() - t_alloc
        self.pool = pool
        self.parent = parent
        self.dev = []
        for b, _ in self.batches:
            self.dev.append(dict(tables=i32(b.block_tables), cached=i32(b.prefix_lens),
                                 cu=i32(b.cu_new_lens),
                                 max_new=int(b.new_lens.max()) if b.n_seqs else 0,
                                 max_total=int((b.prefix_lens + b.new_lens).max())
                                 if b.n_seqs else 0))
        torch.cuda.synchronize()
        self.setup_s = time.time() - t0

    def decode_followup(self, bi, lib, torch):
        """Tables etc. for one decode step after the prefill: commit the suffix, reserve one
        token per tuple (the allocator adds a block where a tuple's length is a multiple of
        16), and draw that token's q/k/v."""
        from tests.gpu_util import i32
        b, sids = self.batches[bi]
        for k, s in enumerate(sids):
            self.pool.commit(s, int(b.new_lens[k]))
            assert self.pool.reserve(s, 1) == lib.PKV_OK
        ctx = (b.prefix_lens + b.new_lens).astype(np.int32)
        mb = int(-(-(ctx + 1).max() // 16))
        tables, lens = self.pool.block_tables(sids, mb)
        assert np.array_equal(lens, ctx)
        g = torch.Generator(device="cuda")
        g.manual_seed(self.case.seed + 7)
        nseq = b.n_seqs

        def rnd(*shape):
            return torch.randn(*shape, generator=g, device="cuda").to(torch.bfloat16)

        return dict(tables=i32(tables), ctx=i32(ctx), seq_lens=i32(ctx + 1),
                    cu=i32(np.arange(nseq + 1)), max_len=int(ctx.max()) + 1,
                    q=rnd(nseq, self.hq, self.d), k=rnd(nseq, self.hkv, self.d),
                    v=rnd(nseq, self.hkv, self.d), host_tables=tables, host_ctx=ctx)


CLOCK_RAMP_S = 0.1
FLUSH_BYTES = 768 << 20   # read between timed steps: three times the 256 MB MALL


class Flush:
    """Reads FLUSH_BYTES of an unrelated buffer between timed steps (outside the events), so
    that no step finds in the memory-side cache (MALL, 256 MB) or the L2s what the previous
    one left there. A read leaves the caches holding clean lines: a write-based flush would
    leave up to 256 MB of dirty lines whose write-back the next step would pay for."""

    def __init__(self, torch):
        self.torch = torch
        self.buf = torch.ones(FLUSH_BYTES // 4, dtype=torch.int32, device="cuda")

    def __call__(self):
        self.torch.sum(self.buf)


def time_steps(torch, stream, fns, steps, warmup, flush=None):
    """Run the callables `steps` times after `warmup` untimed runs, an event before and after
    each; between steps, `flush` (outside the events). Before the warmup the same callables
    run untimed for at least CLOCK_RAMP_S of wall time: on MI355X the shader clock climbs
    from about 1.7 to about 2.05 GHz over the first ~30 ms of sustained load (measured
    in-kernel), and a serving GPU is never cold. Returns (wall seconds per step including the
    flushes, step seconds [steps], per-callable seconds [steps][len(fns)])."""
    t_ramp = time.perf_counter()
    while time.perf_counter() - t_ramp < CLOCK_RAMP_S:
        for f in fns:
            f()
        torch.cuda.synchronize()
    for _ in range(warmup):
        if flush is not None:
            flush()
        for f in fns:
            f()
    torch.cuda.synchronize()
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(len(fns) + 1)]
          for _ in range(steps)]
    t0 = time.perf_counter()
    for s in range(steps):
        if flush is not None:
            flush()
        ev[s][0].record(stream)
        for k, f in enumerate(fns):
            f()
            ev[s][k + 1].record(stream)
    torch.cuda.synchronize()
    wall = (time.perf_counter() - t0) / steps
    per = np.array([[ev[s][k].elapsed_time(ev[s][k + 1]) for k in range(len(fns))]
                    for s in range(steps)]) / 1e3
    step = np.array([ev[s][0].elapsed_time(ev[s][-1]) for s in range(steps)]) / 1e3
    return wall, step, per


def time_events(torch, stream, fns, steps, warmup, flush=None):
    """time_steps reduced to medians: (wall s per step, step s, [per-callable s])."""
    wall, step, per = time_steps(torch, stream, fns, steps, warmup, flush)
    return wall, med(step), [med(per[:, k]) for k in range(len(fns))]


def dist(x, scale=1e3):
    """median / p10 / p90 of a sample (default: seconds -> ms)."""
    x = np.asarray(x, dtype=np.float64) * scale
    return {"median": float(np.median(x)), "p10": float(np.percentile(x, 10)),
            "p90": float(np.percentile(x, 90))}


def med(x):
    return float(np.median(np.asarray(x, dtype=np.float64)))


def frac(a, p):
    return a / p if p else None


# ---------------------------------------------------------------------------------------
# primary: the mixed 70B-shaped layer (the largest single-GPU configuration)
# ---------------------------------------------------------------------------------------
PRIMARY = "mixed_70b_layer"


def primary(args, lib, torch, flush):
    """One step = the serving step of a mixed pipelined batch on one 70B-shaped attention layer
    (64 query / 8 kv heads, head_dim 128): 128 downstream-operator prefills (cached prefix
    U[512,2048], new U[128,512]) and 384 decodes (context U[256,4096]) on one pool:
        kv_append (the prefill suffixes) -> kv_append (one token per decoding sequence)
        -> mixed attention (prefill and decode fused in one launch, then the split merge).
    The same batch as separate prefill and decode launches is timed beside it."""
    import workloads as W
    from tests.gpu_util import i32
    spec = W.BY_NAME[PRIMARY]
    wl = Workload(spec, lib, torch)
    (bp, _), (bd, _) = wl.batches
    dp, dd = wl.dev
    pk, pv = wl.case.pool_k, wl.case.pool_v
    stream = torch.cuda.current_stream()
    Tp = bp.total_new
    op = torch.empty((Tp, wl.hq, wl.d), dtype=torch.bfloat16, device="cuda")
    od = torch.empty((bd.n_seqs, wl.hq, wl.d), dtype=torch.bfloat16, device="cuda")
    seq_lens = bd.prefix_lens + 1
    sl = i32(seq_lens)
    maxl = int(seq_lens.max())
    ws = lib.alloc_workspace(lib.pkv_decode_workspace_bytes(bd.n_seqs, wl.hq, wl.hkv, wl.d,
                                                            maxl))
    app_p = lambda: lib.pkv_kv_append(pk, pv, bp.k_new, bp.v_new, dp["tables"], dp["cached"],
                                      dp["cu"], dp["max_new"])
    app_d = lambda: lib.pkv_kv_append(pk, pv, bd.k_new, bd.v_new, dd["tables"], dd["cached"],
                                      dd["cu"], 1)
    mixed = lambda: lib.pkv_mixed_attention(pk, pv, wl.scale, bp.q, dp["tables"], dp["cached"],
                                            dp["cu"], dp["max_new"], dp["max_total"], op, bd.q,
                                            dd["tables"], sl, maxl, od, workspace=ws)
    pre = lambda: lib.pkv_prefill_attention(pk, pv, bp.q, dp["tables"], dp["cached"], dp["cu"],
                                            dp["max_new"], dp["max_total"], wl.scale, op)
    dec = lambda: lib.pkv_decode_attention(pk, pv, bd.q, dd["tables"], sl, maxl, wl.scale, od,
                                           workspace=ws)
    wall, step, per = time_steps(torch, stream, [app_p, app_d, mixed], args.steps, args.warmup,
                                 flush)
    _, step_s, per_s = time_steps(torch, stream, [app_p, app_d, pre, dec], args.steps,
                                  args.warmup, flush)
    B = bp.n_seqs + bd.n_seqs
    pflops = prefill_flops(bp.prefix_lens, bp.new_lens, wl.hq, wl.d)
    dflops = decode_flops(seq_lens, wl.hq, wl.d)
    pbytes = prefill_bytes(bp.prefix_lens, bp.new_lens, wl.hq, wl.hkv, wl.d)
    dbytes = decode_bytes(seq_lens, wl.hq, wl.hkv, wl.d)
    abytes_p = append_bytes(Tp, wl.hkv, wl.d)
    abytes_d = append_bytes(bd.n_seqs, wl.hkv, wl.d)
    t_mixed = med(per[:, 2])
    t_pre, t_dec = med(per_s[:, 2]), med(per_s[:, 3])
    ideal_mixed = max((pflops + dflops) / (PEAK_BF16_TFLOPS * 1e12),
                      (pbytes + dbytes) / (PEAK_HBM_GBS * 1e9))
    kernels = {
        "kv_append_suffixes": {"ms": dist(per[:, 0]), "tokens": Tp, "alg_bytes": abytes_p,
                               "GB_s": abytes_p / med(per[:, 0]) / 1e9,
                               "frac_hbm": abytes_p / med(per[:, 0]) / 1e9 / PEAK_HBM_GBS},
        "kv_append_decode_tokens": {"ms": dist(per[:, 1]), "tokens": bd.n_seqs,
                                    "alg_bytes": abytes_d,
                                    "note": f"{abytes_d / 1e6:.1f} MB: launch-latency bound; "
                                            "no roofline claim"},
        "mixed_attention": {"ms": dist(per[:, 2]), "alg_flops": pflops + dflops,
                            "alg_bytes": pbytes + dbytes,
                            "TFLOP_s": (pflops + dflops) / t_mixed / 1e12,
                            "ideal_ms": ideal_mixed * 1e3, "frac_of_ideal": ideal_mixed / t_mixed},
        "separate_launches": {
            "step_ms": dist(step_s),
            "prefill_attention": {"ms": dist(per_s[:, 2]), "alg_flops": pflops,
                                  "TFLOP_s": pflops / t_pre / 1e12,
                                  "frac_mfma": pflops / t_pre / 1e12 / PEAK_BF16_TFLOPS},
            "decode_attention": {"ms": dist(per_s[:, 3]), "alg_bytes": dbytes,
                                 "GB_s": dbytes / t_dec / 1e9,
                                 "frac_hbm": dbytes / t_dec / 1e9 / PEAK_HBM_GBS}},
    }
    achieved = (pflops + dflops) / t_mixed / 1e12
    roof = {"bound": "mfma", "achieved": achieved, "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
            "frac": achieved / PEAK_BF16_TFLOPS, "traffic": traffic_from_profiles("mixed"),
            "kernel": "mixed_kernel (pkv_mixed_attention: order + fused prefill/decode + merge)"}
    t_step = med(step)
    res = {
        "metric": METRIC,
        "value": B / t_step,
        "unit": "tuples/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": t_step * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded N(0,1) bf16; no dataset)",
        "config": {"workload": spec.name, "prefill_tuples": bp.n_seqs,
                   "decode_sequences": bd.n_seqs, "q_heads": wl.hq, "kv_heads": wl.hkv,
                   "head_dim": wl.d, "block_size": 16, "prefix": "U[512,2048]",
                   "new_tokens": "U[128,512]", "decode_context": "U[256,4096]",
                   "new_tokens_total": Tp, "pool_blocks": wl.case.num_blocks,
                   "seed": wl.case.seed,
                   "step": "kv_append(suffixes) -> kv_append(decode tokens) -> "
                           "mixed_attention(prefill + decode)",
                   "timing": f"median of {args.steps} event-timed steps; "
                             f"{FLUSH_BYTES >> 20} MiB read between steps, outside the events"},
        "step_ms": dist(step),
        "wall_ms_per_step_with_flush": wall * 1e3,
        "prefill_tflops": pflops / t_pre / 1e12,
        "decode_gbps": dbytes / t_dec / 1e9,
        "kernels": kernels,
        "roofline": roof,
        "host_allocator_ms": wl.alloc_s * 1e3,
    }
    return res, wl


def cpu_baseline(wl, budget_s=15.0):
    """The oracle on the host cores over a bounded sample of the primary step's sequences,
    in the batch's proportion: prefill tuple k (its suffix over its cached prefix), then
    decode sequences 3k .. 3k+2 (one token over its context), until the budget is spent."""
    import contextlib
    import oracle
    from tests.gpu_util import sub_pool_for, to_host_bits
    try:
        from threadpoolctl import threadpool_limits
    except Exception:  # pragma: no cover
        threadpool_limits = None
    cores = len(os.sched_getaffinity(0))
    (bp, _), (bd, _) = wl.batches
    ratio = bd.n_seqs // max(bp.n_seqs, 1)
    q, kn, vn = to_host_bits(bp.q), to_host_bits(bp.k_new), to_host_bits(bp.v_new)
    dq, dk, dvv = to_host_bits(bd.q), to_host_bits(bd.k_new), to_host_bits(bd.v_new)
    n_pre = n_dec = 0
    t_total = 0.0
    limit = threadpool_limits(limits=cores) if threadpool_limits else contextlib.nullcontext()
    with limit:
        for k in range(bp.n_seqs):
            p, n = int(bp.prefix_lens[k]), int(bp.new_lens[k])
            a, e = int(bp.cu_new_lens[k]), int(bp.cu_new_lens[k + 1])
            pk, pv, row = sub_pool_for(wl.case.pool_k, wl.case.pool_v, bp.block_tables[k], p + n)
            t0 = time.perf_counter()
            oracle.prefill_attention(pk, pv, row[None], [p], [0, n], q[a:e], kn[a:e], vn[a:e],
                                     wl.scale, 16)
            t_total += time.perf_counter() - t0
            n_pre += 1
            for i in range(ratio * k, min(ratio * (k + 1), bd.n_seqs)):
                c = int(bd.prefix_lens[i])
                pk, pv, row = sub_pool_for(wl.case.pool_k, wl.case.pool_v, bd.block_tables[i],
                                           c + 1)
                t0 = time.perf_counter()
                oracle.decode_attention(pk, pv, row[None], [c], dq[i:i + 1], dk[i:i + 1],
                                        dvv[i:i + 1], wl.scale, 16)
                t_total += time.perf_counter() - t0
                n_dec += 1
            if t_total >= budget_s:
                break
    return {"value": (n_pre + n_dec) / t_total, "unit": "tuples/s", "cores": cores,
            "kind": "oracle",
            "sample": f"{n_pre} of {bp.n_seqs} prefill tuples and {n_dec} of {bd.n_seqs} decode "
                      f"sequences of {wl.spec.name} (prefill of the suffix / one decode token "
                      f"each), numpy float64, {t_total:.1f} s"}


# ---------------------------------------------------------------------------------------
# secondary workloads (reported beside the primary line; parity cases of their own)
# ---------------------------------------------------------------------------------------
def secondary(args, lib, torch, flush):
    import workloads as W
    from tests.gpu_util import i32
    out = {}
    stream = torch.cuda.current_stream()
    steps, warm = max(5, args.steps // 2), 2

    # tiny: launch-latency bound, reported in microseconds
    spec = W.TINY
    wl = Workload(spec, lib, torch)
    b, _ = wl.batches[0]
    dv = wl.dev[0]
    pk, pv = wl.case.pool_k, wl.case.pool_v
    o = torch.empty((b.total_new, wl.hq, wl.d), dtype=torch.bfloat16, device="cuda")
    fns = [lambda: lib.pkv_kv_append(pk, pv, b.k_new, b.v_new, dv["tables"], dv["cached"],
                                     dv["cu"], dv["max_new"]),
           lambda: lib.pkv_prefill_attention(pk, pv, b.q, dv["tables"], dv["cached"], dv["cu"],
                                             dv["max_new"], dv["max_total"], wl.scale, o)]
    _, step, per = time_steps(torch, stream, fns, steps, warm, flush)
    # the same step captured in a HIP graph (the library's calls launch on the current stream
    # and neither synchronise nor allocate), timed as one replay per step
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        for fn in fns:
            fn()
    _, gstep, _ = time_steps(torch, stream, [graph.replay], steps, warm, flush)
    out[spec.name] = {"step_us": dist(step, 1e6), "append_us": dist(per[:, 0], 1e6),
                      "prefill_us": dist(per[:, 1], 1e6),
                      "graph_replay_step_us": dist(gstep, 1e6),
                      "note": "launch-latency bound (34 MFLOP); no roofline claim"}
    del wl, pk, pv, graph

    # Llama-3-8B prefix-reuse prefill step (+ the first decode step)
    spec = W.LLAMA3_8B_PREFILL
    wl = Workload(spec, lib, torch)
    b, _ = wl.batches[0]
    dv = wl.dev[0]
    pk, pv = wl.case.pool_k, wl.case.pool_v
    T, B = b.total_new, b.n_seqs
    o = torch.empty((T, wl.hq, wl.d), dtype=torch.bfloat16, device="cuda")
    dec = wl.decode_followup(0, lib, torch)
    do = torch.empty((B, wl.hq, wl.d), dtype=torch.bfloat16, device="cuda")
    ws = lib.alloc_workspace(lib.pkv_decode_workspace_bytes(B, wl.hq, wl.hkv, wl.d,
                                                            dec["max_len"]))
    fns = [lambda: lib.pkv_kv_append(pk, pv, b.k_new, b.v_new, dv["tables"], dv["cached"],
                                     dv["cu"], dv["max_new"]),
           lambda: lib.pkv_prefill_attention(pk, pv, b.q, dv["tables"], dv["cached"], dv["cu"],
                                             dv["max_new"], dv["max_total"], wl.scale, o),
           lambda: lib.pkv_kv_append(pk, pv, dec["k"], dec["v"], dec["tables"], dec["ctx"],
                                     dec["cu"], 1),
           lambda: lib.pkv_decode_attention(pk, pv, dec["q"], dec["tables"], dec["seq_lens"],
                                            dec["max_len"], wl.scale, do, workspace=ws)]
    _, step, per = time_steps(torch, stream, fns, steps, warm, flush)
    flops = prefill_flops(b.prefix_lens, b.new_lens, wl.hq, wl.d)
    abytes = append_bytes(T, wl.hkv, wl.d)
    dbytes = decode_bytes(dec["host_ctx"] + 1, wl.hq, wl.hkv, wl.d)
    tp, ta, td = med(per[:, 1]), med(per[:, 0]), med(per[:, 3])
    out[spec.name] = {"step_ms": dist(step), "tuples_per_s": B / med(step),
                      "append_ms": dist(per[:, 0]), "append_GB_s": abytes / ta / 1e9,
                      "append_frac_hbm": abytes / ta / 1e9 / PEAK_HBM_GBS,
                      "prefill_ms": dist(per[:, 1]), "prefill_TFLOP_s": flops / tp / 1e12,
                      "prefill_frac_mfma": flops / tp / 1e12 / PEAK_BF16_TFLOPS,
                      "decode_token_append_us": dist(per[:, 2], 1e6),
                      "decode_ms": dist(per[:, 3]), "decode_GB_s": dbytes / td / 1e9,
                      "decode_frac_hbm": dbytes / td / 1e9 / PEAK_HBM_GBS}
    del wl, pk, pv, dec

    # paged decode, Llama-3-8B layer
    spec = W.LLAMA3_8B_DECODE
    wl = Workload(spec, lib, torch)
    b, _ = wl.batches[0]
    dv = wl.dev[0]
    pk, pv = wl.case.pool_k, wl.case.pool_v
    B = b.n_seqs
    seq_lens = b.prefix_lens + 1
    sl = i32(seq_lens)
    maxl = int(seq_lens.max())
    o = torch.empty((B, wl.hq, wl.d), dtype=torch.bfloat16, device="cuda")
    ws = lib.alloc_workspace(lib.pkv_decode_workspace_bytes(B, wl.hq, wl.hkv, wl.d, maxl))
    fns = [lambda: lib.pkv_kv_append(pk, pv, b.k_new, b.v_new, dv["tables"], dv["cached"],
                                     dv["cu"], 1),
           lambda: lib.pkv_decode_attention(pk, pv, b.q, dv["tables"], sl, maxl, wl.scale, o,
                                            workspace=ws)]
    _, step, per = time_steps(torch, stream, fns, steps, warm, flush)
    dbytes = decode_bytes(seq_lens, wl.hq, wl.hkv, wl.d)
    td = med(per[:, 1])
    out[spec.name] = {"append_us": dist(per[:, 0], 1e6), "decode_ms": dist(per[:, 1]),
                      "decode_GB_s": dbytes / td / 1e9,
                      "decode_frac_hbm": dbytes / td / 1e9 / PEAK_HBM_GBS,
                      "tuples_per_s": B / med(step)}
    del wl, pk, pv

    # long documents with a shared 512-token prompt (with the workspace that lets the prefill
    # take its sequences longest first)
    spec = W.LONG_DOC_SHARED_PROMPT
    wl = Workload(spec, lib, torch)
    b, _ = wl.batches[0]
    dv = wl.dev[0]
    pk, pv = wl.case.pool_k, wl.case.pool_v
    o = torch.empty((b.total_new, wl.hq, wl.d), dtype=torch.bfloat16, device="cuda")
    nb = lib.pkv_prefill_workspace_bytes(b.n_seqs, b.total_new, wl.hq, wl.hkv, wl.d,
                                         dv["max_new"], dv["max_total"])
    lws = lib.alloc_workspace(nb) if nb else None
    fns = [lambda: lib.pkv_kv_append(pk, pv, b.k_new, b.v_new, dv["tables"], dv["cached"],
                                     dv["cu"], dv["max_new"]),
           lambda: lib.pkv_prefill_attention(pk, pv, b.q, dv["tables"], dv["cached"], dv["cu"],
                                             dv["max_new"], dv["max_total"], wl.scale, o,
                                             workspace=lws)]
    _, step, per = time_steps(torch, stream, fns, steps, warm, flush)
    flops = prefill_flops(b.prefix_lens, b.new_lens, wl.hq, wl.d)
    abytes = append_bytes(b.total_new, wl.hkv, wl.d)
    ta, tp = med(per[:, 0]), med(per[:, 1])
    out[spec.name] = {"append_ms": dist(per[:, 0]), "append_GB_s": abytes / ta / 1e9,
                      "append_frac_hbm": abytes / ta / 1e9 / PEAK_HBM_GBS,
                      "prefill_ms": dist(per[:, 1]), "prefill_TFLOP_s": flops / tp / 1e12,
                      "prefill_frac_mfma": flops / tp / 1e12 / PEAK_BF16_TFLOPS,
                      "tuples_per_s": b.n_seqs / med(step),
                      "prefill_workspace_bytes": nb}
    del wl, pk, pv, lws

    # a batch too small to fill the chip (4 tuples of 24-32k cached tokens, short suffixes):
    # the prefill without a workspace (no key split) and with one (key split + merge)
    spec = W.LONG_PREFIX_FEW_TUPLES
    wl = Workload(spec, lib, torch)
    b, _ = wl.batches[0]
    dv = wl.dev[0]
    pk, pv = wl.case.pool_k, wl.case.pool_v
    lib.pkv_kv_append(pk, pv, b.k_new, b.v_new, dv["tables"], dv["cached"], dv["cu"],
                      dv["max_new"])
    o = torch.empty((b.total_new, wl.hq, wl.d), dtype=torch.bfloat16, device="cuda")
    nb = lib.pkv_prefill_workspace_bytes(b.n_seqs, b.total_new, wl.hq, wl.hkv, wl.d,
                                         dv["max_new"], dv["max_total"])
    ws = lib.alloc_workspace(nb)
    fns = [lambda: lib.pkv_prefill_attention(pk, pv, b.q, dv["tables"], dv["cached"], dv["cu"],
                                             dv["max_new"], dv["max_total"], wl.scale, o),
           lambda: lib.pkv_prefill_attention(pk, pv, b.q, dv["tables"], dv["cached"], dv["cu"],
                                             dv["max_new"], dv["max_total"], wl.scale, o,
                                             workspace=ws)]
    _, step, per = time_steps(torch, stream, fns, steps, warm, flush)
    flops = prefill_flops(b.prefix_lens, b.new_lens, wl.hq, wl.d)
    tu, tsp = med(per[:, 0]), med(per[:, 1])
    out[spec.name] = {"unsplit_ms": dist(per[:, 0]), "unsplit_TFLOP_s": flops / tu / 1e12,
                      "split_ms": dist(per[:, 1]), "split_TFLOP_s": flops / tsp / 1e12,
                      "split_frac_mfma": flops / tsp / 1e12 / PEAK_BF16_TFLOPS,
                      "speedup": tu / tsp, "workspace_MB": nb / 1e6,
                      "note": "prefill key split (workspace given) against the launch without "
                              "a workspace, same inputs; split time includes the merge kernel"}
    del wl, pk, pv, ws
    torch.cuda.empty_cache()
    return out


def reuse_vs_recompute(args, lib, torch, flush=None):
    """Kernel-level analog of the paper's prefix reuse (Section 2.1): one downstream attention
    layer with the cached prefix reused (append the N new tokens, prefill them over P cached
    ones) against the same layer recomputed from scratch (append all P + N tokens, prefill all
    of them), on the same data. The recompute runs first: its append places every token's
    K/V, which the reuse step then reads as its cache."""
    import workloads as W
    from tests.gpu_util import i32
    stream = torch.cuda.current_stream()
    steps, warm = max(5, args.steps // 2), 2

    def one(spec):
        b0 = W.plan_case(spec).batches[0]
        P = b0.prefix_lens.astype(np.int64)
        N = b0.new_lens.astype(np.int64)
        L = P + N
        case = W.plan_case(spec, prefix_override=[np.zeros_like(L)], new_override=[L])
        W.fill_device(case, "cuda")
        b = case.batches[0]
        hq, hkv, d = spec.num_q_heads, spec.num_kv_heads, spec.head_dim
        scale = 1.0 / math.sqrt(d)
        pk, pv = case.pool_k, case.pool_v
        tables = i32(b.block_tables)
        zeros = i32(np.zeros(len(L)))
        cu_r = b.cu_new_lens.astype(np.int64)
        suf = torch.from_numpy(np.concatenate(
            [np.arange(cu_r[i] + P[i], cu_r[i + 1]) for i in range(len(L))])).cuda()
        qs, ks, vs = b.q[suf].contiguous(), b.k_new[suf].contiguous(), b.v_new[suf].contiguous()
        cu_l, cu_n, cached = i32(cu_r), i32(np.concatenate([[0], np.cumsum(N)])), i32(P)
        maxl, maxn = int(L.max()), int(N.max())
        o_r = torch.empty((int(L.sum()), hq, d), dtype=torch.bfloat16, device="cuda")
        o_u = torch.empty((int(N.sum()), hq, d), dtype=torch.bfloat16, device="cuda")
        recompute = [lambda: lib.pkv_kv_append(pk, pv, b.k_new, b.v_new, tables, zeros, cu_l,
                                               maxl),
                     lambda: lib.pkv_prefill_attention(pk, pv, b.q, tables, zeros, cu_l, maxl,
                                                       maxl, scale, o_r)]
        reuse = [lambda: lib.pkv_kv_append(pk, pv, ks, vs, tables, cached, cu_n, maxn),
                 lambda: lib.pkv_prefill_attention(pk, pv, qs, tables, cached, cu_n, maxn, maxl,
                                                   scale, o_u)]
        _, g_r, per_r = time_events(torch, stream, recompute, steps, warm, flush)
        _, g_u, per_u = time_events(torch, stream, reuse, steps, warm, flush)
        f_r = prefill_flops(np.zeros_like(L), L, hq, d)
        f_u = prefill_flops(P, N, hq, d)
        res = {"tuples": int(len(L)), "mean_prefix": float(P.mean()), "mean_new": float(N.mean()),
               "reuse_ms": g_u * 1e3, "recompute_ms": g_r * 1e3, "speedup": g_r / g_u,
               "reuse_prefill_TFLOP_s": f_u / per_u[1] / 1e12,
               "recompute_prefill_TFLOP_s": f_r / per_r[1] / 1e12}
        del case, pk, pv, o_r, o_u, qs, ks, vs
        torch.cuda.empty_cache()
        return res

    out = {W.LLAMA3_8B_PREFILL.name: one(W.LLAMA3_8B_PREFILL)}
    for k, p in enumerate((256, 1024, 4096)):
        spec = W.WorkloadSpec(f"prefix_{p}_new_128", 210 + k, 32, 8, 128,
                              (W.BatchSpec("prefill", 64, W.Dist.const(p), W.Dist.const(128)),),
                              ("scale", 1.25))
        out[spec.name] = one(spec)
    return out


def pipelines(args, lib, torch):
    """Section 5's scheduler driving the attention path: the synthetic pipelines (filter then
    map, a map then a 17-way Cartesian product, three stages) run to completion under each
    policy, every engine step's append, block copies and prefill/decode attention on the GPU
    (one attention layer, Llama-3-8B heads). The KV pool holds about 64 first-stage tuples'
    prefixes, so the table does not fit: blocking execution loses its prefixes to the cache
    (Section 2.2's cliff) while the memory-aware schedule keeps them. gpu_ms is the summed GPU
    time of the steps; the host schedules between steps (wall_ms)."""
    from workloads.pipelines import PIPELINES, make_pipeline
    hq, hkv, d, src_rows = 32, 8, 128, 8192
    g = torch.Generator(device="cuda")
    g.manual_seed(7)

    def rnd(*shape):
        return torch.randn(*shape, generator=g, device="cuda").to(torch.bfloat16)
    q_src, k_src, v_src = rnd(src_rows, hq, d), rnd(src_rows, hkv, d), rnd(src_rows, hkv, d)
    names = {0: "adaptive_virtual", 1: "depth_first", 2: "breadth_first", 3: "sequential",
             4: "blocking"}
    out = {}
    for spec in PIPELINES:
        pd = make_pipeline(spec)
        S = len(pd["suffix"])
        mean0 = float(np.mean(pd["suffix"][0]) + np.mean(pd["out_len"][0]))
        nb = int(64 * math.ceil(mean0 / 16)) + 2048
        predicate = [bool(np.max(pd["out_len"][s]) <= 3) for s in range(S)]
        kw = dict(max_out=64, max_batch=64, static_bound=[8 if p else 0 for p in predicate],
                  initial_bound=[16] * S, pinning=lib.PKV_PIN_VIRTUAL)
        pool_k = torch.zeros((nb, hkv, d // 8, 16, 8), dtype=torch.bfloat16, device="cuda")
        pool_v = torch.zeros((nb, hkv, d, 16), dtype=torch.bfloat16, device="cuda")
        dev = dict(k_cache=pool_k, v_cache=pool_v, q_src=q_src, k_src=k_src, v_src=v_src)
        runs = {}
        plist = [(0, lib.PKV_PIN_VIRTUAL, 0), (0, lib.PKV_PIN_EXPLICIT, 0),
                 (0, lib.PKV_PIN_EXPLICIT, 4096), (1, None, 0), (2, None, 0), (4, None, 0)]
        if spec.num_tuples <= 400:
            plist.append((3, None, 0))
        for policy, pin, budget in plist:
            name = names[policy] if policy != 0 or pin == lib.PKV_PIN_VIRTUAL else \
                "adaptive_explicit"
            if budget:
                name += f"_chunked_{budget}"
            over = {"max_step_tokens": budget}
            if pin is not None:
                over["pinning"] = pin
            cfg = lib.sched_config(policy, nb, **{**kw, **over})
            st, _, bud = lib.pkv_sched_run(cfg, pd["fanout"], pd["suffix"], pd["out_len"],
                                           pd["filtered"], device=dev)
            runs[name] = {k: (round(v, 3) if isinstance(v, float) else int(v))
                          for k, v in st.items()}
            runs[name]["input_tuples_per_s_gpu"] = spec.num_tuples / (st["gpu_ms"] / 1e3)
            log(f"[bench]   {spec.name} {name}: gpu {st['gpu_ms']:.1f} ms, steps "
                f"{st['steps']}, hits {st['hits']}, misses {st['misses']}")
        base = runs["blocking"]["gpu_ms"]
        for r in runs.values():
            r["speedup_vs_blocking"] = base / r["gpu_ms"]
        out[spec.name] = {"num_tuples": spec.num_tuples, "num_blocks": nb, "runs": runs}
        del pool_k, pool_v, dev
        torch.cuda.empty_cache()
    return out


def achievable_peaks(torch):
    """Context for the rooflines, measured on the same GPU in the same run: a library bf16
    GEMM (torch.matmul, 8192^3, both operands contiguous along the reduction dimension, the
    layout hipBLASLt runs fastest here) and a plain 1 GiB device copy (read + write). These
    are what stock library code reaches here, not the datasheet peaks the fractions use."""
    stream = torch.cuda.current_stream()
    n = 8192
    a = torch.randn(n, n, device="cuda").to(torch.bfloat16)
    b = torch.randn(n, n, device="cuda").to(torch.bfloat16)
    bt = b.t()  # [K][N] view of a row-major [N][K] operand
    # best of two timed sets: the first one also settles the library's kernel choice
    gemm = max(2.0 * n ** 3 / time_events(torch, stream, [lambda: torch.matmul(a, bt)], 10, 2)[2][0]
               / 1e12 for _ in range(2))
    del a, b, bt
    m = 1 << 30
    x = torch.empty(m, dtype=torch.uint8, device="cuda")
    y = torch.empty_like(x)
    x.fill_(1)
    _, _, per = time_events(torch, stream, [lambda: y.copy_(x)], 10, 2)
    copy = 2 * m / per[0] / 1e9
    del x, y
    torch.cuda.empty_cache()
    return {"gemm_bf16_8192_TFLOP_s": gemm, "gemm_frac_of_peak": gemm / PEAK_BF16_TFLOPS,
            "copy_1GiB_GB_s": copy, "copy_frac_of_peak": copy / PEAK_HBM_GBS}


def profile_copy(args, torch):
    """A plain device copy of known size (1 GiB read + 1 GiB written per launch): the
    reference that scales the L2<->HBM byte counters to bytes."""
    n = 1 << 30
    a = torch.empty(n, dtype=torch.uint8, device="cuda")
    b = torch.empty_like(a)
    a.fill_(1)
    stream = torch.cuda.current_stream()
    _, _, per = time_events(torch, stream, [lambda: b.copy_(a)], args.steps, args.warmup)
    print(json.dumps({"kernel": "copy", "bytes_read": n, "bytes_written": n,
                      "launches": args.steps + args.warmup, "avg_ms": per[0] * 1e3,
                      "GB_s": 2 * n / per[0] / 1e9}), flush=True)


def profile_mixed(args, lib, torch, wl):
    """The mixed launch (prefill and decode batches of one workload fused) `steps` times."""
    from tests.gpu_util import i32
    kinds = [b.kind for b, _ in wl.batches]
    if kinds != ["prefill", "decode"]:
        raise SystemExit(f"{wl.spec.name} is not a prefill + decode workload")
    (bp, _), (bd, _) = wl.batches
    dp, dd = wl.dev
    pk, pv = wl.case.pool_k, wl.case.pool_v
    lib.pkv_kv_append(pk, pv, bp.k_new, bp.v_new, dp["tables"], dp["cached"], dp["cu"],
                      dp["max_new"])
    lib.pkv_kv_append(pk, pv, bd.k_new, bd.v_new, dd["tables"], dd["cached"], dd["cu"], 1)
    op = torch.empty((bp.total_new, wl.hq, wl.d), dtype=torch.bfloat16, device="cuda")
    od = torch.empty((bd.n_seqs, wl.hq, wl.d), dtype=torch.bfloat16, device="cuda")
    sl = i32(bd.prefix_lens + 1)
    maxl = int(bd.prefix_lens.max()) + 1
    ws = lib.alloc_workspace(lib.pkv_decode_workspace_bytes(bd.n_seqs, wl.hq, wl.hkv, wl.d,
                                                            maxl))
    fn = lambda: lib.pkv_mixed_attention(pk, pv, wl.scale, bp.q, dp["tables"], dp["cached"],
                                         dp["cu"], dp["max_new"], dp["max_total"], op, bd.q,
                                         dd["tables"], sl, maxl, od, workspace=ws)
    stream = torch.cuda.current_stream()
    _, gpu, per = time_events(torch, stream, [fn], args.steps, args.warmup, Flush(torch))
    print(json.dumps({"workload": wl.spec.name, "kernel": "mixed",
                      "launches": args.steps + args.warmup, "avg_ms": per[0] * 1e3}),
          flush=True)


def profile_kernel(args, lib, torch):
    """Launch one kernel of the hot path `steps` times on one workload (for rocprofv3)."""
    import workloads as W
    if args.profile_kernel == "copy":
        return profile_copy(args, torch)
    spec = W.BY_NAME[args.workload]
    wl = Workload(spec, lib, torch)
    if args.profile_kernel == "mixed":
        return profile_mixed(args, lib, torch, wl)
    kind = "decode" if args.profile_kernel == "decode" else "prefill"
    bi = [k for k, (b, _) in enumerate(wl.batches) if b.kind == kind]
    if not bi:
        raise SystemExit(f"{spec.name} has no {kind} batch")
    b, _ = wl.batches[bi[0]]
    dv = wl.dev[bi[0]]
    pk, pv = wl.case.pool_k, wl.case.pool_v
    from tests.gpu_util import i32
    if args.profile_kernel == "append":
        fn = lambda: lib.pkv_kv_append(pk, pv, b.k_new, b.v_new, dv["tables"], dv["cached"],
                                       dv["cu"], max(dv["max_new"], 1))
    elif args.profile_kernel == "prefill":
        out = torch.empty((b.total_new, wl.hq, wl.d), dtype=torch.bfloat16, device="cuda")
        lib.pkv_kv_append(pk, pv, b.k_new, b.v_new, dv["tables"], dv["cached"], dv["cu"],
                          dv["max_new"])
        # the workspace that enables the key split, for a batch too small to fill the chip
        nb = lib.pkv_prefill_workspace_bytes(b.n_seqs, b.total_new, wl.hq, wl.hkv, wl.d,
                                             dv["max_new"], dv["max_total"])
        pws = lib.alloc_workspace(nb) if nb else None
        fn = lambda: lib.pkv_prefill_attention(pk, pv, b.q, dv["tables"], dv["cached"],
                                               dv["cu"], dv["max_new"], dv["max_total"],
                                               wl.scale, out, workspace=pws)
    else:
        seq_lens = b.prefix_lens + 1
        maxl = int(seq_lens.max())
        sl = i32(seq_lens)
        out = torch.empty((b.n_seqs, wl.hq, wl.d), dtype=torch.bfloat16, device="cuda")
        ws = lib.alloc_workspace(lib.pkv_decode_workspace_bytes(b.n_seqs, wl.hq, wl.hkv, wl.d,
                                                                maxl))
        lib.pkv_kv_append(pk, pv, b.k_new, b.v_new, dv["tables"], dv["cached"], dv["cu"], 1)
        fn = lambda: lib.pkv_decode_attention(pk, pv, b.q, dv["tables"], sl, maxl, wl.scale,
                                              out, workspace=ws)
    stream = torch.cuda.current_stream()
    _, gpu, per = time_events(torch, stream, [fn], args.steps, args.warmup, Flush(torch))
    print(json.dumps({"workload": spec.name, "kernel": args.profile_kernel,
                      "launches": args.steps + args.warmup, "avg_ms": per[0] * 1e3}),
          flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--no-secondary", action="store_true")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--profile-kernel", choices=("prefill", "decode", "append", "copy", "mixed"))
    ap.add_argument("--workload", default=PRIMARY)
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: this path needs no collective and runs one "
              "process on one MI355X; tuples are independent, so more GPUs would each run "
              "their own share of them.", file=sys.stderr)
        sys.exit(2)
    import torch
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    from paper_2607_23815_amd import lib
    if args.profile_kernel:
        profile_kernel(args, lib, torch)
        return
    flush = Flush(torch)
    log(f"[bench] primary workload {PRIMARY}, steps={args.steps} warmup={args.warmup}")
    res, wl = primary(args, lib, torch, flush)
    log(f"[bench] primary done: {res['ms_per_step']:.3f} ms/step")
    if not args.no_cpu_baseline:
        log("[bench] cpu baseline (oracle) ...")
        res["cpu_baseline"] = cpu_baseline(wl)
        log("[bench] cpu baseline done")
    else:
        res["cpu_baseline"] = None
    del wl
    torch.cuda.empty_cache()
    if not args.no_secondary:
        log("[bench] secondary workloads ...")
        res["secondary"] = secondary(args, lib, torch, flush)
        res["secondary"]["reuse_vs_recompute"] = reuse_vs_recompute(args, lib, torch, flush)
        res["secondary"]["achievable_peaks"] = achievable_peaks(torch)
        log("[bench] pipelines under the scheduler ...")
        res["secondary"]["pipelines"] = pipelines(args, lib, torch)
        log("[bench] secondary done")
    print(json.dumps(res), flush=True)
    summary(res)


def summary(res):
    """The figures of every workload on a few stderr lines (the JSON line is long)."""
    k = res["kernels"]
    sep = k["separate_launches"]
    log(f"[summary] {PRIMARY}: {res['value']:.0f} seq/s, step {res['ms_per_step']:.3f} ms "
        f"(p10 {res['step_ms']['p10']:.3f}, p90 {res['step_ms']['p90']:.3f}); mixed launch "
        f"{k['mixed_attention']['ms']['median']:.3f} ms = {res['roofline']['achieved']:.0f} TFLOP/s "
        f"({100 * res['roofline']['frac']:.1f}% of bf16 peak); separate: prefill "
        f"{sep['prefill_attention']['ms']['median']:.3f} ms ({sep['prefill_attention']['TFLOP_s']:.0f} "
        f"TF, {100 * sep['prefill_attention']['frac_mfma']:.1f}%), decode "
        f"{sep['decode_attention']['ms']['median']:.3f} ms ({sep['decode_attention']['GB_s']:.0f} GB/s, "
        f"{100 * sep['decode_attention']['frac_hbm']:.1f}%); suffix append "
        f"{k['kv_append_suffixes']['ms']['median']:.3f} ms ({100 * k['kv_append_suffixes']['frac_hbm']:.1f}%)")
    cb = res.get("cpu_baseline")
    if cb:
        log(f"[summary] cpu oracle: {cb['value']:.2f} seq/s on {cb['cores']} cores")
    sec = res.get("secondary")
    if not sec:
        return
    t = sec.get("tiny_prefix_reuse_prefill")
    if t:
        log(f"[summary] tiny: step {t['step_us']['median']:.1f} us (append "
            f"{t['append_us']['median']:.1f}, prefill {t['prefill_us']['median']:.1f}); as a "
            f"HIP graph replay {t['graph_replay_step_us']['median']:.1f} us")
    s = sec.get("llama3_8b_prefix_reuse_prefill")
    if s:
        log(f"[summary] llama3_8b prefix reuse: {s['tuples_per_s']:.0f} tuples/s, prefill "
            f"{s['prefill_ms']['median']:.3f} ms ({100 * s['prefill_frac_mfma']:.1f}%), append "
            f"{100 * s['append_frac_hbm']:.1f}% HBM, decode {100 * s['decode_frac_hbm']:.1f}% HBM")
    s = sec.get("llama3_8b_paged_decode")
    if s:
        log(f"[summary] llama3_8b decode: {s['decode_ms']['median']:.3f} ms "
            f"({s['decode_GB_s']:.0f} GB/s, {100 * s['decode_frac_hbm']:.1f}%), append "
            f"{s['append_us']['median']:.1f} us")
    s = sec.get("long_doc_shared_prompt")
    if s:
        log(f"[summary] long docs: prefill {s['prefill_ms']['median']:.3f} ms "
            f"({s['prefill_TFLOP_s']:.0f} TF, {100 * s['prefill_frac_mfma']:.1f}%), append "
            f"{s['append_ms']['median'] * 1e3:.1f} us ({100 * s['append_frac_hbm']:.1f}%)")
    s = sec.get("long_prefix_few_tuples")
    if s:
        log(f"[summary] long prefix, few tuples: prefill {s['unsplit_ms']['median']:.3f} ms "
            f"unsplit, {s['split_ms']['median']:.3f} ms with the key split "
            f"({s['split_TFLOP_s']:.0f} TF, {s['speedup']:.2f}x)")
    r = sec.get("reuse_vs_recompute")
    if r:
        log("[summary] reuse vs recompute: " + ", ".join(
            f"{n} {v['speedup']:.2f}x" for n, v in r.items()))
    a = sec.get("achievable_peaks")
    if a:
        log(f"[summary] achievable: bf16 GEMM {a['gemm_bf16_8192_TFLOP_s']:.0f} TF, copy "
            f"{a['copy_1GiB_GB_s']:.0f} GB/s")


if __name__ == "__main__":
    main()
