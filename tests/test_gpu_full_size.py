"""GPU tier at the workloads' full sizes, in the launch configuration bench.py times.

Inputs are generated on the device (seeded); the oracle recomputes a sample of sequences one
by one from host copies of their blocks taken before the step. Properties that hold at any
size are checked over the whole pool: the append changes exactly total_new * Hkv * D
elements of each cache (every other bit, NaN canaries included, is untouched)."""
import math

import numpy as np
import pytest

import oracle
import workloads as W
from tests.gpu_util import (bf16_to_f64, compare, i32, say, sub_pool_for, to_dev_bits,
                            to_host_bits)
from tests.test_gpu_prefill import LSE_MAX, LSE_MEAN

pytestmark = pytest.mark.gpu


def _samples(b, k):
    """First, last, longest, shortest and a few seeded random sequences."""
    tot = b.prefix_lens + b.new_lens
    idx = {0, b.n_seqs - 1, int(np.argmax(tot)), int(np.argmin(tot))}
    rng = np.random.default_rng(7)
    idx.update(rng.choice(b.n_seqs, size=min(k, b.n_seqs), replace=False).tolist())
    return sorted(idx)


def _snapshot(case, b, seqs):
    """Host copies of each sampled sequence's blocks (whole table row), table remapped."""
    out = {}
    for s in seqs:
        nt = int(b.prefix_lens[s] + b.new_lens[s])
        pk, pv, row = sub_pool_for(case.pool_k, case.pool_v, b.block_tables[s], nt)
        out[s] = (pk, pv, row)
    return out


def _changed(before, after):
    import torch
    return int((before.view(torch.int16) != after.view(torch.int16)).sum().item())


def _run_and_check(spec, n_prefill_samples=4, n_decode_samples=12):
    import torch
    from paper_2607_23815_amd import lib
    say(f"[full size] {spec.name}: generating on the device")
    case = W.plan_case(spec)
    W.fill_device(case, "cuda")
    d = case.d
    scale = 1.0 / math.sqrt(d)
    pk, pv = case.pool_k, case.pool_v
    k_before, v_before = pk.clone(), pv.clone()
    snaps, samples = [], []
    for b in case.batches:
        sel = _samples(b, n_prefill_samples if b.kind == "prefill" else n_decode_samples)
        samples.append(sel)
        snaps.append(_snapshot(case, b, sel))
    outs = []
    total_new = 0
    # the launch set: every batch's append, then prefill and decode attention
    dev = []
    for b in case.batches:
        dv = dict(tables=i32(b.block_tables), cached=i32(b.prefix_lens), cu=i32(b.cu_new_lens),
                  max_new=int(b.new_lens.max()), max_total=int((b.prefix_lens + b.new_lens).max()))
        dev.append(dv)
        lib.pkv_kv_append(pk, pv, b.k_new, b.v_new, dv["tables"], dv["cached"], dv["cu"],
                          dv["max_new"])
        total_new += b.total_new
    for b, dv in zip(case.batches, dev):
        if b.kind == "prefill":
            o = torch.empty((b.total_new, case.hq, d), dtype=torch.bfloat16, device="cuda")
            l = torch.empty((b.total_new, case.hq), dtype=torch.float32, device="cuda")
            lib.pkv_prefill_attention(pk, pv, b.q, dv["tables"], dv["cached"], dv["cu"],
                                      dv["max_new"], dv["max_total"], scale, o, lse=l)
        else:
            sl = b.prefix_lens + 1
            maxl = int(sl.max())
            o = torch.empty((b.n_seqs, case.hq, d), dtype=torch.bfloat16, device="cuda")
            l = torch.empty((b.n_seqs, case.hq), dtype=torch.float32, device="cuda")
            ws = lib.alloc_workspace(lib.pkv_decode_workspace_bytes(b.n_seqs, case.hq, case.hkv,
                                                                    d, maxl))
            lib.pkv_decode_attention(pk, pv, b.q, dv["tables"], i32(sl), maxl, scale, o,
                                     lse=l, workspace=ws)
        outs.append((o, l))
    torch.cuda.synchronize()

    # append: exactly the new slots changed, over the whole pool
    per_cache = total_new * case.hkv * d
    assert _changed(k_before, pk) == per_cache, "K cache: stray or missing writes"
    assert _changed(v_before, pv) == per_cache, "V cache: stray or missing writes"
    del k_before, v_before

    for b, sel, snap, (o, l) in zip(case.batches, samples, snaps, outs):
        q = b.q
        for s in sel:
            spk, spv, row = snap[s]
            p, n = int(b.prefix_lens[s]), int(b.new_lens[s])
            a, e = int(b.cu_new_lens[s]), int(b.cu_new_lens[s + 1])
            qh, kh, vh = to_host_bits(q[a:e]), to_host_bits(b.k_new[a:e]), to_host_bits(b.v_new[a:e])
            # append, bit-exact, on this sequence's blocks
            ek, ev = oracle.kv_append(spk, spv, row[None], [p], [0, n], kh, vh, case.bs)
            gk, gv, _ = sub_pool_for(pk, pv, b.block_tables[s], p + n)
            assert np.array_equal(gk, ek) and np.array_equal(gv, ev), f"append seq {s}"
            if b.kind == "prefill":
                ro, rl = oracle.prefill_attention(spk, spv, row[None], [p], [0, n], qh, kh, vh,
                                                  scale, case.bs)
            else:
                ro, rl = oracle.decode_attention(spk, spv, row[None], [p], qh, kh, vh, scale,
                                                 case.bs)
            rows = slice(a, e) if b.kind == "prefill" else slice(s, s + 1)
            compare(f"{spec.name} {b.kind} seq {s} (P={p}, N={n}) out",
                    bf16_to_f64(to_host_bits(o[rows])), ro)
            compare(f"{spec.name} {b.kind} seq {s} lse", l[rows].cpu().numpy().astype(np.float64),
                    rl, atol_max=LSE_MAX, atol_mean=LSE_MEAN)


@pytest.mark.parametrize("spec", [W.TINY, W.LLAMA3_8B_PREFILL, W.LLAMA3_8B_DECODE, W.MIXED_70B,
                                  W.LONG_DOC_SHARED_PROMPT], ids=lambda s: s.name)
def test_full_size_sampled_parity(gpu_lib, spec):
    _run_and_check(spec, n_prefill_samples=2 if spec is W.LONG_DOC_SHARED_PROMPT else 4)
