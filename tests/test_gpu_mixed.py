"""GPU tier for the mixed prefill + decode launch (pkv_mixed_attention): its outputs and
log-sum-exps equal, bit for bit, a prefill call followed by a decode call on the same pool,
and meet the attention bar against the oracle; empty halves fall back to the single calls;
the full-size 70B-shaped mixed layer is checked bit for bit against the separate calls."""
import numpy as np
import pytest

import oracle
import workloads as W
from tests.gpu_util import (DevBatch, bf16_to_f64, compare, dev_pools, i32, say, scale_for,
                            to_host_bits)
from tests.test_gpu_prefill import LSE_MAX, LSE_MEAN

pytestmark = pytest.mark.gpu


def _run(lib, case, mixed, pools=None, drop=None):
    """Append both batches, then attention by one mixed call or by the two separate calls.
    drop: "prefill" / "decode" empties that half (zero sequences)."""
    import torch
    (bp, bd) = case.batches
    pk, pv = pools if pools is not None else dev_pools(case)
    dp, dd = DevBatch(bp), DevBatch(bd)
    scale = scale_for(case.d)
    lib.pkv_kv_append(pk, pv, dp.k_new, dp.v_new, dp.tables, dp.cached, dp.cu, dp.max_new)
    lib.pkv_kv_append(pk, pv, dd.k_new, dd.v_new, dd.tables, dd.cached, dd.cu, 1)
    nd = bd.n_seqs
    seq_lens = bd.prefix_lens + 1
    maxl = int(seq_lens.max())
    op = torch.full((bp.total_new, case.hq, case.d), float("nan"), dtype=torch.bfloat16,
                    device="cuda")
    lp = torch.full((bp.total_new, case.hq), float("nan"), dtype=torch.float32, device="cuda")
    od = torch.full((nd, case.hq, case.d), float("nan"), dtype=torch.bfloat16, device="cuda")
    ld = torch.full((nd, case.hq), float("nan"), dtype=torch.float32, device="cuda")
    ws = lib.alloc_workspace(lib.pkv_decode_workspace_bytes(nd, case.hq, case.hkv, case.d, maxl))
    sl = i32(seq_lens)
    p_cached, p_cu = dp.cached, dp.cu
    d_sl = sl
    if drop == "prefill":
        p_cached, p_cu = dp.cached[:0], i32(np.zeros(1))
    if drop == "decode":
        d_sl = sl[:0]
    if mixed:
        lib.pkv_mixed_attention(pk, pv, scale, dp.q, dp.tables, p_cached, p_cu, dp.max_new,
                                dp.max_total, op, dd.q, dd.tables, d_sl, maxl, od, lse=lp,
                                d_lse=ld, workspace=ws)
    else:
        if drop != "prefill":
            lib.pkv_prefill_attention(pk, pv, dp.q, dp.tables, dp.cached, dp.cu, dp.max_new,
                                      dp.max_total, scale, op, lse=lp)
        if drop != "decode":
            lib.pkv_decode_attention(pk, pv, dd.q, dd.tables, sl, maxl, scale, od, lse=ld,
                                     workspace=ws)
    torch.cuda.synchronize()
    return [to_host_bits(op), lp.cpu().numpy(), to_host_bits(od), ld.cpu().numpy()]


def _same(a, b):
    return all(np.array_equal(x.view(np.uint32) if x.dtype == np.float32 else x,
                              y.view(np.uint32) if y.dtype == np.float32 else y)
               for x, y in zip(a, b))


SPECS = [W.MIXED_70B.scaled(prefill=4, decode=24),
         W.WorkloadSpec("mixed_small_d64", 230, 8, 2, 64,
                        (W.BatchSpec("prefill", 5, W.Dist.uniform(0, 300), W.Dist.uniform(1, 90)),
                         W.BatchSpec("decode", 37, W.Dist.uniform(0, 3000), W.Dist.const(1))),
                        ("scale", 1.25)),
         W.WorkloadSpec("mixed_short_contexts", 231, 32, 8, 128,
                        (W.BatchSpec("prefill", 3, W.Dist.uniform(16, 64), W.Dist.uniform(1, 300)),
                         W.BatchSpec("decode", 300, W.Dist.uniform(0, 40), W.Dist.const(1))),
                        ("scale", 1.25))]


@pytest.mark.parametrize("spec", SPECS, ids=lambda s: s.name)
def test_mixed_equals_separate_calls_and_the_oracle(gpu_lib, spec):
    say(f"[mixed] {spec.name}")
    case = W.make_case(spec)
    pk, pv = dev_pools(case)
    sep = _run(gpu_lib, case, False, pools=(pk.clone(), pv.clone()))
    mix = _run(gpu_lib, case, True, pools=(pk, pv))
    assert _same(sep, mix), "mixed launch differs from the separate calls"
    bp, bd = case.batches
    scale = scale_for(case.d)
    ro, rl = oracle.prefill_attention(case.pool_k, case.pool_v, bp.block_tables, bp.prefix_lens,
                                      bp.cu_new_lens, bp.q, bp.k_new, bp.v_new, scale, case.bs)
    compare(f"{spec.name} prefill out", bf16_to_f64(mix[0]), ro)
    compare(f"{spec.name} prefill lse", mix[1].astype(np.float64), rl, atol_max=LSE_MAX,
            atol_mean=LSE_MEAN)
    do, dl = oracle.decode_attention(case.pool_k, case.pool_v, bd.block_tables, bd.prefix_lens,
                                     bd.q, bd.k_new, bd.v_new, scale, case.bs)
    compare(f"{spec.name} decode out", bf16_to_f64(mix[2]), do)
    compare(f"{spec.name} decode lse", mix[3].astype(np.float64), dl, atol_max=LSE_MAX,
            atol_mean=LSE_MEAN)


@pytest.mark.parametrize("drop", ["prefill", "decode"])
def test_mixed_with_an_empty_half(gpu_lib, drop):
    say(f"[mixed] empty {drop}")
    case = W.make_case(SPECS[0])
    pk, pv = dev_pools(case)
    sep = _run(gpu_lib, case, False, pools=(pk.clone(), pv.clone()), drop=drop)
    mix = _run(gpu_lib, case, True, pools=(pk, pv), drop=drop)
    assert _same(sep, mix)
    keep = [2, 3] if drop == "prefill" else [0, 1]
    for k in keep:  # the computed half is finite
        assert np.isfinite(bf16_to_f64(mix[k]) if mix[k].dtype == np.uint16 else mix[k]).all()


def test_mixed_full_size_equals_separate_calls(gpu_lib):
    """The 70B-shaped mixed layer at full size (128 prefill tuples, 384 decoding tuples)."""
    say("[mixed] full size: generating on the device")
    case = W.plan_case(W.MIXED_70B)
    W.fill_device(case, "cuda")
    pk, pv = case.pool_k, case.pool_v
    sep = _run(gpu_lib, case, False, pools=(pk.clone(), pv.clone()))
    mix = _run(gpu_lib, case, True, pools=(pk, pv))
    assert _same(sep, mix)
    assert np.isfinite(bf16_to_f64(mix[0])).all() and np.isfinite(bf16_to_f64(mix[2])).all()
