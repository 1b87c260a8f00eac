"""GPU tier: prefix reuse computes exactly the rows a full recompute would (Section 2.1: a
downstream operator reuses the cached prefix's KV and prefills only its suffix).

Recompute view: every sequence's L = P + N tokens are new (nothing cached); its outputs are
checked against the oracle. Reuse view of the same data: the first P tokens of each sequence
are appended first (the upstream operator's cache), then the last N tokens, and prefill runs
with P cached tokens and the last N queries. Its N output rows per sequence must match the
recompute's rows P .. L-1 within the attention bar (both are bf16-in / fp32-accumulate; the
query tiling and therefore the rounding order differ)."""
import numpy as np
import pytest

import oracle
import workloads as W
from tests.gpu_util import bf16_to_f64, compare, dev_pools, i32, say, scale_for, to_dev_bits, to_host_bits
from tests.test_gpu_prefill import LSE_MAX, LSE_MEAN

pytestmark = pytest.mark.gpu


def _rows(cu, lens_from, lens_to):
    """Row indices [cu[i] + lens_from[i], cu[i] + lens_to[i]) of every sequence, concatenated."""
    return np.concatenate([np.arange(cu[i] + a, cu[i] + b) for i, (a, b) in
                           enumerate(zip(lens_from, lens_to))]).astype(np.int64)


# (the shared-prompt workload has no recompute view: its prompt blocks are shared, so every
# sequence would append its own values into the same slots)
SPECS = [W.LLAMA3_8B_PREFILL.scaled(prefill=6), W.MIXED_70B.scaled(prefill=3, decode=0), W.TINY]


@pytest.mark.parametrize("sp", SPECS, ids=lambda s: s.name)
def test_reuse_rows_equal_recompute_rows(gpu_lib, sp):
    import torch
    lib = gpu_lib
    say(f"[reuse] {sp.name}")
    b0 = W.plan_case(sp).batches[0]
    P, N = b0.prefix_lens.astype(np.int64), b0.new_lens.astype(np.int64)
    L = P + N
    # the recompute view: nothing cached, L new tokens per sequence, fresh data
    rest = [None] * (len(sp.batches) - 1)
    case = W.make_case(sp, prefix_override=[np.zeros_like(L)] + rest, new_override=[L] + rest)
    b = case.batches[0]
    cu_r = b.cu_new_lens.astype(np.int64)
    scale = scale_for(case.d)
    # shared-prompt blocks would be written by both views; the reuse view rewrites identical
    # values, so the pools stay interchangeable
    pk, pv = dev_pools(case)
    pk2, pv2 = pk.clone(), pv.clone()
    tables = i32(b.block_tables)
    maxl = int(L.max())

    # recompute: append L, prefill over L new tokens
    q_all, k_all, v_all = to_dev_bits(b.q), to_dev_bits(b.k_new), to_dev_bits(b.v_new)
    out_r = torch.empty((int(L.sum()), case.hq, case.d), dtype=torch.bfloat16, device="cuda")
    lse_r = torch.empty((int(L.sum()), case.hq), dtype=torch.float32, device="cuda")
    zeros = i32(np.zeros(len(L)))
    lib.pkv_kv_append(pk, pv, k_all, v_all, tables, zeros, i32(cu_r), maxl)
    lib.pkv_prefill_attention(pk, pv, q_all, tables, zeros, i32(cu_r), maxl, maxl, scale, out_r,
                              lse=lse_r)

    # reuse: the prefix first (upstream operator), then the suffix, prefill with P cached
    pre = torch.from_numpy(_rows(cu_r, np.zeros_like(P), P)).cuda()
    suf = torch.from_numpy(_rows(cu_r, P, L)).cuda()
    cu_p = np.concatenate([[0], np.cumsum(P)]).astype(np.int32)
    cu_n = np.concatenate([[0], np.cumsum(N)]).astype(np.int32)
    if int(P.max()) > 0:
        lib.pkv_kv_append(pk2, pv2, k_all[pre].contiguous(), v_all[pre].contiguous(), tables,
                          zeros, i32(cu_p), int(P.max()))
    out_u = torch.empty((int(N.sum()), case.hq, case.d), dtype=torch.bfloat16, device="cuda")
    lse_u = torch.empty((int(N.sum()), case.hq), dtype=torch.float32, device="cuda")
    lib.pkv_kv_append(pk2, pv2, k_all[suf].contiguous(), v_all[suf].contiguous(), tables,
                      i32(P), i32(cu_n), int(N.max()))
    lib.pkv_prefill_attention(pk2, pv2, q_all[suf].contiguous(), tables, i32(P), i32(cu_n),
                              int(N.max()), maxl, scale, out_u, lse=lse_u)
    torch.cuda.synchronize()

    # both views end with the same pool contents over every sequence's L tokens
    assert torch.equal(pk.view(torch.int16), pk2.view(torch.int16))
    assert torch.equal(pv.view(torch.int16), pv2.view(torch.int16))
    # recompute against the oracle
    ro, rl = oracle.prefill_attention(case.pool_k, case.pool_v, b.block_tables, b.prefix_lens,
                                      b.cu_new_lens, b.q, b.k_new, b.v_new, scale, case.bs)
    compare(f"{sp.name} recompute out", bf16_to_f64(to_host_bits(out_r)), ro)
    compare(f"{sp.name} recompute lse", lse_r.cpu().numpy().astype(np.float64), rl,
            atol_max=LSE_MAX, atol_mean=LSE_MEAN)
    # reuse rows against the recompute's rows P..L-1
    sufh = _rows(cu_r, P, L)
    compare(f"{sp.name} reuse vs recompute out", bf16_to_f64(to_host_bits(out_u)),
            bf16_to_f64(to_host_bits(out_r))[sufh])
    compare(f"{sp.name} reuse vs recompute lse", lse_u.cpu().numpy().astype(np.float64),
            lse_r.cpu().numpy().astype(np.float64)[sufh], atol_max=LSE_MAX, atol_mean=LSE_MEAN)
