"""GPU tier: the allocation-free decode entry point (pkv_decode_attention_noalloc) against the
decode entry point that takes a caller-owned workspace, through the C ABI.

The no-alloc call runs the same kernels with the library's fixed per-GPU scratch array as
workspace, so its outputs must be bit-identical to pkv_decode_attention's; both are also held
to the oracle's bar. Two calls in a row, the second smaller, check that what the first call
left in the shared array does not leak into the second."""
import numpy as np
import pytest

import oracle
import workloads as W
from tests.gpu_util import DevBatch, bf16_to_f64, compare, dev_pools, i32, say, scale_for, to_host_bits
from tests.test_gpu_prefill import LSE_MAX, LSE_MEAN

pytestmark = pytest.mark.gpu


def _case(n_seqs, lo, hi, seed):
    spec = W.WorkloadSpec(f"noalloc_{n_seqs}_{hi}", seed, 32, 8, 128,
                          (W.BatchSpec("decode", n_seqs, W.Dist.uniform(lo, hi),
                                       W.Dist.const(1)),), ("scale", 1.25))
    return W.make_case(spec)


def _run(lib, case, noalloc):
    import torch
    b = case.batches[0]
    pk, pv = dev_pools(case)
    db = DevBatch(b)
    seq_lens = b.prefix_lens + 1
    max_len = int(seq_lens.max())
    out = torch.empty((b.n_seqs, case.hq, case.d), dtype=torch.bfloat16, device="cuda")
    lse = torch.empty((b.n_seqs, case.hq), dtype=torch.float32, device="cuda")
    lib.pkv_kv_append(pk, pv, db.k_new, db.v_new, db.tables, db.cached, db.cu, 1)
    if noalloc:
        lib.pkv_decode_attention_noalloc(pk, pv, db.q, db.tables, i32(seq_lens), max_len,
                                         scale_for(case.d), out, lse=lse)
    else:
        ws = lib.alloc_workspace(lib.pkv_decode_workspace_bytes(b.n_seqs, case.hq, case.hkv,
                                                                case.d, max_len))
        lib.pkv_decode_attention(pk, pv, db.q, db.tables, i32(seq_lens), max_len,
                                 scale_for(case.d), out, lse=lse, workspace=ws)
    torch.cuda.synchronize()
    return to_host_bits(out), lse.cpu().numpy()


def test_noalloc_decode_matches_workspace_decode_twice(gpu_lib):
    """Call 1: 64 sequences of up to 3,000 keys (several splits per sequence, so the scratch
    holds the order and the partial results). Call 2: 16 shorter sequences."""
    lib = gpu_lib
    for k, (n, lo, hi) in enumerate([(64, 1500, 3000), (16, 100, 900)]):
        case = _case(n, lo, hi, 170 + k)
        b = case.batches[0]
        need = lib.pkv_decode_workspace_bytes(n, case.hq, case.hkv, case.d,
                                              int(b.prefix_lens.max()) + 1)
        say(f"[noalloc] call {k + 1}: {n} sequences, contexts U[{lo},{hi}], workspace {need} B")
        assert 0 < need <= lib.PKV_DECODE_NOALLOC_MAX_BYTES
        got = _run(lib, case, noalloc=True)
        ref = _run(lib, case, noalloc=False)
        assert np.array_equal(got[0], ref[0]), "output differs from pkv_decode_attention"
        assert np.array_equal(got[1].view(np.uint32), ref[1].view(np.uint32)), "lse differs"
        o, l = oracle.decode_attention(case.pool_k, case.pool_v, b.block_tables, b.prefix_lens,
                                       b.q, b.k_new, b.v_new, scale_for(case.d), case.bs)
        compare(f"noalloc call {k + 1} vs oracle", bf16_to_f64(got[0]), o)
        compare(f"noalloc call {k + 1} lse vs oracle", got[1].astype(np.float64), l,
                atol_max=LSE_MAX, atol_mean=LSE_MEAN)
