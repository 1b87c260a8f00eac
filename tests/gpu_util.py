"""Helpers of the GPU tests: move a generated case to the device, run the library through
its C ABI, and compare against the oracle (test infrastructure)."""
import math
import sys

import numpy as np

ATOL_MAX = 2e-2   # max-abs bound for bf16-in / fp32-accumulate attention outputs
ATOL_MEAN = 2e-3  # mean-abs bound


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def to_dev_bits(arr, device="cuda"):
    """numpy uint16 bf16 bits -> torch bf16 device tensor (same bits)."""
    import torch
    return torch.from_numpy(np.ascontiguousarray(arr).view(np.int16)).to(device).view(torch.bfloat16)


def to_host_bits(t):
    import torch
    return t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def bf16_to_f64(bits):
    return (np.asarray(bits, np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def i32(arr, device="cuda"):
    import torch
    return torch.from_numpy(np.ascontiguousarray(arr, dtype=np.int32)).to(device)


class DevBatch:
    """Device copies of one generated batch plus its host maxima."""

    def __init__(self, batch, device="cuda"):
        import torch
        self.host = batch
        self.tables = i32(batch.block_tables, device)
        self.cached = i32(batch.prefix_lens, device)
        self.cu = i32(batch.cu_new_lens, device)
        self.seq_lens = i32(batch.prefix_lens + batch.new_lens, device)
        self.max_new = int(batch.new_lens.max()) if batch.n_seqs else 0
        self.max_total = int((batch.prefix_lens + batch.new_lens).max()) if batch.n_seqs else 0

        def dev(x):
            if x is None:
                return None
            if isinstance(x, torch.Tensor):
                return x
            return to_dev_bits(x, device)

        self.q = dev(batch.q)
        self.k_new = dev(batch.k_new)
        self.v_new = dev(batch.v_new)


def dev_pools(case, device="cuda"):
    import torch
    if isinstance(case.pool_k, torch.Tensor):
        return case.pool_k, case.pool_v
    return to_dev_bits(case.pool_k, device), to_dev_bits(case.pool_v, device)


def compare(name, got_f64, ref_f64, atol_max=ATOL_MAX, atol_mean=ATOL_MEAN):
    err = np.abs(got_f64 - ref_f64)
    assert np.all(np.isfinite(got_f64)), f"{name}: non-finite output"
    mx, mean = float(err.max()) if err.size else 0.0, float(err.mean()) if err.size else 0.0
    say(f"  {name}: max-abs {mx:.3e}  mean-abs {mean:.3e}  over {err.size} values")
    assert mx <= atol_max, f"{name}: max-abs {mx} > {atol_max}"
    assert mean <= atol_mean, f"{name}: mean-abs {mean} > {atol_mean}"
    return mx, mean


def sub_pool_for(pool_k, pool_v, table_row, n_tokens, bs=16):
    """Host copy of just the blocks one sequence uses (torch device pools), with the table row
    remapped to them; the oracle then gathers from this small pool."""
    import torch
    nblk = -(-n_tokens // bs)
    ids = torch.as_tensor(np.asarray(table_row[:nblk], dtype=np.int64), device=pool_k.device)
    pk = to_host_bits(pool_k.index_select(0, ids))
    pv = to_host_bits(pool_v.index_select(0, ids))
    return pk, pv, np.arange(nblk, dtype=np.int32)


def scale_for(d):
    return 1.0 / math.sqrt(d)
