"""Seeded synthetic inputs for the paged prefix-reuse attention path.

Both the oracle tests and the GPU tests draw their inputs here, so this module deliberately
contains none of the path's arithmetic (no attention, no scatter, no gather): it draws
lengths, places blocks, and fills tensors with N(0,1) values rounded to bf16.

Pool layout (the library's documented layout, see include/pkv.h):
  K cache: bf16 [num_blocks][num_kv_heads][head_dim / 8][block_size][8]
           (for each block and kv head, 16-byte chunks of 8 dims, chunk-major, slot-minor)
  V cache: bf16 [num_blocks][num_kv_heads][head_dim][block_size]
           (for each block and kv head, the slab is stored dim-major: slot is fastest)
A slot that holds no cached token (tail slots of a sequence's last block, the slots the new
tokens will be appended into, and every slot of an unowned block) is filled with bf16 NaN
(0x7FC0), so any read of it that leaks into a result shows up as NaN.

Block placement: the pool's blocks are handed out in the order of a seeded permutation
`free_order`; the shared prompt (if any) takes the first blocks, then every sequence of every
batch takes ceil((prefix + new) / block_size) consecutive entries, in batch and sequence order.
This is exactly what the library's allocator does when it is created with the same free order
and sequences reserve their full length in that order.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import Any, List, Optional

import numpy as np

from .configs import WorkloadSpec, Dist

BF16_NAN = np.uint16(0x7FC0)


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bf16 (round to nearest, ties to even); returns uint16 bits.
    Inputs here are finite normal draws, so no NaN handling is needed."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    u = u + 0x7FFF + ((u >> 16) & 1)
    return (u >> 16).astype(np.uint16)


def _draw(dist: Dist, n: int, rng: np.random.Generator) -> np.ndarray:
    if dist.kind == "const":
        return np.full(n, dist.params[0], dtype=np.int64)
    if dist.kind == "uniform":
        lo, hi = dist.params
        return rng.integers(lo, hi + 1, size=n, dtype=np.int64)
    if dist.kind == "lognormal":
        median, sigma, lo, hi = dist.params
        z = rng.standard_normal(n)
        v = np.rint(np.exp(math.log(median) + sigma * z)).astype(np.int64)
        return np.clip(v, lo, hi)
    raise ValueError(f"unknown distribution {dist.kind}")


@dataclass
class BatchData:
    kind: str                 # "prefill" or "decode"
    prefix_lens: np.ndarray   # int32 [B]: tokens cached before this step (P_i, or C_i)
    new_lens: np.ndarray      # int32 [B]: tokens appended this step (N_i, 1 for decode)
    cu_new_lens: np.ndarray   # int32 [B+1]: exclusive prefix sum of new_lens
    block_tables: np.ndarray  # int32 [B][max_blocks], -1 padded
    q: Any = None             # bf16 [T][Hq][D]
    k_new: Any = None         # bf16 [T][Hkv][D]
    v_new: Any = None         # bf16 [T][Hkv][D]

    @property
    def n_seqs(self) -> int:
        return int(self.prefix_lens.shape[0])

    @property
    def total_new(self) -> int:
        return int(self.cu_new_lens[-1])

    @property
    def total_lens(self) -> np.ndarray:
        return (self.prefix_lens + self.new_lens).astype(np.int32)

    @property
    def max_blocks(self) -> int:
        return int(self.block_tables.shape[1])


@dataclass
class Case:
    spec: WorkloadSpec
    seed: int
    num_blocks: int
    free_order: np.ndarray    # int32 [num_blocks], the placement permutation
    shared_blocks: np.ndarray # int32 [n_shared], blocks of the shared prompt (may be empty)
    valid_slots: np.ndarray   # int32 [num_blocks], cached slots per block before the step
    batches: List[BatchData] = field(default_factory=list)
    pool_k: Any = None
    pool_v: Any = None

    @property
    def hq(self) -> int:
        return self.spec.num_q_heads

    @property
    def hkv(self) -> int:
        return self.spec.num_kv_heads

    @property
    def d(self) -> int:
        return self.spec.head_dim

    @property
    def bs(self) -> int:
        return self.spec.block_size

    def pool_shapes(self):
        nb, h, d, bs = self.num_blocks, self.hkv, self.d, self.bs
        return (nb, h, d // 8, bs, 8), (nb, h, d, bs)


def plan_case(spec: WorkloadSpec, seed: Optional[int] = None,
              prefix_override=None, new_override=None) -> Case:
    """Draw lengths and place blocks (metadata only; tensors are filled separately).

    prefix_override / new_override: optional list (one int array per batch) that replaces the
    drawn lengths, for structured tests (e.g. a zero-length prefix)."""
    seed = spec.seed if seed is None else int(seed)
    ss = np.random.SeedSequence(seed)
    len_ss, place_ss = ss.spawn(2)
    rng = np.random.default_rng(len_ss)
    bs = spec.block_size
    n_shared_tokens = spec.shared_prompt_tokens
    if n_shared_tokens % bs:
        raise ValueError("the shared prompt must be whole blocks")
    n_shared = n_shared_tokens // bs

    drawn = []
    for bi, b in enumerate(spec.batches):
        p = _draw(b.prefix, b.n_seqs, rng)
        n = _draw(b.new, b.n_seqs, rng)
        if prefix_override is not None and prefix_override[bi] is not None:
            p = np.asarray(prefix_override[bi], dtype=np.int64)
        if new_override is not None and new_override[bi] is not None:
            n = np.asarray(new_override[bi], dtype=np.int64)
        p = p + n_shared_tokens  # the shared prompt is part of every cached prefix
        drawn.append((p, n))

    private_needed = []
    for (p, n) in drawn:
        total = p + n
        private_needed.append(-(-total // bs) - n_shared)
    needed = n_shared + int(sum(int(x.sum()) for x in private_needed))

    kind, val = spec.pool[0], spec.pool[1]
    if kind == "min":
        num_blocks = max(int(val), needed)
    elif kind == "fixed":
        num_blocks = int(val)
        if num_blocks < needed:
            raise ValueError(f"{spec.name}: fixed pool of {num_blocks} < {needed} needed")
    elif kind == "scale":
        num_blocks = int(math.ceil(float(val) * needed))
    else:
        raise ValueError(kind)

    free_order = np.random.default_rng(place_ss).permutation(num_blocks).astype(np.int32)
    cursor = 0
    shared = free_order[cursor:cursor + n_shared].copy()
    cursor += n_shared
    valid = np.zeros(num_blocks, dtype=np.int32)
    valid[shared] = bs

    batches = []
    for (p, n), priv, bspec in zip(drawn, private_needed, spec.batches):
        nseq = p.shape[0]
        max_blocks = int((n_shared + priv).max()) if nseq else 0
        tables = np.full((nseq, max(max_blocks, 1)), -1, dtype=np.int32)
        for i in range(nseq):
            row = list(shared) + list(free_order[cursor:cursor + int(priv[i])])
            cursor += int(priv[i])
            tables[i, :len(row)] = row
            # cached slots before the step: the first p[i] tokens
            full, rem = divmod(int(p[i]), bs)
            for blk in range(n_shared, full):
                valid[row[blk]] = bs
            if rem:
                valid[row[full]] = rem
        cu = np.zeros(nseq + 1, dtype=np.int32)
        cu[1:] = np.cumsum(n)
        batches.append(BatchData(bspec.kind, p.astype(np.int32), n.astype(np.int32), cu, tables))
    return Case(spec, seed, num_blocks, free_order, shared.astype(np.int32), valid, batches)


def _tensor_seeds(case: Case):
    ss = np.random.SeedSequence([case.seed, 0xB16])
    kids = ss.spawn(2 + 3 * len(case.batches))
    return kids


def fill_host(case: Case) -> Case:
    """Fill every tensor on the host as numpy uint16 (bf16 bits)."""
    kids = _tensor_seeds(case)
    shp_k, shp_v = case.pool_shapes()
    bs = case.bs

    def normal_bf16(seed_seq, shape):
        r = np.random.default_rng(seed_seq)
        return f32_to_bf16_bits(r.standard_normal(shape, dtype=np.float32)).reshape(shape)

    pool_k = normal_bf16(kids[0], shp_k)
    pool_v = normal_bf16(kids[1], shp_v)
    stale = np.arange(bs)[None, :] >= case.valid_slots[:, None]  # [num_blocks][bs]
    pool_k.transpose(0, 3, 1, 2, 4)[stale] = BF16_NAN
    pool_v.transpose(0, 3, 1, 2)[stale] = BF16_NAN
    case.pool_k, case.pool_v = pool_k, pool_v
    for bi, b in enumerate(case.batches):
        t = b.total_new
        b.q = normal_bf16(kids[2 + 3 * bi], (t, case.hq, case.d))
        b.k_new = normal_bf16(kids[3 + 3 * bi], (t, case.hkv, case.d))
        b.v_new = normal_bf16(kids[4 + 3 * bi], (t, case.hkv, case.d))
    return case


def fill_device(case: Case, device="cuda") -> Case:
    """Fill every tensor directly in device memory with torch's seeded generator (for the
    full-size workloads, whose pools are several GB). Values differ from fill_host's for the
    same seed; within one case every consumer sees the same bits."""
    import torch

    g = torch.Generator(device=device)
    g.manual_seed(case.seed)
    shp_k, shp_v = case.pool_shapes()

    def normal_bf16(shape):
        out = torch.empty(shape, dtype=torch.bfloat16, device=device)
        flat = out.view(-1)
        step = 1 << 28
        for s in range(0, flat.numel(), step):
            e = min(flat.numel(), s + step)
            flat[s:e] = torch.randn(e - s, generator=g, device=device,
                                    dtype=torch.float32).to(torch.bfloat16)
        return out

    pool_k = normal_bf16(shp_k)
    pool_v = normal_bf16(shp_v)
    valid = torch.from_numpy(case.valid_slots).to(device)
    stale = torch.arange(case.bs, device=device)[None, :] >= valid[:, None]
    nan = float("nan")
    pool_k.masked_fill_(stale[:, None, None, :, None], nan)
    pool_v.masked_fill_(stale[:, None, None, :], nan)
    case.pool_k, case.pool_v = pool_k, pool_v
    for b in case.batches:
        t = b.total_new
        b.q = normal_bf16((t, case.hq, case.d))
        b.k_new = normal_bf16((t, case.hkv, case.d))
        b.v_new = normal_bf16((t, case.hkv, case.d))
    return case


def make_case(spec: WorkloadSpec, seed: Optional[int] = None, **overrides) -> Case:
    """Plan and fill a case on the host (small workloads)."""
    return fill_host(plan_case(spec, seed, **overrides))
