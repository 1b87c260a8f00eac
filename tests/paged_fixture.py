"""Test-side brute-force construction of paged pools from contiguous K/V.

Written element by element from the layout's definition, independently of oracle/paged.py,
so that pins comparing oracle results on a pool against a library routine on the contiguous
tensors check the oracle's gather as well as its arithmetic."""
import numpy as np

NAN_BITS = 0x7FC0


def empty_pools(num_blocks, hkv, d, bs):
    pk = np.full((num_blocks, hkv, d // 8, bs, 8), NAN_BITS, dtype=np.uint16)
    pv = np.full((num_blocks, hkv, d, bs), NAN_BITS, dtype=np.uint16)
    return pk, pv


def place(pk, pv, table_row, k_bits, v_bits, bs):
    """Write logical tokens 0..len(k_bits)-1 of one sequence into the pools, one element at a
    time: dim d of token t, kv head h goes to block table_row[t // bs], slot t % bs."""
    n, hkv, d = k_bits.shape
    for t in range(n):
        blk = table_row[t // bs]
        slot = t % bs
        for h in range(hkv):
            for dim in range(d):
                pk[blk, h, dim // 8, slot, dim % 8] = k_bits[t, h, dim]
                pv[blk, h, dim, slot] = v_bits[t, h, dim]


def rand_bf16(rng, shape):
    x = rng.standard_normal(shape).astype(np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    u = u + 0x7FFF + ((u >> 16) & 1)
    return (u >> 16).astype(np.uint16)


def widen(bits):
    return (np.asarray(bits, np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)
