"""Byte-exact paged KV append and gather (oracle; test infrastructure only).

The KV cache is a pool of fixed-size blocks addressed through a per-sequence block table,
like virtual-memory pages ("vLLM memory model", Section 2.1). Logical token t of a sequence
lives in physical block table[t // block_size], slot t % block_size.

Pool layout (the library's documented layout):
  K: [num_blocks][num_kv_heads][head_dim / 8][block_size][8]  -- dim d of slot s is at
     [.., d // 8, s, d % 8]
  V: [num_blocks][num_kv_heads][head_dim][block_size]         -- dim d of slot s is at [.., d, s]
Arrays are uint16 bf16 bit patterns; nothing here does arithmetic on the values.
"""
import numpy as np


def _k_slot(pool_k, blk, slot):
    """K row [num_kv_heads][head_dim] of one slot."""
    h, c, _, e = pool_k.shape[1], pool_k.shape[2], pool_k.shape[3], pool_k.shape[4]
    return pool_k[blk, :, :, slot, :].reshape(h, c * e)


def gather_seq(pool_k, pool_v, table_row, n_tokens, block_size):
    """Logical tokens 0..n_tokens-1 of one sequence -> (K, V), each [n][Hkv][D] uint16."""
    hkv = pool_k.shape[1]
    d = pool_k.shape[2] * pool_k.shape[4]
    k = np.empty((n_tokens, hkv, d), dtype=np.uint16)
    v = np.empty((n_tokens, hkv, d), dtype=np.uint16)
    for t in range(n_tokens):
        blk = int(table_row[t // block_size])
        slot = t % block_size
        if blk < 0:
            raise IndexError(f"token {t} maps to an unassigned table entry")
        k[t] = _k_slot(pool_k, blk, slot)
        v[t] = pool_v[blk, :, :, slot]
    return k, v


def gather_kv(pool_k, pool_v, block_tables, lens, block_size):
    """All sequences' first lens[i] tokens, concatenated in sequence order:
    (K, V), each [sum(lens)][Hkv][D] uint16."""
    ks, vs = [], []
    for i in range(len(lens)):
        k, v = gather_seq(pool_k, pool_v, block_tables[i], int(lens[i]), block_size)
        ks.append(k)
        vs.append(v)
    hkv = pool_k.shape[1]
    d = pool_k.shape[2] * pool_k.shape[4]
    if not ks:
        return np.empty((0, hkv, d), np.uint16), np.empty((0, hkv, d), np.uint16)
    return np.concatenate(ks), np.concatenate(vs)


def kv_append(pool_k, pool_v, block_tables, cached_lens, cu_new_lens, k_new, v_new,
              block_size):
    """Return copies of the pools with each sequence's new tokens written after its cached
    prefix: new token j of sequence i goes to logical position cached_lens[i] + j.
    k_new, v_new: [T][Hkv][D] uint16, rows cu_new_lens[i] .. cu_new_lens[i+1]-1 belong to i."""
    pk = np.array(pool_k, copy=True)
    pv = np.array(pool_v, copy=True)
    hkv, nchunk, _, e = pk.shape[1], pk.shape[2], pk.shape[3], pk.shape[4]
    for i in range(len(cached_lens)):
        p = int(cached_lens[i])
        a, b = int(cu_new_lens[i]), int(cu_new_lens[i + 1])
        for j in range(b - a):
            t = p + j
            blk = int(block_tables[i][t // block_size])
            slot = t % block_size
            if blk < 0:
                raise IndexError(f"sequence {i} token {t} maps to an unassigned table entry")
            pk[blk, :, :, slot, :] = np.asarray(k_new[a + j]).reshape(hkv, nchunk, e)
            pv[blk, :, :, slot] = v_new[a + j]
    return pk, pv


def copy_blocks(pool_k, pool_v, pairs):
    """Copy-on-write's device half: return copies of the pools in which block `dst` holds
    block `src`'s K and V (every kv head, every slot) for each (src, dst) in pairs. Sources are
    read from the pools as given (no pair sees another's copy). A pair naming a block outside
    the pool is skipped, as the library documents."""
    pk = np.array(pool_k, copy=True)
    pv = np.array(pool_v, copy=True)
    nb = pk.shape[0]
    for src, dst in pairs:
        src, dst = int(src), int(dst)
        if not (0 <= src < nb and 0 <= dst < nb):
            continue
        pk[dst] = pool_k[src]
        pv[dst] = pool_v[src]
    return pk, pv
