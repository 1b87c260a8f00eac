"""Softmax attention over a paged KV cache, in float64 (oracle; test infrastructure only).

Definitions followed:
  * Section 2.1 ("Background"): prefill processes all prompt tokens and materialises per-layer
    K/V; decode produces one token at a time, attending over all previously computed K/V.
  * Section 2.1 ("Prefix caching", "Prefix sharing in semantic operators"): the KV of a cached
    prompt prefix is reused and only the novel suffix is computed. So a downstream operator's
    prefill of N new tokens over a cached prefix of P tokens gives new token j (0-based) the
    keys 0 .. P + j: the whole cached prefix plus new tokens 0..j. These are exactly rows
    P .. P+N-1 of ordinary causal attention over the concatenated P + N tokens.
  * Scaled dot-product attention: score s_t = scale * <q, k_t>, weights softmax over the
    visible keys, output sum_t w_t v_t; the log-sum-exp of the scaled scores (natural log) is
    returned alongside. Query head h reads kv head h // (Hq / Hkv) (grouped-query attention,
    consecutive groups).

The prefix K/V are read from the pool *before* the append, and the new tokens' K/V from the
input arrays, so attention results do not depend on the append's correctness.
"""
import numpy as np

from .bf16 import bf16_bits_to_f64
from .paged import gather_seq


def softmax_attention(q, k, v, visible, scale):
    """q [n][D], k [L][D], v [L][Dv] float64; visible[r] = number of leading keys row r sees.
    Returns (o [n][Dv], lse [n]). Every row must see at least one key."""
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    visible = np.asarray(visible)
    n, L = q.shape[0], k.shape[0]
    if n and visible.min() < 1:
        raise ValueError("a query row with no visible key")
    s = scale * (q @ k.T)                                   # [n][L]
    seen = np.arange(L)[None, :] < visible[:, None]
    s = np.where(seen, s, -np.inf)
    m = s.max(axis=1, keepdims=True)
    p = np.exp(s - m)                                       # exp(-inf) = 0 for hidden keys
    l = p.sum(axis=1, keepdims=True)
    o = (p / l) @ v
    lse = m[:, 0] + np.log(l[:, 0])
    return o, lse


def _check_heads(num_q_heads, num_kv_heads):
    if num_q_heads % num_kv_heads:
        raise ValueError("num_q_heads must be a multiple of num_kv_heads")
    return num_q_heads // num_kv_heads


def prefill_attention(pool_k, pool_v, block_tables, cached_lens, cu_new_lens, q, k_new, v_new,
                      scale, block_size):
    """Prefix-reuse prefill. q [T][Hq][D], k_new/v_new [T][Hkv][D] as bf16 bits (uint16);
    pools as bf16 bits in the library layout, holding each sequence's cached prefix.
    Returns (o [T][Hq][D] float64, lse [T][Hq] float64)."""
    q = np.asarray(q)
    t_total, hq, d = q.shape
    hkv = np.asarray(k_new).shape[1]
    g = _check_heads(hq, hkv)
    out = np.zeros((t_total, hq, d), dtype=np.float64)
    lse = np.zeros((t_total, hq), dtype=np.float64)
    for i in range(len(cached_lens)):
        p = int(cached_lens[i])
        a, b = int(cu_new_lens[i]), int(cu_new_lens[i + 1])
        n = b - a
        if n == 0:
            continue
        kc, vc = gather_seq(pool_k, pool_v, block_tables[i], p, block_size)
        keys = np.concatenate([bf16_bits_to_f64(kc), bf16_bits_to_f64(k_new[a:b])])
        vals = np.concatenate([bf16_bits_to_f64(vc), bf16_bits_to_f64(v_new[a:b])])
        visible = p + np.arange(n) + 1
        qi = bf16_bits_to_f64(q[a:b])
        for h in range(hq):
            o, l = softmax_attention(qi[:, h], keys[:, h // g], vals[:, h // g], visible, scale)
            out[a:b, h] = o
            lse[a:b, h] = l
    return out, lse


def decode_attention(pool_k, pool_v, block_tables, context_lens, q, k_new, v_new, scale,
                     block_size):
    """One decode step: sequence i has context_lens[i] cached tokens, appends one token
    (k_new[i], v_new[i]) and its query q[i] attends over all context_lens[i] + 1 keys.
    q [B][Hq][D], k_new/v_new [B][Hkv][D] bf16 bits. Returns (o [B][Hq][D], lse [B][Hq])."""
    bsz = len(context_lens)
    cu = np.arange(bsz + 1, dtype=np.int64)
    return prefill_attention(pool_k, pool_v, block_tables, context_lens, cu, q, k_new, v_new,
                             scale, block_size)
