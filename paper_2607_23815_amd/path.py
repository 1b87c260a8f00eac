"""The hot path as two calls on torch device tensors (every step runs in libpkv's kernels).

prefill_step: a downstream operator's suffix extends each tuple's cached prefix -- KV append
              of the new tokens, then prefix-reuse prefill attention over prefix + suffix.
decode_step:  one generated token per sequence -- KV append of its K/V at position C_i, then
              split-K decode attention over all C_i + 1 keys.
Both enqueue on `stream` (torch's current stream by default) and return without waiting."""
from . import lib


def prefill_step(k_cache, v_cache, q, k_new, v_new, block_tables, cached_lens, cu_new_lens,
                 max_new_len, max_total_len, scale, out, lse=None, workspace=None,
                 stream=None):
    lib.pkv_kv_append(k_cache, v_cache, k_new, v_new, block_tables, cached_lens, cu_new_lens,
                      max_new_len, stream=stream)
    lib.pkv_prefill_attention(k_cache, v_cache, q, block_tables, cached_lens, cu_new_lens,
                              max_new_len, max_total_len, scale, out, lse=lse,
                              workspace=workspace, stream=stream)


def decode_step(k_cache, v_cache, q, k_new, v_new, block_tables, context_lens, cu_one,
                seq_lens, max_seq_len, scale, out, lse=None, workspace=None, stream=None):
    """context_lens: int32 [B] cached tokens; cu_one: int32 [B+1] = 0..B (one new token per
    sequence); seq_lens: int32 [B] = context_lens + 1."""
    lib.pkv_kv_append(k_cache, v_cache, k_new, v_new, block_tables, context_lens, cu_one, 1,
                      stream=stream)
    lib.pkv_decode_attention(k_cache, v_cache, q, block_tables, seq_lens, max_seq_len, scale,
                             out, lse=lse, workspace=workspace, stream=stream)
