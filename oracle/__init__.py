"""CPU oracle for the paged prefix-reuse attention path -- TEST INFRASTRUCTURE ONLY.

Only tests/, __graft_entry__.smoke() and bench.py's CPU-baseline leg may import this package.
The library (paper_2607_23815_amd) never imports or calls it, and it imports nothing from the
library: the two share no code. Inputs come from the seeded generators in `workloads`.

What it computes, and the passage of the paper each part follows:
  * attention.py -- softmax attention in float64 over keys gathered into contiguous buffers.
    Prefill and decode over a KV cache are the two phases of Section 2.1 ("Background");
    reusing the cached KV of an identical prompt prefix and computing only the novel suffix is
    the "Prefix caching" paragraph of Section 2.1, and the filter -> map example of the
    "Prefix sharing in semantic operators" paragraph (prompt [S | C(t) | I_op], shared prefix
    [S | C(t)]) fixes that the downstream prefill attends over the cached prefix plus its own
    suffix. The attention formula itself is the standard scaled dot-product softmax attention
    the paper cites for autoregressive inference.
  * paged.py -- byte-exact KV append (scatter) into, and gather out of, a pool of fixed-size
    blocks addressed through per-sequence block tables ("vLLM memory model" paragraph of
    Section 2.1: a global pool of fixed-size blocks, analogous to virtual-memory pages).
  * block_pool.py -- a plain model of the block pool's bookkeeping: blocks allocated on
    admission and returned on completion, requests deferred (refused, state unchanged) when
    blocks run short (Section 2.1), pruned tuples free their memory (Section 4, predicate
    contract), a parent's memory released only once all its children are done (Section 5.3,
    Algorithm 1, the Complete procedure's release step).
  * sizes.py -- the KV-cache footprint closed form behind Section 2.2's "112 KB/token".

Every function here is pinned by `-m "not gpu"` tests in tests/test_oracle_pins.py and
tests/test_block_pool_model.py (library routines, closed forms, invariants, brute force).
"""
from .bf16 import bf16_bits_to_f64, bf16_bits_to_f32
from .paged import gather_seq, gather_kv, kv_append, copy_blocks
from .attention import softmax_attention, prefill_attention, decode_attention
from .block_pool import BlockPoolModel, Status
from .sizes import kv_bytes_per_token
