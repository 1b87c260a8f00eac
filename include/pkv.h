/*
 * pkv.h -- paged prefix-reuse attention for MI355X (gfx950): the C ABI.
 *
 * The library keeps a pool of fixed-size KV blocks addressed through per-sequence block
 * tables, appends new tokens' K/V into it, and runs attention over it for two phases:
 *   - a downstream operator's prefill, which reuses the KV cache a tuple's cached prompt
 *     prefix already holds and computes only the new suffix tokens, and
 *   - decode, one new token per sequence attending over the whole cached context.
 * This is the KV-cache reuse that pipelining semantic operators relies on: the filter -> map
 * example of Section 2.1 ("Prefix sharing in semantic operators") has prompts
 * [S | C(t) | I_filter] and [S | C(t) | I_map] whose shared prefix [S | C(t)] is cached once
 * and reused, so the map "only prefills the map-specific suffix". The block pool follows the
 * "vLLM memory model" paragraph of Section 2.1 (fixed-size blocks like virtual-memory pages,
 * taken on admission, returned on completion, requests deferred when blocks run out).
 *
 * Conventions
 *   - Every call returns pkv_status. On failure pkv_last_error() gives a message (thread-
 *     local, valid until this thread's next pkv call). Argument checks happen on the host
 *     before any launch; a failed call has launched nothing and changed no state.
 *   - Supported shapes: block_size 16; head_dim 64 or 128; num_q_heads a multiple of
 *     num_kv_heads; decode additionally needs num_q_heads / num_kv_heads <= 16. Anything else
 *     returns PKV_ERR_UNSUPPORTED_SHAPE. Zero sequences or zero tokens is a successful no-op.
 *   - Device calls take device pointers (caller-owned) and a hipStream_t passed as void*
 *     (NULL = the null stream). They never allocate or free device memory (the decode's
 *     workspace is the caller's, or the fixed scratch of pkv_decode_attention_noalloc); the
 *     one call that does is pkv_sched_run in device mode, which allocates its own metadata,
 *     output and workspace buffers for the run and frees them before returning. Device calls
 *     are asynchronous; results are ready when the stream has drained. A launch failure
 *     returns PKV_ERR_HIP with hipGetErrorString's text. Device calls are reentrant.
 *   - The contents of device metadata (block ids within the pool, lengths within the host
 *     maxima and the table, monotone token offsets) are the caller's contract: the host cannot
 *     check them without a device-to-host copy. The kernels only bound what they index (a
 *     table index by max_blocks; an id outside the pool reads a stand-in block; a length past
 *     the planned launch is cut), so bad metadata gives finite but wrong results, never an
 *     access outside the pool, the table or the workspace. Opt-in checking: with
 *     PKV_DEBUG_VALIDATE set in the environment (any value but "0"), or after
 *     pkv_set_debug_validate(1), every device call first runs a validation kernel over its
 *     metadata, waits for the stream, and returns PKV_ERR_BAD_METADATA (launching nothing
 *     else) naming what failed and the first offending sequence. This synchronises every
 *     call: a debugging aid, not for graph capture or timed runs.
 *   - Interface choices: the block pool is host bookkeeping only (it takes the order in which
 *     blocks are handed out, not device pointers or a seed; the caller allocates the K/V
 *     tensors); device calls take host maxima (max_new_len, max_total_len, max_seq_len,
 *     max_len) that size the launch without a device-to-host read; the pool layout below is
 *     chunk-major K and dim-major V rather than row-major slabs; the prefill's workspace is
 *     optional (it enables the key split of batches too small to fill the chip).
 *   - bf16 is IEEE binary16 "brain float" (1 sign, 8 exponent, 7 mantissa bits), stored as
 *     16-bit words.
 *
 * KV pool layout (one attention layer; caller-allocated, 256-byte aligned):
 *   K cache: bf16 [num_blocks][num_kv_heads][head_dim/8][block_size][8]
 *            dim d of the token in slot s is element [.., d/8, s, d%8]: a block's slab for one
 *            kv head is head_dim/8 runs of block_size 16-byte chunks.
 *   V cache: bf16 [num_blocks][num_kv_heads][head_dim][block_size]
 *            dim d of slot s is element [.., d, s]: the slab is stored dim-major.
 *   Logical token t of a sequence lives in block block_tables[seq][t / block_size], slot
 *   t % block_size. Both layouts let attention feed the matrix cores straight from 16-byte
 *   loads (K rows for the score product, V columns for the value product).
 */
#ifndef PKV_H
#define PKV_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  PKV_OK = 0,
  PKV_ERR_INVALID_ARG = 1,        /* null pointer, negative size, inconsistent sizes */
  PKV_ERR_OUT_OF_BLOCKS = 2,      /* reserve refused: too few free blocks; nothing changed */
  PKV_ERR_SHARED_BLOCK_WRITE = 3, /* reserve refused: the write range hits a shared block */
  PKV_ERR_UNSUPPORTED_SHAPE = 4,  /* block_size / head_dim / head ratio not supported */
  PKV_ERR_NOT_FOUND = 5,          /* unknown sequence id */
  PKV_ERR_HIP = 6,                /* a HIP runtime call or launch failed */
  PKV_ERR_KEY_EXISTS = 7,         /* prefix publish refused: the key is already cached */
  PKV_ERR_BAD_METADATA = 8        /* PKV_DEBUG_VALIDATE refused a call's device metadata */
} pkv_status;

/* Message of this thread's last failed call ("" if none). */
const char* pkv_last_error(void);

/* ABI version, bumped on any incompatible change. */
int32_t pkv_abi_version(void);

/* Turn the opt-in metadata validation on (non-zero) or off for the process (see Conventions);
 * overrides PKV_DEBUG_VALIDATE. pkv_get_debug_validate returns the current setting. */
pkv_status pkv_set_debug_validate(int32_t on);
int32_t pkv_get_debug_validate(void);

/* ---------------------------------------------------------------------------------------
 * Block pool: host-side bookkeeping of which physical blocks each sequence (tuple) holds.
 * Section 2.1 ("vLLM memory model"): a global pool of fixed-size blocks, taken when a
 * request is admitted and returned when it completes; when blocks run short the request is
 * deferred. Section 4 (predicate contract): a dropped tuple frees its prefix. Section 5.3
 * (Algorithm 1): a parent's memory is released only after all its children.
 * A pool is not thread-safe; distinct pools are independent. It owns no device memory.
 * --------------------------------------------------------------------------------------- */
typedef struct pkv_pool pkv_pool;

/* Create a pool of num_blocks blocks of block_size tokens. free_order (host, may be NULL):
 * the order in which blocks are handed out, a permutation of 0..num_blocks-1 (NULL means
 * ascending); a seeded permutation gives the random block placement of a fragmented pool.
 * The array is copied. *out receives the pool. */
pkv_status pkv_pool_create(int32_t num_blocks, int32_t block_size, const int32_t* free_order,
                           pkv_pool** out);
void pkv_pool_destroy(pkv_pool* pool);
int32_t pkv_pool_num_free(const pkv_pool* pool);  /* -1 for a NULL pool */

/* New empty sequence; ids start at 1 and are never reused within a pool. */
pkv_status pkv_seq_create(pkv_pool* pool, int64_t* seq_id);

/* New sequence sharing the first shared_tokens tokens of parent (a multiple of block_size,
 * at most the parent's committed length) by reference: the shared blocks' reference counts
 * go up, and they return to the free list only when every holder has been freed. */
pkv_status pkv_seq_fork(pkv_pool* pool, int64_t parent, int32_t shared_tokens, int64_t* child);

/* Reserve room for new_tokens more tokens after the sequence's committed and already
 * reserved tokens. When too few blocks are free, unpinned cached prefixes are evicted
 * first (see the prefix cache below). All-or-nothing: OUT_OF_BLOCKS when even eviction
 * cannot free enough blocks and SHARED_BLOCK_WRITE when the range would write into a block
 * held by another sequence or a cached prefix; in both cases nothing changes (no eviction
 * either). Blocks come from the front of the free list, in order. */
pkv_status pkv_seq_reserve(pkv_pool* pool, int64_t seq, int32_t new_tokens);

/* Mark new_tokens reserved tokens as written (after kv_append); 0 <= new_tokens <= reserved. */
pkv_status pkv_seq_commit(pkv_pool* pool, int64_t seq, int32_t new_tokens);

/* Drop a sequence: each of its blocks loses one reference; a block whose count reaches zero
 * goes to the back of the free list (in table order). */
pkv_status pkv_seq_free(pkv_pool* pool, int64_t seq);

/* Committed length of a sequence. */
pkv_status pkv_seq_len(const pkv_pool* pool, int64_t seq, int32_t* len);

/* ---------------------------------------------------------------------------------------
 * Prefix cache, eviction and pinning (the allocator side of Section 6).
 *
 * Section 2.1 (automatic prefix caching): the KV of an identical prefix is reused and only
 * the new suffix computed; the reuse is opportunistic because a finished request's blocks
 * can be reclaimed. A sequence publishes its first `tokens` committed tokens under a 64-bit
 * key chosen by the caller (e.g. a hash of the tuple's prompt tokens). The entry holds one
 * reference on each of the ceil(tokens / block_size) blocks, so they stay resident after the
 * sequence is freed; attach turns a hit into a new sequence that shares them.
 *
 * Eviction: when a reservation (pkv_seq_reserve / pkv_seq_reserve_cow) finds too few free
 * blocks, entries are dropped in policy order until enough are free, all-or-nothing like
 * the reservation itself. Policy (Section 2.2 weighs both): least recently used first
 * (default) or most recently used first, by a logical clock that each publish and each hit
 * advances. Dropping an entry releases its references only: a block returns to the back of
 * the free list when its last holder (sequence or entry) lets go, so a running sequence
 * keeps the blocks it shares.
 *
 * Pinning (Section 6): under explicit pinning (default) an entry whose pin count is positive
 * is never evicted until it is unpinned; under virtual pinning pins protect nothing and the
 * eviction order alone decides. Pin counts are kept in both modes. Deadlock check
 * (Section 6): requests waiting while none runs means the pipeline is stuck on pinned
 * memory; recovery unpins every entry and switches to virtual pinning.
 * --------------------------------------------------------------------------------------- */
enum { PKV_EVICT_LRU = 0, PKV_EVICT_MRU = 1 };
enum { PKV_PIN_EXPLICIT = 0, PKV_PIN_VIRTUAL = 1 };

pkv_status pkv_pool_set_eviction(pkv_pool* pool, int32_t policy); /* PKV_EVICT_* */
pkv_status pkv_pool_set_pinning(pkv_pool* pool, int32_t mode);    /* PKV_PIN_* */

/* Deadlock hook, to be polled with the serving engine's queue state: if waiting > 0 and
 * running == 0, every entry's pin count is set to zero and pinning becomes virtual
 * (*recovered = 1); otherwise nothing changes (*recovered = 0). The caller may switch back
 * to explicit pinning with pkv_pool_set_pinning once the pipeline drains. */
pkv_status pkv_pool_check_deadlock(pkv_pool* pool, int32_t waiting, int32_t running,
                                   int32_t* recovered);

/* Publish the first tokens (1 <= tokens <= committed length) of seq under key; KEY_EXISTS
 * if the key is cached already (nothing changes). The last block may be partly filled: the
 * publishing sequence then shares it, and writing further into it needs
 * pkv_seq_reserve_cow. */
pkv_status pkv_prefix_publish(pkv_pool* pool, int64_t seq, uint64_t key, int32_t tokens);

/* Look the key up. Hit: a new sequence (*seq) shares the entry's blocks, its committed
 * length is the entry's token count (*tokens), and the entry becomes most recently used.
 * Miss: NOT_FOUND, and nothing changes but the miss count. */
pkv_status pkv_prefix_attach(pkv_pool* pool, uint64_t key, int64_t* seq, int32_t* tokens);

/* Tokens cached under key (0 when absent). A pure query: no hit or miss is counted and the
 * entry's recency does not change (a scheduler sizes a task's reservation with it before
 * deciding to admit the task). */
pkv_status pkv_prefix_lookup(const pkv_pool* pool, uint64_t key, int32_t* tokens);

/* Pin counts of an entry (NOT_FOUND for an unknown key; unpin of an unpinned entry is
 * INVALID_ARG). */
pkv_status pkv_prefix_pin(pkv_pool* pool, uint64_t key);
pkv_status pkv_prefix_unpin(pkv_pool* pool, uint64_t key);

/* Drop an entry now, whatever its pins (the scheduler knows no task will reuse it). */
pkv_status pkv_prefix_release(pkv_pool* pool, uint64_t key);

/* Copy-on-write reservation: as pkv_seq_reserve, but each block of the write range that
 * another holder shares is replaced in the sequence's table by a fresh private block (taken
 * from the free list before the blocks the growth needs; eviction counts both). The pairs
 * (source block, copy) go to copies[2k], copies[2k+1] (host, room for max_copies pairs),
 * *num_copies receives their number; before appending, the caller copies those blocks'
 * contents on the device (pkv_copy_blocks). INVALID_ARG if more than max_copies copies are
 * needed; on any refusal nothing changes and *num_copies is 0. A block whose other holders
 * are all evicted by this very reservation is private by then and is not copied. */
pkv_status pkv_seq_reserve_cow(pkv_pool* pool, int64_t seq, int32_t new_tokens, int32_t* copies,
                               int32_t max_copies, int32_t* num_copies);

typedef struct {
  int32_t num_free;        /* blocks on the free list */
  int32_t num_entries;     /* cached prefixes */
  int32_t cached_blocks;   /* blocks held only by cached prefixes (evictable if unpinned) */
  int32_t pinned_entries;  /* entries with a positive pin count */
  int32_t eviction;        /* PKV_EVICT_* */
  int32_t pinning;         /* PKV_PIN_* */
  int64_t hits, misses;    /* attach outcomes */
  int64_t evictions;       /* entries dropped by reservations */
  int64_t cow_copies;      /* blocks copied on write */
} pkv_pool_stats;
pkv_status pkv_pool_get_stats(const pkv_pool* pool, pkv_pool_stats* out);

/* Export block tables: host_tables [n][max_blocks] receives each sequence's physical block
 * ids (reserved blocks included), padded with -1; host_lens [n] (may be NULL) receives the
 * committed lengths, i.e. the cached_lens of a following append/prefill. INVALID_ARG if a
 * sequence holds more than max_blocks blocks. Nothing is written on failure. */
pkv_status pkv_fill_block_tables(const pkv_pool* pool, const int64_t* seq_ids, int32_t n,
                                 int32_t max_blocks, int32_t* host_tables, int32_t* host_lens);

/* ---------------------------------------------------------------------------------------
 * Device calls.
 * --------------------------------------------------------------------------------------- */
typedef struct {
  void* k_cache;        /* bf16, layout above */
  void* v_cache;        /* bf16, layout above */
  int32_t num_blocks;
  int32_t block_size;   /* 16 */
  int32_t num_kv_heads;
  int32_t head_dim;     /* 64 or 128 */
} pkv_paged_kv;

/* KV append / scatter. Prefill materialises per-layer K/V for the prompt tokens and decode
 * adds one token at a time (Section 2.1, "Background"); a downstream operator extends the
 * tuple's cached prefix with its own suffix. For each sequence i < num_seqs and each new
 * token j < N_i = cu_new_lens[i+1] - cu_new_lens[i], row cu_new_lens[i] + j of k_new / v_new
 * (bf16 [total_new][num_kv_heads][head_dim], row-major) is copied bit-exactly into logical
 * position cached_lens[i] + j of sequence i. No other byte of the pool is modified (a
 * partially covered 16-byte V chunk is read and written back unchanged outside the new
 * slots). block_tables: int32 [num_seqs][max_blocks]; cached_lens: int32 [num_seqs];
 * cu_new_lens: int32 [num_seqs + 1], cu_new_lens[0] = 0, non-decreasing,
 * cu_new_lens[num_seqs] = total_new. max_new_len (host) >= every N_i sizes the grid. The
 * target blocks must be private to the sequence (the allocator guarantees this). */
pkv_status pkv_kv_append(const pkv_paged_kv* kv, const void* k_new, const void* v_new,
                         const int32_t* block_tables, int32_t max_blocks,
                         const int32_t* cached_lens, const int32_t* cu_new_lens,
                         int32_t num_seqs, int32_t total_new, int32_t max_new_len,
                         void* stream);

/* Prefix-reuse prefill attention. Section 2.1: the cached prefix's KV is reused and only the
 * suffix is computed. For sequence i with P_i = cached_lens[i] cached tokens and N_i new
 * tokens (already appended at positions P_i .. P_i + N_i - 1), new token j and query head h
 * attend over keys 0 .. P_i + j of kv head h / (num_q_heads / num_kv_heads):
 *   out[r][h] = sum_t softmax_t(scale * <q[r][h], K[t]>) V[t],   r = cu_new_lens[i] + j,
 * and lse[r][h] = ln sum_t exp(scale * <q[r][h], K[t]>). These are rows P_i.. of causal
 * attention over the whole P_i + N_i tokens. q, out: bf16 [total_new][num_q_heads][head_dim];
 * lse: float [total_new][num_q_heads] or NULL. bf16 inputs, fp32 accumulation, bf16 output
 * (round to nearest even). max_new_len (host) >= every N_i; max_total_len (host) >= every
 * P_i + N_i.
 * Key split (optional): a batch whose work items -- sequences x kv heads x tiles of 128
 * query columns, a column being one (new token, query head of the kv group) -- number
 * fewer than 2048 cannot keep the chip busy; when its keys are long (max_total_len >= 2048)
 * and the caller passes a workspace of at least pkv_prefill_workspace_bytes (16-byte
 * aligned, caller-owned, not read back), every item's keys are cut at multiples of a split
 * size (a multiple of 1024 keys chosen from the host arguments) into parts run as separate
 * work items; a row whose keys end in the first part is finished there, the others are
 * merged from their parts' partial results by log-sum-exp weights in a second kernel. The
 * cut points depend on key positions and host arguments only, so results are
 * deterministic. Order (optional, the same workspace): a batch of more than one sequence
 * whose keys reach 8192 (max_total_len >= 8192) takes its sequences longest first (a small
 * kernel writes the order into the workspace), so the launch does not end on a few long
 * items; the order moves work items, not arithmetic, so the results are bit-identical to
 * the unordered launch. With workspace NULL (or when the size is 0) the launch neither
 * splits nor orders; a non-NULL workspace smaller than the size is refused. Calls sharing a
 * workspace must not overlap. */
pkv_status pkv_prefill_attention(const pkv_paged_kv* kv, const void* q, int32_t num_q_heads,
                                 const int32_t* block_tables, int32_t max_blocks,
                                 const int32_t* cached_lens, const int32_t* cu_new_lens,
                                 int32_t num_seqs, int32_t total_new, int32_t max_new_len,
                                 int32_t max_total_len, float scale, void* out, float* lse,
                                 void* workspace, size_t workspace_bytes, void* stream);
/* Workspace that enables the prefill's plan: num_seqs int32 rounded up to 256 bytes when the
 * batch is ordered, plus total_new x num_q_heads x splits x (head_dim + 2) floats when it
 * splits; 0 when it does neither (or for arguments the call would refuse). */
size_t pkv_prefill_workspace_bytes(int32_t num_seqs, int32_t total_new, int32_t num_q_heads,
                                   int32_t num_kv_heads, int32_t head_dim,
                                   int32_t max_new_len, int32_t max_total_len);

/* Paged decode attention (Section 2.1: decode generates one token at a time, attending over
 * all previously computed K/V). Sequence i's single query q[i] attends over all
 * seq_lens[i] keys (the cached context plus the token this step appended):
 *   out[i][h] = sum_{t < seq_lens[i]} softmax_t(scale * <q[i][h], K[t]>) V[t].
 * The key range is cut into splits whose boundaries depend only on key positions; each split
 * writes a partial result to the workspace and a second kernel merges them with their
 * log-sum-exp weights. q, out: bf16 [num_seqs][num_q_heads][head_dim]; lse: float
 * [num_seqs][num_q_heads] or NULL; seq_lens: int32 [num_seqs], each >= 1. max_seq_len (host)
 * >= every seq_lens[i]. workspace: device memory of at least pkv_decode_workspace_bytes
 * (non-zero whenever num_seqs > 0: it also holds the order in which sequences are
 * scheduled, longest first), 16-byte aligned, owned by the caller, not read back; calls
 * that share a workspace must not overlap. */
pkv_status pkv_decode_attention(const pkv_paged_kv* kv, const void* q, int32_t num_q_heads,
                                const int32_t* block_tables, int32_t max_blocks,
                                const int32_t* seq_lens, int32_t num_seqs, int32_t max_seq_len,
                                float scale, void* out, float* lse, void* workspace,
                                size_t workspace_bytes, void* stream);
size_t pkv_decode_workspace_bytes(int32_t num_seqs, int32_t num_q_heads, int32_t num_kv_heads,
                                  int32_t head_dim, int32_t max_seq_len);

/* Allocation-free decode, for callers that cannot allocate device memory: code under HIP
 * graph capture, tight serving loops, harnesses that forbid hipMalloc. The same computation
 * as pkv_decode_attention (same kernels, bit-identical results) with the same arguments but
 * no workspace: the library uses a fixed device array of PKV_DECODE_NOALLOC_MAX_BYTES bytes per
 * GPU instead, loaded with the library's code object and held until the process ends. Calls
 * whose pkv_decode_workspace_bytes exceeds that size return PKV_ERR_INVALID_ARG before any
 * launch. The call itself allocates nothing (no hipMalloc, no library allocation); its first
 * call on a device looks the array's address up once. Every call on a GPU shares that GPU's
 * array, so calls that overlap on one GPU (different streams, or different host threads)
 * race and must be serialised by the caller. Nothing in the array needs to start at zero:
 * each call writes every word it later reads. */
#define PKV_DECODE_NOALLOC_MAX_BYTES (((size_t)32) << 20)
pkv_status pkv_decode_attention_noalloc(const pkv_paged_kv* kv, const void* q,
                                        int32_t num_q_heads, const int32_t* block_tables,
                                        int32_t max_blocks, const int32_t* seq_lens,
                                        int32_t num_seqs, int32_t max_seq_len, float scale,
                                        void* out, float* lse, void* stream);

/* Block copy (the device half of copy-on-write): for each k < num_pairs, the K and V of
 * every kv head in block pairs[2k] are copied bit-exactly into block pairs[2k+1]. pairs:
 * int32 device memory [num_pairs][2], e.g. the pairs pkv_seq_reserve_cow returned; every
 * copy must be distinct from every other block named in the call (the copies run
 * concurrently). A pair naming a block outside 0..num_blocks-1 is skipped. */
pkv_status pkv_copy_blocks(const pkv_paged_kv* kv, const int32_t* pairs, int32_t num_pairs,
                           void* stream);

/* Mixed prefill + decode (the mixed batch of a serving step: downstream operators
 * prefilling their suffixes while other tuples decode). Identical results, bit for bit, to
 * pkv_prefill_attention on the prefill arguments (q .. lse, as there, without a workspace:
 * the fused launch does not split keys) followed by pkv_decode_attention on the decode arguments (dq .. d_lse, with workspace and
 * workspace_bytes as there), with the same num_q_heads and scale; either batch may be empty
 * (zero sequences or zero new tokens). Both read the same pool, so the new tokens of both
 * batches must have been appended before the call. One fused kernel runs prefill workgroups
 * (matrix-core bound) and decode workgroups (HBM bound) side by side on every compute unit,
 * between the decode's ordering and merge kernels. The two batches' outputs must not
 * overlap. Errors are those of the two calls. */
pkv_status pkv_mixed_attention(const pkv_paged_kv* kv, int32_t num_q_heads, float scale,
                               const void* q, const int32_t* block_tables, int32_t max_blocks,
                               const int32_t* cached_lens, const int32_t* cu_new_lens,
                               int32_t num_seqs, int32_t total_new, int32_t max_new_len,
                               int32_t max_total_len, void* out, float* lse, const void* dq,
                               const int32_t* d_block_tables, int32_t d_max_blocks,
                               const int32_t* seq_lens, int32_t d_num_seqs,
                               int32_t max_seq_len, void* d_out, float* d_lse,
                               void* workspace, size_t workspace_bytes, void* stream);

/* Paged gather (test support): copies the first lens[i] tokens of every sequence out of the
 * pool into contiguous k_out / v_out, bf16 [sum lens][num_kv_heads][head_dim], sequence i
 * starting at row cu_lens[i] (int32 [num_seqs + 1]). Bit-exact. max_len (host) >= every
 * lens[i]. */
pkv_status pkv_gather_kv(const pkv_paged_kv* kv, const int32_t* block_tables,
                         int32_t max_blocks, const int32_t* lens, const int32_t* cu_lens,
                         int32_t num_seqs, int32_t max_len, void* k_out, void* v_out,
                         void* stream);

/* ---------------------------------------------------------------------------------------
 * Pipeline scheduler (Section 5, Algorithm 1; Section 6, memory management).
 *
 * A semantic query pipeline of num_stages stages: stage s runs one operator per task; a
 * surviving task of a non-final stage is joined (Cartesian product) with fanout[s] right-side
 * rows, creating dependent tasks that reuse its cached KV as their prefix; a final-stage task's
 * result is output; a task whose predicate drops its tuple ends its branch. Tasks of stage 0
 * are the num_tuples input tuples; task t of stage s+1 is row t % fanout[s] joined with task
 * t / fanout[s] of stage s. Per task (all stages concatenated in stage order, stage s holding
 * count_s = num_tuples * fanout[0] * ... * fanout[s-1] entries; fanout[num_stages-1] is
 * ignored): suffix (tokens the task appends to its parent's prefix), out_len (tokens its
 * request generates, 1..max_out) and filtered (non-zero: the predicate drops the tuple). These
 * are the inputs that fix every outcome, so a run is deterministic.
 *
 * The scheduler is the paper's adaptive memory-aware scheduler (Algorithm 1, Section 5.3)
 * restated as an engine loop. Each iteration: an admission pass lets every stage hand its
 * queued tasks, in order, to the engine while their KV reservations fit the stage's budget;
 * the engine advances the first max_batch admitted tasks by one step (a task's first step
 * prefills its prompt and yields one token, each later step appends the previous token's KV
 * and yields the next; with max_step_tokens, prompts are prefilled in chunks that fit the
 * step's token budget after the batch's decodes); finished tasks are handled (one that
 * reaches its token bound before its output is complete is interrupted, its bound doubled (at
 * most max_out) and queued again; a survivor of a non-final stage creates its children, which
 * reuse its cached prefix, and keeps its charge until all of them are done; results and
 * filtered tasks free their memory); and the budgets adapt: a middle stage with a high
 * backlog moves delta blocks to the last stage (from its own unused budget, else from the
 * first stage with delta unused), and, from the last stage back to the second, a stage with
 * a low backlog gives delta to the stage before it (high: waiting > alpha * budget /
 * minBudget; low: waiting < beta * budget / minBudget). Token bounds: static per stage, or the nearest-rank 99th percentile of
 * the output/input ratio of completed requests times the task's input length, once min_obs
 * requests have completed (initial_bound before that). Memory is counted in 16-token blocks of
 * a pool of num_blocks blocks that the run creates; completed prefixes are published in its
 * prefix cache and, under explicit pinning, pinned until their children are released.
 *
 * Policies: ADAPTIVE is Algorithm 1; DEPTH_FIRST keeps its initial budgets (minBudget for all
 * stages but the last, which takes the rest) and never rebalances; BREADTH_FIRST gives the
 * first stage breadth_share of the pool statically; SEQUENTIAL runs one task at a time, the
 * deepest ready stage first; BLOCKING runs each stage to completion before the next and leaves
 * prefixes to the cache's eviction order (the materialising execution of Section 2.2, ablated in
 * Section 7.4).
 * --------------------------------------------------------------------------------------- */
#define PKV_MAX_STAGES 8
enum { PKV_SCHED_ADAPTIVE = 0, PKV_SCHED_DEPTH_FIRST = 1, PKV_SCHED_BREADTH_FIRST = 2,
       PKV_SCHED_SEQUENTIAL = 3, PKV_SCHED_BLOCKING = 4 };
/* trace events: int32 quintuples (step, kind, stage, task, value) */
enum {
  PKV_EV_LAUNCH = 1,   /* value = 2 * charged blocks + 1 if the prefix is reused */
  PKV_EV_DONE = 2,     /* completed and passed on; value = output tokens */
  PKV_EV_FILTERED = 3, /* completed, dropped by its predicate; value = output tokens */
  PKV_EV_OUTPUT = 4,   /* final-stage result; value = output tokens */
  PKV_EV_RETRY = 5,    /* interrupted at its bound; value = the new bound */
  PKV_EV_RELEASE = 6,  /* memory charge released; value = blocks */
  PKV_EV_TRANSFER = 7  /* budget moved: stage = from, task = to, value = blocks */
};

typedef struct {
  int32_t policy;        /* PKV_SCHED_* */
  int32_t num_blocks;    /* KV blocks the pipeline may use */
  int32_t max_out;       /* largest output of any request; bounds never exceed it */
  int32_t delta;         /* budget transfer unit in blocks; 0 = the largest minBudget */
  double alpha, beta;    /* queue thresholds */
  double breadth_share;  /* BREADTH_FIRST: the first stage's share of num_blocks */
  int32_t pinning;       /* PKV_PIN_* */
  int32_t eviction;      /* PKV_EVICT_* */
  int32_t min_obs;       /* completed requests before the percentile estimate is used */
  int32_t max_batch;     /* tasks the engine advances per step */
  int64_t max_steps;     /* the run fails (INVALID_ARG) if it has not finished by then */
  int32_t max_step_tokens; /* > 0: chunked prefill, at most this many tokens per step (the
                              batch's decodes first, one each, then prompt chunks in queue
                              order); 0: whole prompts */
  int32_t static_bound[PKV_MAX_STAGES];   /* > 0: the stage's static token bound */
  int32_t initial_bound[PKV_MAX_STAGES];  /* > 0: bound before min_obs observations
                                             (0: max_out) */
} pkv_sched_config;

/* Device mode: each engine step also runs its attention work on the GPU through this
 * library's calls (block copies for copy-on-write, KV append, prefill attention for tasks in
 * their first step, decode attention for the others; a step with both sends its last prefill
 * group and its decode group out together as one pkv_mixed_attention launch), on `stream`,
 * timed with HIP events. The
 * step's K/V rows and queries are read from rows 0.. of the caller's synthetic sources
 * (bf16 [src_rows][num_kv_heads][head_dim] and [src_rows][num_q_heads][head_dim]; src_rows
 * >= max_batch and >= the longest prefix plus suffix of any task, checked before anything
 * runs). kv is a pool of at least num_blocks blocks; its contents
 * are overwritten. The run allocates its own metadata, output and workspace buffers and frees
 * them before returning. */
typedef struct {
  int64_t step;            /* engine step */
  int32_t phase;           /* 0: before the group's KV append (every earlier launch has completed
                              and the metadata is on the device); 1: after its attention */
  int32_t decode;          /* 1: a decode group (one new token each), 0: a prefill group */
  int32_t num_seqs;
  int32_t max_blocks;
  const int32_t* tables;   /* host [num_seqs][max_blocks]: the block tables the launches use */
  const int32_t* cached;   /* host [num_seqs]: tokens in the pool before the append */
  const int32_t* cu_new;   /* host [num_seqs + 1]: sequence k appends rows cu_new[k] .. of k_src /
                              v_src; a prefill group's queries are the same rows of q_src, a
                              decode group's query of sequence k is row k */
  const void* out;         /* device bf16 [rows][num_q_heads][head_dim]: the group's attention
                              output (prefill: row per new token; decode: row per sequence),
                              valid in phase 1 */
} pkv_sched_group;
/* Optional observer of device mode (tests, tracing): called on the calling thread twice per
 * group of sequences launched together, with the stream drained; it may read the pool and the
 * output but must not modify them. When a prefill group and a decode group go out in one
 * fused launch, both phase-0 calls (prefill first) come before both phase-1 calls, and each
 * group's output is at its own address. */
typedef void (*pkv_sched_group_hook)(void* user, const pkv_sched_group* group);

typedef struct {
  pkv_paged_kv kv;
  int32_t num_q_heads;
  const void* q_src;
  const void* k_src;
  const void* v_src;
  int32_t src_rows;
  void* stream;
  pkv_sched_group_hook group_hook;  /* NULL: none */
  void* hook_user;
} pkv_sched_device;

typedef struct {
  int64_t steps, launches, retries, hits, misses;
  int64_t prefill_tokens;  /* tokens prefilled (prompts, and recomputed prefixes on misses) */
  int64_t reused_tokens;   /* prefix tokens taken from the cache instead */
  int64_t decode_tokens;
  int64_t cow_copies, evictions, outputs;
  int64_t prefill_chunks;  /* prompt pieces prefilled (one per prompt without a budget) */
  int32_t max_batch;       /* largest batch the engine ran */
  double gpu_ms;           /* device mode: GPU time of the steps' launches (events around the
                              block copies, appends and attention; not the metadata uploads or
                              the host's work between launches); 0 otherwise */
  double wall_ms;          /* host wall time of the run */
} pkv_sched_stats;

/* Run the pipeline to completion (see above). num_tasks: the length of suffix, out_len and
 * filtered, which must equal the sum of count_s (INVALID_ARG otherwise). dev NULL: scheduling
 * only. trace (may be NULL
 * when max_events is 0): room for max_events events; *num_events receives the number of
 * events the run produced (those beyond max_events are counted, not written).
 * final_budgets (may be NULL): int64 [num_stages]. INVALID_ARG for a bad configuration, a
 * pool smaller than the stages' minimum budgets, or a run that cannot progress. */
pkv_status pkv_sched_run(const pkv_sched_config* cfg, int32_t num_stages, int32_t num_tuples,
                         const int32_t* fanout, int64_t num_tasks, const int32_t* suffix,
                         const int32_t* out_len, const uint8_t* filtered,
                         const pkv_sched_device* dev, int32_t* trace,
                         int64_t max_events, int64_t* num_events, int64_t* final_budgets,
                         pkv_sched_stats* stats);

#ifdef __cplusplus
}
#endif

#endif /* PKV_H */
