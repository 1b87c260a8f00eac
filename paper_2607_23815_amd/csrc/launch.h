// Internal launch entry points of the gfx950 kernels (called by api.cpp after argument
// validation). Every pointer is device memory; every size was checked on the host.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace pkv {

struct KvView {
  uint16_t* k;  // bf16 [num_blocks][hkv][D/8][16][8]
  uint16_t* v;  // bf16 [num_blocks][hkv][D][16]
  int32_t num_blocks;
  int32_t hkv;
  int32_t head_dim;
};

hipError_t launch_kv_append(const KvView& kv, const uint16_t* k_new, const uint16_t* v_new,
                            const int32_t* block_tables, int32_t max_blocks,
                            const int32_t* cached_lens, const int32_t* cu_new_lens,
                            int32_t num_seqs, int32_t max_new_len, hipStream_t stream);

hipError_t launch_gather_kv(const KvView& kv, const int32_t* block_tables, int32_t max_blocks,
                            const int32_t* lens, const int32_t* cu_lens, int32_t num_seqs,
                            int32_t max_len, uint16_t* k_out, uint16_t* v_out,
                            hipStream_t stream);

hipError_t launch_copy_blocks(const KvView& kv, const int32_t* pairs, int32_t num_pairs,
                              hipStream_t stream);

// Prefill plan, from the host arguments only. Key split: a batch whose work items cannot
// fill the chip (few sequences, few new tokens) and whose keys are long has each item's keys
// cut at multiples of split_keys (a multiple of 1024) into nsplit parts, run as separate work
// items and merged; otherwise split_keys = 0 and nsplit = 1. Order: a batch with long keys
// (up to at least 8192) takes its sequences longest first.
struct PrefillSplit {
  int32_t split_keys;
  int32_t nsplit;
  bool order;
};
PrefillSplit prefill_split_plan(int32_t num_seqs, int32_t hq, int32_t hkv, int32_t max_new_len,
                                int32_t max_total_len);
// Workspace of the plan (0 when it needs none): the sequence order when ordered, then when
// split the fp32 partial outputs [total_new][hq][nsplit][head_dim] and their (maximum, weight
// sum) pairs.
size_t prefill_workspace_bytes(int32_t num_seqs, int32_t total_new, int32_t hq, int32_t hkv,
                               int32_t head_dim, int32_t max_new_len, int32_t max_total_len);
// With workspace == nullptr the launch does not split.
hipError_t launch_prefill(const KvView& kv, const uint16_t* q, int32_t hq,
                          const int32_t* block_tables, int32_t max_blocks,
                          const int32_t* cached_lens, const int32_t* cu_new_lens,
                          int32_t num_seqs, int32_t total_new, int32_t max_new_len,
                          int32_t max_total_len, float scale, uint16_t* out, float* lse,
                          void* workspace, hipStream_t stream);

// Decode: keys are cut into splits of `split_keys` (a multiple of 32) keys.
int32_t decode_split_keys(int32_t num_seqs, int32_t hkv, int32_t max_seq_len);
size_t decode_workspace_bytes(int32_t num_seqs, int32_t hq, int32_t hkv, int32_t head_dim,
                              int32_t max_seq_len);
// The pieces of a decode launch, shared with the mixed launch: the split plan and the
// workspace layout (the sequence order, then the splits' partial results), the ordering
// kernel, and the merge of partial results (nothing when no sequence splits).
struct DecodePlan {
  int32_t split, max_splits;
  int32_t* order;
  float* ws_o;
  float* ws_ml;
  int64_t items;  // (sequence, kv head, split) work items
};
DecodePlan decode_plan(const KvView& kv, int32_t hq, int32_t num_seqs, int32_t max_seq_len,
                       void* workspace);
hipError_t launch_decode_order(const int32_t* seq_lens, int32_t num_seqs, int32_t* order,
                               hipStream_t stream);
// Longest-first order of sequences by lens[i] (+ cu[i + 1] - cu[i] when cu is given), and the
// bytes it takes in a workspace (256-byte rounded).
hipError_t launch_seq_order(const int32_t* lens, const int32_t* cu, int32_t num_seqs,
                            int32_t* order, hipStream_t stream);
size_t order_bytes(int32_t num_seqs);
hipError_t launch_decode_merge(const KvView& kv, const DecodePlan& p, int32_t hq,
                               const int32_t* seq_lens, int32_t num_seqs, uint16_t* out,
                               float* lse, hipStream_t stream);
hipError_t launch_decode(const KvView& kv, const uint16_t* q, int32_t hq,
                         const int32_t* block_tables, int32_t max_blocks,
                         const int32_t* seq_lens, int32_t num_seqs, int32_t max_seq_len,
                         float scale, uint16_t* out, float* lse, void* workspace,
                         hipStream_t stream);

// The allocation-free decode's workspace (a file-scope device array of kDecodeScratchBytes):
// its address on the current device, looked up on the first call per device.
constexpr size_t kDecodeScratchBytes = size_t(32) << 20;
hipError_t decode_scratch(void** ptr);

// Opt-in metadata validation (PKV_DEBUG_VALIDATE). One check per batch of a call: for
// append / prefill, `lens` are the cached lengths and `cu` the new-token offsets (ending at
// `total`), each sequence's new tokens at most `max_len` and cached + new at most
// `max_total`; for decode, `lens` are the sequence lengths (1 .. max_len); for gather, `lens`
// the gathered lengths (at most max_len, equal to the cu steps). Every table entry the call
// reads or writes must name a pool block.
enum : int32_t { kMetaAppend = 0, kMetaPrefill = 1, kMetaDecode = 2, kMetaGather = 3 };
enum : uint32_t { kMetaBadBlockId = 1u, kMetaBadLength = 2u, kMetaBadOffsets = 4u };
struct MetaCheck {
  int32_t mode;
  const int32_t* tables;
  int32_t max_blocks;
  int32_t num_blocks;
  const int32_t* lens;
  const int32_t* cu;  // null for decode
  int32_t num_seqs;
  int64_t total;      // cu[num_seqs] must equal it (< 0: not checked)
  int64_t max_len;
  int64_t max_total;
};
// Runs the checks in order on `stream` and waits for each; *bad = the failed check's bits
// (0 if all pass), *first_seq its lowest offending sequence, *which its index.
hipError_t validate_metadata(const MetaCheck* checks, int n_checks, hipStream_t stream,
                             uint32_t* bad, int32_t* first_seq, int32_t* which);

// Mixed launch: a prefill batch (arguments as launch_prefill) and a decode batch (d_*, as
// launch_decode, with its workspace) in one fused kernel between the decode's ordering
// kernel and its merge. Both batches must be non-empty.
hipError_t launch_mixed(const KvView& kv, int32_t hq, float scale, const uint16_t* q,
                        const int32_t* block_tables, int32_t max_blocks,
                        const int32_t* cached_lens, const int32_t* cu_new_lens, int32_t num_seqs,
                        int32_t max_new_len, uint16_t* out, float* lse, const uint16_t* dq,
                        const int32_t* d_block_tables, int32_t d_max_blocks,
                        const int32_t* seq_lens, int32_t d_num_seqs, int32_t max_seq_len,
                        uint16_t* d_out, float* d_lse, void* workspace, hipStream_t stream);

}  // namespace pkv
