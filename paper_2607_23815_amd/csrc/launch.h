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

hipError_t launch_prefill(const KvView& kv, const uint16_t* q, int32_t hq,
                          const int32_t* block_tables, int32_t max_blocks,
                          const int32_t* cached_lens, const int32_t* cu_new_lens,
                          int32_t num_seqs, int32_t max_new_len, float scale, uint16_t* out,
                          float* lse, hipStream_t stream);

// Decode: keys are cut into splits of `split_keys` (a multiple of 32) keys.
int32_t decode_split_keys(int32_t num_seqs, int32_t hkv, int32_t max_seq_len);
size_t decode_workspace_bytes(int32_t num_seqs, int32_t hq, int32_t hkv, int32_t head_dim,
                              int32_t max_seq_len);
hipError_t launch_decode(const KvView& kv, const uint16_t* q, int32_t hq,
                         const int32_t* block_tables, int32_t max_blocks,
                         const int32_t* seq_lens, int32_t num_seqs, int32_t max_seq_len,
                         float scale, uint16_t* out, float* lse, void* workspace,
                         hipStream_t stream);

}  // namespace pkv
