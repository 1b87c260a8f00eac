// Prefix-reuse paged prefill attention for gfx950: the prefill-only launch. The workgroup
// body (work items, staging, the matrix-core products and the online softmax) is in
// prefill_impl.h.
#include "launch.h"
#include "prefill_impl.h"

namespace pkv {
namespace {

template <int D>
__global__ __attribute__((amdgpu_flat_work_group_size(pre::kThreads, pre::kThreads),
                          amdgpu_waves_per_eu(2, 2)))
void prefill_kernel(const uint16_t* __restrict__ q, const uint16_t* __restrict__ k_cache,
                    const uint16_t* __restrict__ v_cache, const int32_t* __restrict__ block_tables,
                    int32_t max_blocks, const int32_t* __restrict__ cached_lens,
                    const int32_t* __restrict__ cu_new_lens, int32_t num_seqs, int32_t hq,
                    int32_t hkv, int32_t num_blocks, int32_t qtiles, float scale_log2,
                    uint16_t* __restrict__ out, float* __restrict__ lse) {
  pre::prefill_body<D>(q, k_cache, v_cache, block_tables, max_blocks, cached_lens, cu_new_lens,
                       num_seqs, hq, hkv, num_blocks, qtiles, scale_log2, out, lse,
                       blockIdx.x);
}

}  // namespace

hipError_t launch_prefill(const KvView& kv, const uint16_t* q, int32_t hq,
                          const int32_t* block_tables, int32_t max_blocks,
                          const int32_t* cached_lens, const int32_t* cu_new_lens,
                          int32_t num_seqs, int32_t max_new_len, float scale, uint16_t* out,
                          float* lse, hipStream_t stream) {
  const pre::PrefillGrid pg = pre::prefill_grid(hq, kv.hkv, num_seqs, max_new_len);
  if (pg.items > INT32_MAX) return hipErrorInvalidValue;
  const int64_t qtiles = pg.qtiles;
  const dim3 grid((unsigned)pg.items);
  const float scale_log2 = scale * kLog2e;
  if (kv.head_dim == 128)
    hipLaunchKernelGGL(prefill_kernel<128>, grid, dim3(pre::kThreads), 0, stream, q, kv.k, kv.v,
                       block_tables, max_blocks, cached_lens, cu_new_lens, num_seqs, hq, kv.hkv,
                       kv.num_blocks, (int32_t)qtiles, scale_log2, out, lse);
  else
    hipLaunchKernelGGL(prefill_kernel<64>, grid, dim3(pre::kThreads), 0, stream, q, kv.k, kv.v,
                       block_tables, max_blocks, cached_lens, cu_new_lens, num_seqs, hq, kv.hkv,
                       kv.num_blocks, (int32_t)qtiles, scale_log2, out, lse);
  return hipGetLastError();
}

}  // namespace pkv
