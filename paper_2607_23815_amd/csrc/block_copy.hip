// Whole-block copies for copy-on-write, for gfx950. A block's K region for all kv heads is one
// contiguous span of hkv * D * 16 elements of the K cache ([block][hkv][D/8][16][8]), and
// likewise its V region ([block][hkv][D][16]), so a copy is a plain 16-byte vector copy,
// coalesced across the workgroup.
#include "device_utils.h"
#include "launch.h"

namespace pkv {
namespace {

// workgroup (k, which) copies the K (which = 0) or V (which = 1) region of block pairs[2k]
// to block pairs[2k+1]; a pair naming a block outside the pool is skipped
__global__ __launch_bounds__(256) void copy_blocks_kernel(uint16_t* __restrict__ k_cache,
                                                          uint16_t* __restrict__ v_cache,
                                                          const int32_t* __restrict__ pairs,
                                                          int32_t num_blocks, int64_t span) {
  const int32_t src = pairs[2 * blockIdx.x];
  const int32_t dst = pairs[2 * blockIdx.x + 1];
  if (src < 0 || src >= num_blocks || dst < 0 || dst >= num_blocks || src == dst) return;
  uint16_t* base = blockIdx.y == 0 ? k_cache : v_cache;
  const u32x4* from = reinterpret_cast<const u32x4*>(base + (size_t)src * span);
  u32x4* to = reinterpret_cast<u32x4*>(base + (size_t)dst * span);
  const int64_t n = span / 8;  // 16-byte chunks
  for (int64_t c = threadIdx.x; c < n; c += 256) to[c] = from[c];
}

}  // namespace

hipError_t launch_copy_blocks(const KvView& kv, const int32_t* pairs, int32_t num_pairs,
                              hipStream_t stream) {
  const int64_t span = (int64_t)kv.hkv * kv.head_dim * kBlockSize;
  hipLaunchKernelGGL(copy_blocks_kernel, dim3(num_pairs, 2), dim3(256), 0, stream, kv.k, kv.v,
                     pairs, kv.num_blocks, span);
  return hipGetLastError();
}

}  // namespace pkv
