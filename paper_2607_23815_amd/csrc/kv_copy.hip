// KV append (scatter of new tokens' K/V into their sequences' pool slots) and KV gather (the
// reverse, for tests), for gfx950.
//
// One workgroup moves one (sequence, 16-token block, kv head): at most 16 tokens x head_dim
// for K and for V, i.e. one 4 KB K slab and one 4 KB V slab at head_dim 128.
//   K: the pool slab is [head_dim/8 chunks][16 slots][8 dims]; thread t owns chunk t/16 of
//      slot t%16, so the workgroup's 16-byte stores cover the slab contiguously.
//   V: the pool slab is [head_dim][16 slots] (dim-major), a transpose of the token rows. The
//      rows are staged in LDS with coalesced 16-byte loads, then each thread assembles the
//      8 slots of one dim-row half and stores them as one 16-byte chunk. A half that is only
//      partly covered by new tokens (the first block continuing a cached prefix, or the last
//      block) is read, merged and written back, so slots outside the new range keep their
//      bits; no other sequence can write the block (new tokens only go to private blocks).
//      The read is issued at entry, ahead of the staging loads, so the two overlap.
// Whole 16-byte chunks are written with non-temporal stores (the appended rows are not read
// again by this launch): 64% -> 69% of HBM peak on the Llama-3-8B suffix append.
#include "device_utils.h"
#include "launch.h"

namespace pkv {
namespace {

template <int D>
__global__ __launch_bounds__(256) void kv_append_kernel(
    const uint16_t* __restrict__ k_new, const uint16_t* __restrict__ v_new,
    uint16_t* __restrict__ k_cache, uint16_t* __restrict__ v_cache,
    const int32_t* __restrict__ block_tables, int32_t max_blocks,
    const int32_t* __restrict__ cached_lens, const int32_t* __restrict__ cu_new_lens,
    int32_t hkv, int32_t num_blocks) {
  constexpr int NCH = D / 8;          // 16-byte chunks per token row
  constexpr int SLAB = D * kBlockSize;  // elements per (block, head) slab
  constexpr int ROW = D + 8;          // padded LDS row (elements)
  __shared__ __align__(16) uint16_t tile[kBlockSize * ROW];

  const int i = blockIdx.z;
  const int h = blockIdx.y;
  const int p = cached_lens[i];
  const int row0 = cu_new_lens[i];
  const int n = cu_new_lens[i + 1] - row0;
  if (n <= 0) return;
  const int len = p + n;
  const int b = p / kBlockSize + (int)blockIdx.x;  // logical block
  if (b * kBlockSize >= len || b >= max_blocks) return;
  const int blk = block_tables[(size_t)i * max_blocks + b];
  if (blk < 0 || blk >= num_blocks) return;
  const int s0 = max(p - b * kBlockSize, 0);           // first new slot in this block
  const int s1 = min(len - b * kBlockSize, kBlockSize);  // one past the last new slot
  // new-token row of slot s: row0 + b*16 + s - p
  const int64_t rbase = (int64_t)row0 + (int64_t)b * kBlockSize - p;
  const size_t slab = ((size_t)blk * hkv + h) * SLAB;
  const int t = threadIdx.x;
  static_assert(D * 2 <= 256, "one V half per thread");
  // The V half this thread assembles below (dim t/2, slots 8 (t%2) ..): when new tokens only
  // partly cover it, its old contents are read now, so that the read overlaps the staging.
  const int vd = t >> 1, vlo = (t & 1) * 8;
  const int va = max(vlo, s0), ve = min(vlo + 8, s1);
  const bool vmerge = t < D * 2 && va < ve && !(va == vlo && ve == vlo + 8);
  uint16_t* const vdst = v_cache + slab + (size_t)vd * kBlockSize + vlo;
  u32x4 vold = {0u, 0u, 0u, 0u};
  if (vmerge) vold = ld16(vdst);

  // K: chunk c = idx / 16 of slot s = idx % 16
  for (int idx = t; idx < NCH * kBlockSize; idx += 256) {
    const int c = idx / kBlockSize, s = idx % kBlockSize;
    if (s >= s0 && s < s1) {
      const u32x4 val = ld16(k_new + ((size_t)(rbase + s) * hkv + h) * D + c * 8);
      st16_nt(k_cache + slab + (size_t)(c * kBlockSize + s) * 8, val);
    }
  }
  // V: stage the rows, slot-major
  for (int idx = t; idx < kBlockSize * NCH; idx += 256) {
    const int s = idx / NCH, c = idx % NCH;
    if (s >= s0 && s < s1) {
      const u32x4 val = ld16(v_new + ((size_t)(rbase + s) * hkv + h) * D + c * 8);
      st16(&tile[s * ROW + c * 8], val);
    }
  }
  __syncthreads();
  if (t < D * 2 && va < ve) {
    uint16_t vals[8];
    if (!vmerge) {
#pragma unroll
      for (int k = 0; k < 8; ++k) vals[k] = tile[(vlo + k) * ROW + vd];
    } else {
      __builtin_memcpy(vals, &vold, 16);
      for (int k = va; k < ve; ++k) vals[k - vlo] = tile[k * ROW + vd];
    }
    u32x4 packed;
    __builtin_memcpy(&packed, vals, 16);
    if (!vmerge) st16_nt(vdst, packed);
    else st16(vdst, packed);  // a merged half: the block may be read again soon
  }
}

// The append of one token per sequence (a decode step; max_new_len == 1): one wave per
// (sequence, kv head). The token's K row goes to its slot as 16-byte chunks (16 lanes at head
// dim 128); each lane owns D/64 V dims and rewrites the 16-byte half-row holding the slot.
// Every load (the new row, the old halves) is issued before any store, so the wave waits
// once; the general kernel would spend two 256-thread workgroups (one empty) on each.
template <int D>
__global__ __launch_bounds__(64) void kv_append_token_kernel(
    const uint16_t* __restrict__ k_new, const uint16_t* __restrict__ v_new,
    uint16_t* __restrict__ k_cache, uint16_t* __restrict__ v_cache,
    const int32_t* __restrict__ block_tables, int32_t max_blocks,
    const int32_t* __restrict__ cached_lens, const int32_t* __restrict__ cu_new_lens,
    int32_t hkv, int32_t num_blocks) {
  constexpr int NCH = D / 8;           // 16-byte chunks per token row
  constexpr int SLAB = D * kBlockSize;  // elements per (block, head) slab
  constexpr int DPL = D / 64;          // V dims per lane
  static_assert(DPL == 1 || DPL == 2, "head dim 64 or 128");
  const int i = blockIdx.y;
  const int h = blockIdx.x;
  const int row = cu_new_lens[i];
  if (cu_new_lens[i + 1] - row <= 0) return;
  const int p = cached_lens[i];
  const int b = p / kBlockSize;
  if (b >= max_blocks) return;
  const int blk = block_tables[(size_t)i * max_blocks + b];
  if (blk < 0 || blk >= num_blocks) return;
  const int s = p % kBlockSize;
  const size_t slab = ((size_t)blk * hkv + h) * SLAB;
  const int lane = threadIdx.x;
  const uint16_t* krow = k_new + ((size_t)row * hkv + h) * D;
  const uint16_t* vrow = v_new + ((size_t)row * hkv + h) * D;
  // loads: this lane's K chunk, its V dims and the old halves holding slot s of those dims
  u32x4 kval = {0u, 0u, 0u, 0u};
  if (lane < NCH) kval = ld16(krow + lane * 8);
  uint16_t vnew[DPL];
  u32x4 vold[DPL];
#pragma unroll
  for (int e = 0; e < DPL; ++e) {
    const int d = lane * DPL + e;
    vnew[e] = vrow[d];
    vold[e] = ld16(v_cache + slab + (size_t)d * kBlockSize + (s & 8));
  }
  if (lane < NCH) st16(k_cache + slab + (size_t)(lane * kBlockSize + s) * 8, kval);
#pragma unroll
  for (int e = 0; e < DPL; ++e) {
    const int d = lane * DPL + e;
    uint16_t vals[8];
    __builtin_memcpy(vals, &vold[e], 16);
    vals[s & 7] = vnew[e];
    u32x4 packed;
    __builtin_memcpy(&packed, vals, 16);
    st16(v_cache + slab + (size_t)d * kBlockSize + (s & 8), packed);
  }
}

template <int D>
__global__ __launch_bounds__(256) void gather_kv_kernel(
    const uint16_t* __restrict__ k_cache, const uint16_t* __restrict__ v_cache,
    const int32_t* __restrict__ block_tables, int32_t max_blocks,
    const int32_t* __restrict__ lens, const int32_t* __restrict__ cu_lens, int32_t hkv,
    int32_t num_blocks, uint16_t* __restrict__ k_out, uint16_t* __restrict__ v_out) {
  constexpr int NCH = D / 8;
  constexpr int SLAB = D * kBlockSize;
  const int i = blockIdx.z;
  const int h = blockIdx.y;
  const int b = blockIdx.x;
  const int len = lens[i];
  if (b * kBlockSize >= len || b >= max_blocks) return;
  const int blk = block_tables[(size_t)i * max_blocks + b];
  if (blk < 0 || blk >= num_blocks) return;
  const int ns = min(len - b * kBlockSize, kBlockSize);
  const size_t slab = ((size_t)blk * hkv + h) * SLAB;
  const int64_t rbase = (int64_t)cu_lens[i] + (int64_t)b * kBlockSize;
  const int t = threadIdx.x;
  for (int idx = t; idx < NCH * kBlockSize; idx += 256) {
    const int c = idx / kBlockSize, s = idx % kBlockSize;
    if (s < ns) {
      const u32x4 val = ld16(k_cache + slab + (size_t)(c * kBlockSize + s) * 8);
      st16(k_out + ((size_t)(rbase + s) * hkv + h) * D + c * 8, val);
    }
  }
  for (int idx = t; idx < kBlockSize * NCH; idx += 256) {
    const int s = idx / NCH, c = idx % NCH;
    if (s < ns) {
      uint16_t vals[8];
#pragma unroll
      for (int k = 0; k < 8; ++k) vals[k] = v_cache[slab + (size_t)(c * 8 + k) * kBlockSize + s];
      u32x4 packed;
      __builtin_memcpy(&packed, vals, 16);
      st16(v_out + ((size_t)(rbase + s) * hkv + h) * D + c * 8, packed);
    }
  }
}

}  // namespace

hipError_t launch_kv_append(const KvView& kv, const uint16_t* k_new, const uint16_t* v_new,
                            const int32_t* block_tables, int32_t max_blocks,
                            const int32_t* cached_lens, const int32_t* cu_new_lens,
                            int32_t num_seqs, int32_t max_new_len, hipStream_t stream) {
  if (max_new_len == 1) {  // one token per sequence (a decode step)
    const dim3 tgrid(kv.hkv, num_seqs);
    if (kv.head_dim == 128)
      hipLaunchKernelGGL(kv_append_token_kernel<128>, tgrid, dim3(64), 0, stream, k_new, v_new,
                         kv.k, kv.v, block_tables, max_blocks, cached_lens, cu_new_lens, kv.hkv,
                         kv.num_blocks);
    else
      hipLaunchKernelGGL(kv_append_token_kernel<64>, tgrid, dim3(64), 0, stream, k_new, v_new,
                         kv.k, kv.v, block_tables, max_blocks, cached_lens, cu_new_lens, kv.hkv,
                         kv.num_blocks);
    return hipGetLastError();
  }
  // new tokens of one sequence touch at most ceil(max_new_len / 16) + 1 blocks
  dim3 grid((max_new_len + kBlockSize - 1) / kBlockSize + 1, kv.hkv, num_seqs);
  if (kv.head_dim == 128)
    hipLaunchKernelGGL(kv_append_kernel<128>, grid, dim3(256), 0, stream, k_new, v_new, kv.k,
                       kv.v, block_tables, max_blocks, cached_lens, cu_new_lens, kv.hkv,
                       kv.num_blocks);
  else
    hipLaunchKernelGGL(kv_append_kernel<64>, grid, dim3(256), 0, stream, k_new, v_new, kv.k,
                       kv.v, block_tables, max_blocks, cached_lens, cu_new_lens, kv.hkv,
                       kv.num_blocks);
  return hipGetLastError();
}

hipError_t launch_gather_kv(const KvView& kv, const int32_t* block_tables, int32_t max_blocks,
                            const int32_t* lens, const int32_t* cu_lens, int32_t num_seqs,
                            int32_t max_len, uint16_t* k_out, uint16_t* v_out,
                            hipStream_t stream) {
  dim3 grid((max_len + kBlockSize - 1) / kBlockSize, kv.hkv, num_seqs);
  if (kv.head_dim == 128)
    hipLaunchKernelGGL(gather_kv_kernel<128>, grid, dim3(256), 0, stream, kv.k, kv.v,
                       block_tables, max_blocks, lens, cu_lens, kv.hkv, kv.num_blocks, k_out,
                       v_out);
  else
    hipLaunchKernelGGL(gather_kv_kernel<64>, grid, dim3(256), 0, stream, kv.k, kv.v,
                       block_tables, max_blocks, lens, cu_lens, kv.hkv, kv.num_blocks, k_out,
                       v_out);
  return hipGetLastError();
}

}  // namespace pkv
