// Paged decode attention for gfx950: the decode launch (an ordering kernel, the split work
// items, and the merge of split partial results). The work-item body is in decode_impl.h.
#include <math.h>

#include <mutex>

#include "decode_impl.h"
#include "launch.h"

namespace pkv {
namespace {

constexpr int kWaves = 4;  // waves per workgroup of the merge kernel

// Work item = (sequence, kv head, split) = one single-wave workgroup, so a compute unit takes
// new work as soon as any wave ends (work items differ in length).
template <int D>
__global__ __launch_bounds__(64) __attribute__((amdgpu_waves_per_eu(2, 2))) void decode_partial_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k_cache,
    const uint16_t* __restrict__ v_cache, const int32_t* __restrict__ block_tables,
    int32_t max_blocks, const int32_t* __restrict__ seq_lens, int32_t num_seqs, int32_t hq,
    int32_t hkv, int32_t num_blocks, int32_t split_keys, int32_t max_splits, float scale_log2,
    float* __restrict__ ws_o, float* __restrict__ ws_ml, uint16_t* __restrict__ out,
    float* __restrict__ lse, const int32_t* __restrict__ order) {
  dec::decode_body<D>(q, k_cache, v_cache, block_tables, max_blocks, seq_lens, num_seqs, hq, hkv,
                      num_blocks, split_keys, max_splits, scale_log2, ws_o, ws_ml, out, lse,
                      order, blockIdx.x);
}

// One wave per (sequence, query head): combine the splits' partial (m_s, l_s, acc_s):
//   out = sum_s 2^(m_s - M) acc_s / sum_s 2^(m_s - M) l_s,   M = max_s m_s.
template <int D>
__global__ __launch_bounds__(256) void decode_merge_kernel(
    const float* __restrict__ ws_o, const float* __restrict__ ws_ml,
    const int32_t* __restrict__ seq_lens, int32_t num_seqs, int32_t hq, int32_t split_keys,
    int32_t max_splits, uint16_t* __restrict__ out, float* __restrict__ lse) {
  constexpr int PER = D / 64;  // dims per lane
  const int64_t item = (int64_t)blockIdx.x * kWaves + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (item >= (int64_t)num_seqs * hq) return;
  const int i = (int)(item / hq);
  // the partial kernel's cut of an over-long length (at most max_splits splits)
  const int len = min(seq_lens[i], max_splits * split_keys);
  const int nsplit = (len + split_keys - 1) / split_keys;
  if (nsplit <= 1) return;  // written directly by the partial kernel
  const size_t base = (size_t)item * max_splits;
  float mmax = -INFINITY;
  for (int s = 0; s < nsplit; ++s) mmax = fmaxf(mmax, ws_ml[(base + s) * 2]);
  float den = 0.f;
  float o[PER];
#pragma unroll
  for (int e = 0; e < PER; ++e) o[e] = 0.f;
  for (int s = 0; s < nsplit; ++s) {
    const float w = fast_exp2(ws_ml[(base + s) * 2] - mmax);
    den += w * ws_ml[(base + s) * 2 + 1];
    const float* src = ws_o + (base + s) * D + lane * PER;
#pragma unroll
    for (int e = 0; e < PER; ++e) o[e] += w * src[e];
  }
  const float inv = 1.f / den;
  uint16_t* dst = out + (size_t)item * D + lane * PER;
  if constexpr (PER == 2) {
    *reinterpret_cast<uint32_t*>(dst) = pack_bf16x2(o[0] * inv, o[1] * inv);
  } else {
    dst[0] = (uint16_t)(pack_bf16x2(o[0] * inv, 0.f) & 0xFFFFu);
  }
  if (lse != nullptr && lane == 0) lse[item] = (mmax + log2f(den)) * kLn2;
}

// Longest-first sequence order for a decode or prefill grid: work is dispatched in item
// order, so taking the longest sequences first keeps the launch from ending on a few long
// items. A sequence's length is lens[i], plus cu[i + 1] - cu[i] when cu is given (a prefill's
// cached and new tokens). Sequences are bucketed by length on a log scale (32 buckets per
// factor of two), counted, scanned in descending bucket order and scattered; order within a
// bucket follows the scatter's atomics and may differ from run to run, which the results do
// not depend on.
constexpr int kOrderBuckets = 2048;
constexpr int kOrderThreads = 1024;
__global__ __launch_bounds__(kOrderThreads) void decode_order_kernel(
    const int32_t* __restrict__ seq_lens, const int32_t* __restrict__ cu, int32_t num_seqs,
    int32_t* __restrict__ order) {
  constexpr int kWavesO = kOrderThreads / 64;
  __shared__ int count[kOrderBuckets];
  __shared__ int base[kOrderBuckets];
  __shared__ int wsum[kWavesO];
  const int t = threadIdx.x;
  const int lane = t & 63, w = t >> 6;
  for (int b = t; b < kOrderBuckets; b += kOrderThreads) count[b] = 0;
  __syncthreads();
  auto bucket_of = [&](int i) {
    const int len = seq_lens[i] + (cu != nullptr ? cu[i + 1] - cu[i] : 0);
    if (len < 1) return 0;
    return min(1 + (int)(log2f((float)len) * 32.f), kOrderBuckets - 1);
  };
  for (int i = t; i < num_seqs; i += kOrderThreads) atomicAdd(&count[bucket_of(i)], 1);
  __syncthreads();
  // exclusive scan in descending bucket order: thread t owns descending positions 2t, 2t+1;
  // an inclusive scan within each wave (lane shuffles), then one over the waves' totals
  const int b0 = kOrderBuckets - 1 - 2 * t, b1 = b0 - 1;
  const int c0 = count[b0], c1 = count[b1];
  const int v = c0 + c1;
  int incl = v;
  for (int off = 1; off < 64; off <<= 1) {
    const int u = __shfl_up(incl, off, 64);
    if (lane >= off) incl += u;
  }
  if (lane == 63) wsum[w] = incl;
  __syncthreads();
  if (w == 0) {
    const int x = lane < kWavesO ? wsum[lane] : 0;
    int inc = x;
    for (int off = 1; off < kWavesO; off <<= 1) {
      const int u = __shfl_up(inc, off, 64);
      if (lane >= off) inc += u;
    }
    if (lane < kWavesO) wsum[lane] = inc - x;  // waves before this one
  }
  __syncthreads();
  const int excl = wsum[w] + incl - v;
  base[b0] = excl;
  base[b1] = excl + c0;
  __syncthreads();
  for (int i = t; i < num_seqs; i += kOrderThreads) order[atomicAdd(&base[bucket_of(i)], 1)] = i;
}


constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

}  // namespace

// The allocation-free decode's workspace: one array per GPU, loaded with the code object and
// held until the process ends. Its device address comes from hipGetSymbolAddress, taken once
// per device with that device current; the array's name in host code is a host-side stand-in
// and never goes to a kernel or a copy.
static __device__ __align__(256) unsigned char scratch[kDecodeScratchBytes];

hipError_t decode_scratch(void** ptr) {
  int dev = 0;
  hipError_t err = hipGetDevice(&dev);
  if (err != hipSuccess) return err;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void* p = nullptr;
    err = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (err != hipSuccess) return err;
    g_scratch_ptr[dev] = p;
  }
  *ptr = g_scratch_ptr[dev];
  return hipSuccess;
}

int32_t decode_split_keys(int32_t num_seqs, int32_t hkv, int32_t max_seq_len) {
  // Longest split first (every split pays a prologue of dependent table and first KV loads
  // plus a partial write, so fewer, longer splits stream better); shorten it while the grid
  // would hold too few waves to keep all 256 compute units streaming (aim for >= 8 waves
  // per unit). A function of the call's sizes only, so a given call always splits
  // identically.
  int32_t split = 4096;
  while (split > 64) {
    const int64_t waves =
        (int64_t)num_seqs * hkv * ((max_seq_len + split - 1) / split);
    if (waves >= 2048) break;
    split /= 2;
  }
  return split;
}

size_t decode_workspace_bytes(int32_t num_seqs, int32_t hq, int32_t hkv, int32_t head_dim,
                              int32_t max_seq_len) {
  const int32_t split = decode_split_keys(num_seqs, hkv, max_seq_len);
  const int64_t max_splits = (max_seq_len + split - 1) / split;
  // the sequence order, then (when sequences split) the partial results
  size_t bytes = order_bytes(num_seqs);
  if (max_splits > 1) bytes += (size_t)num_seqs * hq * max_splits * (head_dim + 2) * sizeof(float);
  return bytes;
}

DecodePlan decode_plan(const KvView& kv, int32_t hq, int32_t num_seqs, int32_t max_seq_len,
                       void* workspace) {
  DecodePlan p;
  p.split = decode_split_keys(num_seqs, kv.hkv, max_seq_len);
  p.max_splits = (max_seq_len + p.split - 1) / p.split;
  p.order = static_cast<int32_t*>(workspace);
  p.ws_o = nullptr;
  p.ws_ml = nullptr;
  if (p.max_splits > 1) {
    p.ws_o = reinterpret_cast<float*>(static_cast<char*>(workspace) + order_bytes(num_seqs));
    p.ws_ml = p.ws_o + (size_t)num_seqs * hq * p.max_splits * kv.head_dim;
  }
  p.items = (int64_t)num_seqs * kv.hkv * p.max_splits;
  return p;
}

size_t order_bytes(int32_t num_seqs) {
  return ((size_t)num_seqs * sizeof(int32_t) + 255) / 256 * 256;
}

hipError_t launch_seq_order(const int32_t* lens, const int32_t* cu, int32_t num_seqs,
                            int32_t* order, hipStream_t stream) {
  hipLaunchKernelGGL(decode_order_kernel, dim3(1), dim3(kOrderThreads), 0, stream, lens, cu,
                     num_seqs, order);
  return hipGetLastError();
}

hipError_t launch_decode_order(const int32_t* seq_lens, int32_t num_seqs, int32_t* order,
                               hipStream_t stream) {
  return launch_seq_order(seq_lens, nullptr, num_seqs, order, stream);
}

hipError_t launch_decode_merge(const KvView& kv, const DecodePlan& p, int32_t hq,
                               const int32_t* seq_lens, int32_t num_seqs, uint16_t* out,
                               float* lse, hipStream_t stream) {
  if (p.max_splits <= 1) return hipSuccess;
  const int64_t rows = (int64_t)num_seqs * hq;
  const dim3 mgrid((unsigned)((rows + kWaves - 1) / kWaves));
  if (kv.head_dim == 128)
    hipLaunchKernelGGL(decode_merge_kernel<128>, mgrid, dim3(256), 0, stream, p.ws_o, p.ws_ml,
                       seq_lens, num_seqs, hq, p.split, p.max_splits, out, lse);
  else
    hipLaunchKernelGGL(decode_merge_kernel<64>, mgrid, dim3(256), 0, stream, p.ws_o, p.ws_ml,
                       seq_lens, num_seqs, hq, p.split, p.max_splits, out, lse);
  return hipGetLastError();
}

hipError_t launch_decode(const KvView& kv, const uint16_t* q, int32_t hq,
                         const int32_t* block_tables, int32_t max_blocks,
                         const int32_t* seq_lens, int32_t num_seqs, int32_t max_seq_len,
                         float scale, uint16_t* out, float* lse, void* workspace,
                         hipStream_t stream) {
  const DecodePlan p = decode_plan(kv, hq, num_seqs, max_seq_len, workspace);
  const dim3 grid((unsigned)p.items);
  const float scale_log2 = scale * kLog2e;
  hipError_t err = launch_decode_order(seq_lens, num_seqs, p.order, stream);
  if (err != hipSuccess) return err;
  if (kv.head_dim == 128)
    hipLaunchKernelGGL(decode_partial_kernel<128>, grid, dim3(64), 0, stream, q, kv.k, kv.v,
                       block_tables, max_blocks, seq_lens, num_seqs, hq, kv.hkv,
                       kv.num_blocks, p.split, p.max_splits, scale_log2, p.ws_o, p.ws_ml, out,
                       lse, p.order);
  else
    hipLaunchKernelGGL(decode_partial_kernel<64>, grid, dim3(64), 0, stream, q, kv.k, kv.v,
                       block_tables, max_blocks, seq_lens, num_seqs, hq, kv.hkv,
                       kv.num_blocks, p.split, p.max_splits, scale_log2, p.ws_o, p.ws_ml, out,
                       lse, p.order);
  err = hipGetLastError();
  if (err != hipSuccess) return err;
  return launch_decode_merge(kv, p, hq, seq_lens, num_seqs, out, lse, stream);
}

}  // namespace pkv
