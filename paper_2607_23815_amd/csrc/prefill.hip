// Prefix-reuse paged prefill attention for gfx950: the prefill-only launch, the key-split
// plan for batches too small to fill the chip, and the merge of split results. The
// workgroup body (work items, staging, the matrix-core products and the online softmax) is in
// prefill_impl.h.
#include <algorithm>

#include "launch.h"
#include "prefill_impl.h"

namespace pkv {
namespace {

// kPlan: the launch follows a plan (key splits and/or a longest-first sequence order; a
// separate instantiation, so that the common launch without either compiles as before)
template <int D, bool kPlan>
__global__ __attribute__((amdgpu_flat_work_group_size(pre::kThreads, pre::kThreads),
                          amdgpu_waves_per_eu(2, 2)))
void prefill_kernel(const uint16_t* __restrict__ q, const uint16_t* __restrict__ k_cache,
                    const uint16_t* __restrict__ v_cache, const int32_t* __restrict__ block_tables,
                    int32_t max_blocks, const int32_t* __restrict__ cached_lens,
                    const int32_t* __restrict__ cu_new_lens, int32_t num_seqs, int32_t hq,
                    int32_t hkv, int32_t num_blocks, int32_t qtiles, float scale_log2,
                    uint16_t* __restrict__ out, float* __restrict__ lse, int32_t split_keys,
                    int32_t nsplit, float* __restrict__ ws_o, float* __restrict__ ws_ml,
                    const int32_t* __restrict__ order) {
  if constexpr (kPlan)
    pre::prefill_body<D>(q, k_cache, v_cache, block_tables, max_blocks, cached_lens,
                         cu_new_lens, num_seqs, hq, hkv, num_blocks, qtiles, scale_log2, out,
                         lse, blockIdx.x, split_keys, nsplit, ws_o, ws_ml, order);
  else
    pre::prefill_body<D>(q, k_cache, v_cache, block_tables, max_blocks, cached_lens,
                         cu_new_lens, num_seqs, hq, hkv, num_blocks, qtiles, scale_log2, out,
                         lse, blockIdx.x);
}

// Merge of the split partial results: one wave per (new token, query head) row of sequence
// blockIdx.y. A row whose keys end in split 0 was written by the prefill kernel; any other
// row ends in split L = (P + j) / split_keys and has partials (acc_s, m_s, l_s) for
// s = 0 .. L:  out = sum_s 2^(m_s - M) acc_s / sum_s 2^(m_s - M) l_s, M = max_s m_s.
template <int D>
__global__ __launch_bounds__(256) void prefill_merge_kernel(
    const int32_t* __restrict__ cached_lens, const int32_t* __restrict__ cu_new_lens,
    int32_t hq, int32_t split_keys, int32_t nsplit, const float* __restrict__ ws_o,
    const float* __restrict__ ws_ml, uint16_t* __restrict__ out, float* __restrict__ lse) {
  const int i = blockIdx.y;
  const int lane = threadIdx.x & 63;
  const int r = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int row0 = cu_new_lens[i];
  const int n = cu_new_lens[i + 1] - row0;
  const int j = r / hq, h = r % hq;
  if (j >= n) return;
  const int last = (cached_lens[i] + j) / split_keys;  // the row's last split
  if (last == 0) return;
  const size_t slot0 = ((size_t)(row0 + j) * hq + h) * nsplit;
  // lane s holds split s's maximum and weight sum (splits past the row's last: none)
  float ms = -INFINITY, ls = 0.f;
  if (lane <= last) {
    ms = ws_ml[(slot0 + lane) * 2 + 0];
    ls = ws_ml[(slot0 + lane) * 2 + 1];
  }
  float mx = ms;
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o));
  const float w = lane <= last ? exp2f(ms - mx) : 0.f;
  float den = w * ls;
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) den += __shfl_xor(den, o);
  const float inv = 1.f / den;
  constexpr int PER = D / 64;  // dims per lane
  float acc[PER];
#pragma unroll
  for (int e = 0; e < PER; ++e) acc[e] = 0.f;
  for (int s = 0; s <= last; ++s) {
    const float ws = __shfl(w, s);
    const float* src = ws_o + (slot0 + s) * D + lane * PER;
#pragma unroll
    for (int e = 0; e < PER; ++e) acc[e] += ws * src[e];
  }
  uint16_t* dst = out + ((size_t)(row0 + j) * hq + h) * D + lane * PER;
  if constexpr (PER == 2) {
    *reinterpret_cast<uint32_t*>(dst) = pack_bf16x2(acc[0] * inv, acc[1] * inv);
  } else {
    const __bf16 b = (__bf16)(acc[0] * inv);
    *dst = __builtin_bit_cast(uint16_t, b);
  }
  if (lse != nullptr && lane == 0) lse[(size_t)(row0 + j) * hq + h] = (mx + log2f(den)) * kLn2;
}

}  // namespace

// Work items below which a prefill launch cannot keep every compute unit busy (two
// workgroups on each of the 256 compute units, four times over), and the smallest key split.
// On 4 tuples of 24-32k cached tokens (224 items) a target of 1024 items gave 5 splits and
// 0.323 ms, 2048 gave 8 splits and 0.306 ms, 16384 gave 32 splits and 0.397 ms (the
// partial results and the merge outweigh the balance).
constexpr int64_t kFillItems = 2048;
constexpr int32_t kSplitUnit = 1024;   // split_keys is a multiple of this (one table chunk)
constexpr int32_t kMaxSplits = 64;
// Keys from which a batch's sequences are taken longest first (a one-workgroup ordering
// kernel and one more dependent load per workgroup): with documents up to 16k keys the
// longest items would otherwise start anywhere in the launch and extend its end.
constexpr int32_t kOrderKeys = 8192;

PrefillSplit prefill_split_plan(int32_t num_seqs, int32_t hq, int32_t hkv, int32_t max_new_len,
                                int32_t max_total_len) {
  if (num_seqs <= 0 || hkv <= 0 || hq % hkv != 0 || max_new_len <= 0)
    return PrefillSplit{0, 1, false};
  const bool order = max_total_len >= kOrderKeys && num_seqs > 1;
  const PrefillSplit none{0, 1, order};
  if (max_total_len < 2 * kSplitUnit) return none;
  const pre::PrefillGrid pg = pre::prefill_grid(hq, hkv, num_seqs, max_new_len);
  const int64_t items = (int64_t)num_seqs * hkv * pg.qtiles;
  if (items >= kFillItems) return none;
  const int64_t want = std::min<int64_t>((kFillItems + items - 1) / items, kMaxSplits);
  int64_t keys = (max_total_len + want - 1) / want;
  keys = (keys + kSplitUnit - 1) / kSplitUnit * kSplitUnit;
  const int64_t nsplit = (max_total_len + keys - 1) / keys;
  if (nsplit <= 1) return none;
  return PrefillSplit{(int32_t)keys, (int32_t)nsplit, order};
}

size_t prefill_workspace_bytes(int32_t num_seqs, int32_t total_new, int32_t hq, int32_t hkv,
                               int32_t head_dim, int32_t max_new_len, int32_t max_total_len) {
  const PrefillSplit sp = prefill_split_plan(num_seqs, hq, hkv, max_new_len, max_total_len);
  if (total_new <= 0) return 0;
  size_t bytes = sp.order ? order_bytes(num_seqs) : 0;
  if (sp.nsplit > 1) bytes += (size_t)total_new * hq * sp.nsplit * (head_dim + 2) * sizeof(float);
  return bytes;
}

hipError_t launch_prefill(const KvView& kv, const uint16_t* q, int32_t hq,
                          const int32_t* block_tables, int32_t max_blocks,
                          const int32_t* cached_lens, const int32_t* cu_new_lens,
                          int32_t num_seqs, int32_t total_new, int32_t max_new_len,
                          int32_t max_total_len, float scale, uint16_t* out, float* lse,
                          void* workspace, hipStream_t stream) {
  PrefillSplit sp{0, 1, false};
  if (workspace != nullptr)
    sp = prefill_split_plan(num_seqs, hq, kv.hkv, max_new_len, max_total_len);
  int32_t* order = nullptr;
  float* ws_o = nullptr;
  float* ws_ml = nullptr;
  char* ws = static_cast<char*>(workspace);
  if (sp.order) {
    order = reinterpret_cast<int32_t*>(ws);
    ws += order_bytes(num_seqs);
    const hipError_t err = launch_seq_order(cached_lens, cu_new_lens, num_seqs, order, stream);
    if (err != hipSuccess) return err;
  }
  if (sp.nsplit > 1) {
    ws_o = reinterpret_cast<float*>(ws);
    ws_ml = ws_o + (size_t)total_new * hq * sp.nsplit * kv.head_dim;
  }
  const bool plan = sp.order || sp.nsplit > 1;
  const pre::PrefillGrid pg = pre::prefill_grid(hq, kv.hkv, num_seqs, max_new_len, sp.nsplit);
  if (pg.items > INT32_MAX) return hipErrorInvalidValue;
  const int64_t qtiles = pg.qtiles;
  const dim3 grid((unsigned)pg.items);
  const float scale_log2 = scale * kLog2e;
  auto* kern = kv.head_dim == 128 ? (plan ? prefill_kernel<128, true> : prefill_kernel<128, false>)
                                  : (plan ? prefill_kernel<64, true> : prefill_kernel<64, false>);
  hipLaunchKernelGGL(kern, grid, dim3(pre::kThreads), 0, stream, q, kv.k, kv.v, block_tables,
                     max_blocks, cached_lens, cu_new_lens, num_seqs, hq, kv.hkv, kv.num_blocks,
                     (int32_t)qtiles, scale_log2, out, lse, sp.split_keys, sp.nsplit, ws_o,
                     ws_ml, order);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess || sp.nsplit <= 1) return err;
  const dim3 mgrid((unsigned)(((int64_t)max_new_len * hq + 3) / 4), (unsigned)num_seqs);
  if (kv.head_dim == 128)
    hipLaunchKernelGGL(prefill_merge_kernel<128>, mgrid, dim3(256), 0, stream, cached_lens,
                       cu_new_lens, hq, sp.split_keys, sp.nsplit, ws_o, ws_ml, out, lse);
  else
    hipLaunchKernelGGL(prefill_merge_kernel<64>, mgrid, dim3(256), 0, stream, cached_lens,
                       cu_new_lens, hq, sp.split_keys, sp.nsplit, ws_o, ws_ml, out, lse);
  return hipGetLastError();
}

}  // namespace pkv
