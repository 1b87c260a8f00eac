// Mixed prefill + decode attention for gfx950: one fused launch in which some workgroups run
// prefill work items (the matrix-core-bound body of prefill_impl.h) and others run four
// decode work items, one per wave (the HBM-bound body of decode_impl.h), so that each compute
// unit overlaps the two kinds of work instead of running them one launch after the other.
//
// Workgroup b runs on XCD b % 8. Each XCD's list of positions b / 8 is dealt between prefill
// and decode workgroups in proportion to their counts, spread evenly along the list; a
// prefill workgroup keeps the XCD its index would have in a prefill-only launch (its index
// has the same residue mod 8), so the (sequence, kv head) groups keep their XCD and L2. The
// decode items follow the longest-first order of the decode launch, and the results are
// bit-identical to a prefill launch followed by a decode launch.
#include "decode_impl.h"
#include "launch.h"
#include "prefill_impl.h"

namespace pkv {
namespace {

constexpr int kDecodePerWg = pre::kThreads / 64;  // one decode item per wave

template <int D>
__global__ __attribute__((amdgpu_flat_work_group_size(pre::kThreads, pre::kThreads),
                          amdgpu_waves_per_eu(2, 2)))
void mixed_kernel(const uint16_t* __restrict__ q, const uint16_t* __restrict__ k_cache,
                  const uint16_t* __restrict__ v_cache, const int32_t* __restrict__ block_tables,
                  int32_t max_blocks, const int32_t* __restrict__ cached_lens,
                  const int32_t* __restrict__ cu_new_lens, int32_t num_seqs, int32_t hq,
                  int32_t hkv, int32_t num_blocks, int32_t qtiles, float scale_log2,
                  uint16_t* __restrict__ out, float* __restrict__ lse,
                  const uint16_t* __restrict__ dq, const int32_t* __restrict__ d_tables,
                  int32_t d_max_blocks, const int32_t* __restrict__ seq_lens, int32_t d_num_seqs,
                  int32_t split_keys, int32_t max_splits, float* __restrict__ ws_o,
                  float* __restrict__ ws_ml, uint16_t* __restrict__ d_out,
                  float* __restrict__ d_lse, const int32_t* __restrict__ order, int32_t p8,
                  int32_t d8, int64_t d_items) {
  const unsigned x = blockIdx.x & 7;
  const unsigned pos = blockIdx.x >> 3;
  const int64_t t8 = (int64_t)p8 + d8;
  // decode workgroups before position pos, and up to and including it
  const int64_t before = (int64_t)pos * d8 / t8;
  const int64_t upto = ((int64_t)pos + 1) * d8 / t8;
  if (upto > before) {
    const int64_t item =
        ((int64_t)before * 8 + x) * kDecodePerWg + (int64_t)(threadIdx.x >> 6);
    if (item >= d_items) return;
    dec::decode_body<D>(dq, k_cache, v_cache, d_tables, d_max_blocks, seq_lens, d_num_seqs, hq,
                        hkv, num_blocks, split_keys, max_splits, scale_log2, ws_o, ws_ml, d_out,
                        d_lse, order, item);
  } else {
    pre::prefill_body<D>(q, k_cache, v_cache, block_tables, max_blocks, cached_lens,
                         cu_new_lens, num_seqs, hq, hkv, num_blocks, qtiles, scale_log2, out,
                         lse, (unsigned)((pos - before) * 8 + x));
  }
}

}  // namespace

hipError_t launch_mixed(const KvView& kv, int32_t hq, float scale, const uint16_t* q,
                        const int32_t* block_tables, int32_t max_blocks,
                        const int32_t* cached_lens, const int32_t* cu_new_lens, int32_t num_seqs,
                        int32_t max_new_len, uint16_t* out, float* lse, const uint16_t* dq,
                        const int32_t* d_block_tables, int32_t d_max_blocks,
                        const int32_t* seq_lens, int32_t d_num_seqs, int32_t max_seq_len,
                        uint16_t* d_out, float* d_lse, void* workspace, hipStream_t stream) {
  const pre::PrefillGrid pg = pre::prefill_grid(hq, kv.hkv, num_seqs, max_new_len);
  const DecodePlan dp = decode_plan(kv, hq, d_num_seqs, max_seq_len, workspace);
  const int64_t d_wgs = (dp.items + kDecodePerWg - 1) / kDecodePerWg;
  const int64_t p8 = pg.items / 8;  // a multiple of 8 by construction
  const int64_t d8 = (d_wgs + 7) / 8;
  if (8 * (p8 + d8) > INT32_MAX) return hipErrorInvalidValue;
  const dim3 grid((unsigned)(8 * (p8 + d8)));
  const float scale_log2 = scale * kLog2e;
  hipError_t err = launch_decode_order(seq_lens, d_num_seqs, dp.order, stream);
  if (err != hipSuccess) return err;
  if (kv.head_dim == 128)
    hipLaunchKernelGGL(mixed_kernel<128>, grid, dim3(pre::kThreads), 0, stream, q, kv.k, kv.v,
                       block_tables, max_blocks, cached_lens, cu_new_lens, num_seqs, hq, kv.hkv,
                       kv.num_blocks, (int32_t)pg.qtiles, scale_log2, out, lse, dq,
                       d_block_tables, d_max_blocks, seq_lens, d_num_seqs, dp.split,
                       dp.max_splits, dp.ws_o, dp.ws_ml, d_out, d_lse, dp.order, (int32_t)p8,
                       (int32_t)d8, dp.items);
  else
    hipLaunchKernelGGL(mixed_kernel<64>, grid, dim3(pre::kThreads), 0, stream, q, kv.k, kv.v,
                       block_tables, max_blocks, cached_lens, cu_new_lens, num_seqs, hq, kv.hkv,
                       kv.num_blocks, (int32_t)pg.qtiles, scale_log2, out, lse, dq,
                       d_block_tables, d_max_blocks, seq_lens, d_num_seqs, dp.split,
                       dp.max_splits, dp.ws_o, dp.ws_ml, d_out, d_lse, dp.order, (int32_t)p8,
                       (int32_t)d8, dp.items);
  err = hipGetLastError();
  if (err != hipSuccess) return err;
  return launch_decode_merge(kv, dp, hq, seq_lens, d_num_seqs, d_out, d_lse, stream);
}

}  // namespace pkv
