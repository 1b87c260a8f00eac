// Paged decode attention for gfx950 (the per-wave work-item body, shared by the decode
// launch and the mixed prefill + decode launch): one query token per sequence over its whole cached
// context, split along the key axis ("split-K") so that every compute unit streams KV at the
// HBM rate, followed by a merge of the splits' partial results by their log-sum-exp weights.
//
// Work item = (sequence, kv head, split) = one single-wave workgroup, so a compute unit
// takes new work as soon as any wave ends (work items differ in length); there are no
// barriers and no LDS. Sequences are taken longest first (a small ordering kernel runs
// before the launch), so the launch does not end on a few long waves. Each wave streams its split
// 32 keys (two 16-token blocks) at a time straight from HBM into the matrix-core operands:
//   scores  S^T[32 keys][16 cols] = K[keys][D] . Q^T[D][cols]      (v_mfma 16x16x32 bf16)
//   values  O^T[D][16 cols]      += V^T[D][32 keys] . P^T[keys][cols]
// The columns are the g = Hq/Hkv query heads that share the kv head (g <= 16; unused columns
// carry zero queries), so every KV byte is read once per kv head, never once per query head.
// Both products take 16-byte K loads and 8-byte V loads that are contiguous across the wave:
// the K pool slab is chunk-major ([D/8][16 slots][8]), so lane (slot s, chunk group q) of
// load kk reads chunk q + 4kk of slot s and one instruction covers 1 KB contiguous; the V pool
// slab is dim-major ([D][16 slots]), so lanes read 4 consecutive slots of one dim.
// The online softmax runs in the base-2 domain (scale * log2 e folded in fp32); per-column
// max and sum are combined across the four lane groups holding a column with cross-lane
// shuffles. Keys outside the sequence (tail slots of its last block, which may hold any bits,
// NaN included) are removed by selection -- scores to -inf and V operands to zero -- never by
// multiplying by a zero weight.
// Split boundaries are multiples of the split size in key position only, so results are
// bit-identical from run to run and independent of where blocks sit in the pool.
#pragma once

#include <math.h>

#include "device_utils.h"

namespace pkv {
namespace dec {

__device__ __forceinline__ float wave_max16(float x) {
  // max over the four lanes l, l^16, l^32, l^48 (the lane groups holding one column)
  x = fmaxf(x, __shfl_xor(x, 16));
  x = fmaxf(x, __shfl_xor(x, 32));
  return x;
}
__device__ __forceinline__ float wave_sum16(float x) {
  x += __shfl_xor(x, 16);
  x += __shfl_xor(x, 32);
  return x;
}

// zero the 16-bit lanes of a 4-element V fragment whose key index (base + e) >= nvalid
__device__ __forceinline__ u32x2 mask_v4(u32x2 v, int base, int nvalid) {
  uint32_t w0 = v[0], w1 = v[1];
  if (base + 0 >= nvalid) w0 &= 0xFFFF0000u;
  if (base + 1 >= nvalid) w0 &= 0x0000FFFFu;
  if (base + 2 >= nvalid) w1 &= 0xFFFF0000u;
  if (base + 3 >= nvalid) w1 &= 0x0000FFFFu;
  u32x2 r = {w0, w1};
  return r;
}

// K and V operands of one 32-key step (two blocks) of one wave, straight from HBM:
// K: lane (slot col, group grp) holds chunk grp + 4 kk of slot col of each block;
// V: lane holds slots 4 grp .. 4 grp + 3 of dim row 16 db + col of each block.
template <int D>
struct DecodeFrag {
  u32x4 k[2][D / 32];
  u32x2 v[2][D / 16];
};

template <int D>
__device__ __forceinline__ void decode_load(DecodeFrag<D>& f, const uint16_t* __restrict__ k_cache,
                                            const uint16_t* __restrict__ v_cache, size_t b0_off,
                                            size_t b1_off, int col, int grp) {
  // wave-uniform slab bases plus 32-bit per-lane byte offsets
  constexpr int SLAB_BYTES = D * kBlockSize * 2;
  const uint16_t* k0 = k_cache + b0_off;
  const uint16_t* k1 = k_cache + b1_off;
  const uint16_t* v0 = v_cache + b0_off;
  const uint16_t* v1 = v_cache + b1_off;
#pragma unroll
  for (int kk = 0; kk < D / 32; ++kk) {
    const int o = ((grp + 4 * kk) * kBlockSize + col) * 16;
    f.k[0][kk] = buf_ld16(k0, SLAB_BYTES, o);
    f.k[1][kk] = buf_ld16(k1, SLAB_BYTES, o);
  }
#pragma unroll
  for (int db = 0; db < D / 16; ++db) {
    const int o = ((db * 16 + col) * kBlockSize + 4 * grp) * 2;
    f.v[0][db] = buf_ld8(v0, SLAB_BYTES, o);
    f.v[1][db] = buf_ld8(v1, SLAB_BYTES, o);
  }
}

// The body of one decode work item (sequence rank, kv head, split), run by one wave.
template <int D>
__device__ __forceinline__ void decode_body(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k_cache,
    const uint16_t* __restrict__ v_cache, const int32_t* __restrict__ block_tables,
    int32_t max_blocks, const int32_t* __restrict__ seq_lens, int32_t num_seqs, int32_t hq,
    int32_t hkv, int32_t num_blocks, int32_t split_keys, int32_t max_splits, float scale_log2,
    float* __restrict__ ws_o, float* __restrict__ ws_ml, uint16_t* __restrict__ out,
    float* __restrict__ lse, const int32_t* __restrict__ order, const int64_t item) {
  constexpr int KK = D / 32;   // k-steps of the score product
  constexpr int DB = D / 16;   // 16-dim blocks of the value product
  constexpr int SLAB = D * kBlockSize;
  const int g = hq / hkv;
  const int lane = threadIdx.x & 63;
  const int col = lane & 15;   // query head within the kv group (column)
  const int grp = lane >> 4;   // lane group 0..3
  const int64_t per_seq = (int64_t)hkv * max_splits;
  const int rank = (int)(item / per_seq);
  if (rank >= num_seqs) return;
  const int i = order[rank];  // longest sequences first
  const int rem = (int)(item % per_seq);
  const int kvh = rem / max_splits;
  const int sp = rem % max_splits;
  // A length above the host's max_seq_len breaks the caller's contract; it is cut to the
  // splits the launch planned (the merge cuts it the same way), and keys past the table are
  // not attended, so such a call computes over fewer keys but never leaves its workspace.
  // With max_seq_len <= max_blocks * 16 (checked on the host) every planned split starts
  // inside the table, so no split is empty.
  const int len = min(seq_lens[i], max_splits * split_keys);
  const int nsplit = (len + split_keys - 1) / split_keys;  // 0 for a length < 1: no output
  if (sp >= nsplit) return;
  const int k0 = sp * split_keys;
  int k1 = min(len, k0 + split_keys);
  if ((k1 - 1) / kBlockSize >= max_blocks) k1 = max_blocks * kBlockSize;  // (no overflow)
  const bool col_ok = col < g;
  const int h = kvh * g + col;

  bf16x8 qf[KK];
#pragma unroll
  for (int kk = 0; kk < KK; ++kk) {
    u32x4 v = {0u, 0u, 0u, 0u};
    if (col_ok) v = ld16(q + ((size_t)i * hq + h) * D + kk * 32 + grp * 8);
    qf[kk] = as_bf16x8(v);
  }

  // The split's blocks in per-lane register tables of 64 entries: chunk c holds, in lane l,
  // the pool offset of the split's block 64 c + l, or of pool block 0 (a stand-in that is
  // read but masked) for blocks past the split, past the table or out of the pool. Two
  // chunks are live (the current one and the next), so every load below is unconditional
  // and a step's 24 loads issue back to back and overlap the previous step.
  const int32_t* table = block_tables + (size_t)i * max_blocks;
  const int b_first = k0 / kBlockSize;
  const int nblk = (k1 - k0 + kBlockSize - 1) / kBlockSize;
  // (the load and the check are separate steps, so that the first two chunks' loads are both
  // in flight before either is checked)
  auto raw_chunk = [&](int c) -> int {
    const int r = 64 * c + lane;
    const int b = b_first + r;
    return (r < nblk && b < max_blocks) ? table[b] : 0;
  };
  auto checked = [&](int e) -> int { return (e < 0 || e >= num_blocks) ? 0 : e; };
  auto load_chunk = [&](int c) -> int { return checked(raw_chunk(c)); };
  int chunk = 0;
  const int raw0 = raw_chunk(0), raw1 = raw_chunk(1);
  int tab = checked(raw0);
  int tab_next = checked(raw1);
  const size_t head_off = (size_t)kvh * SLAB;
  // block b (0 <= b < 128) counted from the start of the current chunk
  auto block_off = [&](int b) -> size_t {
    const int e = b < 64 ? __builtin_amdgcn_readlane(tab, b)
                         : __builtin_amdgcn_readlane(tab_next, b - 64);
    return (size_t)e * hkv * SLAB + head_off;
  };

  f32x4 acc[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) acc[db] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m = -INFINITY;
  float lpart = 0.f;

  auto compute = [&](const DecodeFrag<D>& f, int t0) {
    const int nvalid = min(32, k1 - t0);
    f32x4 s0 = {0.f, 0.f, 0.f, 0.f}, s1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
      s0 = mfma16(as_bf16x8(f.k[0][kk]), qf[kk], s0);
      s1 = mfma16(as_bf16x8(f.k[1][kk]), qf[kk], s1);
    }
    // lane holds keys 4*grp + r (block 0) and 16 + 4*grp + r (block 1) of column col
    float sv[8];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      sv[r] = s0[r] * scale_log2;
      sv[4 + r] = s1[r] * scale_log2;
    }
    if (nvalid < 32) {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        sv[r] = 4 * grp + r < nvalid ? sv[r] : -INFINITY;
        sv[4 + r] = 16 + 4 * grp + r < nvalid ? sv[4 + r] : -INFINITY;
      }
    }
    float mx = fmaxf(fmaxf(fmaxf(sv[0], sv[1]), fmaxf(sv[2], sv[3])),
                     fmaxf(fmaxf(sv[4], sv[5]), fmaxf(sv[6], sv[7])));
    mx = wave_max16(mx);
    const float m_new = fmaxf(m, mx);
    const float alpha = fast_exp2(m - m_new);
    float pv[8];
    float ps = 0.f;
#pragma unroll
    for (int r = 0; r < 8; ++r) {
      pv[r] = fast_exp2(sv[r] - m_new);
      ps += pv[r];
    }
    lpart = lpart * alpha + ps;
    m = m_new;
    u32x4 pb;
    pb[0] = pack_bf16x2(pv[0], pv[1]);
    pb[1] = pack_bf16x2(pv[2], pv[3]);
    pb[2] = pack_bf16x2(pv[4], pv[5]);
    pb[3] = pack_bf16x2(pv[6], pv[7]);
    const bf16x8 pfrag = as_bf16x8(pb);
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      u32x2 va = f.v[0][db], vb = f.v[1][db];
      if (nvalid < 32) {
        va = mask_v4(va, 4 * grp, nvalid);
        vb = mask_v4(vb, 16 + 4 * grp, nvalid);
      }
      u32x4 vv = {va[0], va[1], vb[0], vb[1]};
      f32x4 c = acc[db];
#pragma unroll
      for (int r = 0; r < 4; ++r) c[r] *= alpha;
      acc[db] = mfma16(as_bf16x8(vv), pfrag, c);
    }
  };

  // two-stage register pipeline: the next step's loads are in flight while this one is
  // multiplied (the load after the last step reads stand-in blocks and is discarded)
  DecodeFrag<D> fa, fb;
  decode_load<D>(fa, k_cache, v_cache, block_off(0), block_off(1), col, grp);
  for (int t0 = k0, sb = 0;; t0 += 64, sb += 4) {
    if (sb == 64) {  // step into the next chunk of the table
      sb = 0;
      ++chunk;
      tab = tab_next;
      tab_next = load_chunk(chunk + 1);
    }
    decode_load<D>(fb, k_cache, v_cache, block_off(sb + 2), block_off(sb + 3), col, grp);
    compute(fa, t0);
    if (t0 + 32 >= k1) break;
    decode_load<D>(fa, k_cache, v_cache, block_off(sb + 4), block_off(sb + 5), col, grp);
    compute(fb, t0 + 32);
    if (t0 + 64 >= k1) break;
  }

  const float l = wave_sum16(lpart);
  if (!col_ok) return;
  if (nsplit == 1) {
    const float inv = 1.f / l;
    uint16_t* o = out + ((size_t)i * hq + h) * D;
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      u32x2 w = {pack_bf16x2(acc[db][0] * inv, acc[db][1] * inv),
                 pack_bf16x2(acc[db][2] * inv, acc[db][3] * inv)};
      st8(o + db * 16 + 4 * grp, w);
    }
    if (lse != nullptr && grp == 0) lse[(size_t)i * hq + h] = (m + log2f(l)) * kLn2;
    return;
  }
  const size_t slot = ((size_t)i * hq + h) * max_splits + sp;
  float* o = ws_o + slot * D;
#pragma unroll
  for (int db = 0; db < DB; ++db) {
    f32x4 c = acc[db];
    st16(o + db * 16 + 4 * grp, __builtin_bit_cast(u32x4, c));
  }
  if (grp == 0) {
    ws_ml[slot * 2 + 0] = m;
    ws_ml[slot * 2 + 1] = l;
  }
}

}  // namespace dec
}  // namespace pkv
