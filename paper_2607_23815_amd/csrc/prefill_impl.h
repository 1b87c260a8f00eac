// Prefix-reuse paged prefill attention for gfx950: the workgroup body, shared by the
// prefill launch and the mixed prefill + decode launch.
//
// A downstream operator's prefill computes attention only for its N new tokens; the keys are
// the sequence's cached prefix (left in the pool by the upstream operator) followed by the new
// tokens, all read through the block table. New token j sees keys 0 .. P + j.
//
// Work item = (sequence, kv head, tile of 32 x kWaves query columns). A column is one (new token,
// query head) pair of the kv head's group, token-major, so the g = Hq/Hkv heads that share
// the kv head are packed into the matrix-core M dimension and every K/V byte staged in LDS
// serves all of them. The workgroup has kWaves waves (4: two independent workgroups per
// compute unit overlap each other's stalls) of 32 columns each and walks the keys in tiles
// of 64 (four 16-token blocks):
//   1. K and V tiles are staged in LDS (double-buffered: the next tile's global loads are in
//      flight while the current tile is multiplied). Staging is a 16-byte copy of whole pool
//      slabs with a swizzle on the 16-byte unit index, so the matrix-core operand reads below
//      hit distinct LDS banks.
//   2. Scores S^T[64 keys][32 cols] = K . Q^T with v_mfma_f32_32x32x16_bf16; Q stays in
//      registers for the whole work item.
//   3. Online softmax in the base-2 domain (scale * log2 e folded in fp32). Each lane owns one
//      column, so the running max, sum and output rescale are lane-local except for one
//      exchange with the lane 32 apart that holds the column's other keys.
//   4. O^T[D][32 cols] += V^T . P^T, again 32x32x16, with P^T taken straight from the score
//      registers (rounded to bf16). For this to need no data movement, score row m of the
//      32-key half-tile is loaded with key sigma(m), sigma swapping bits 2 and 3 of the key
//      index; then the 8 keys a lane contributes to each value-product step are 8
//      consecutive slots, i.e. one 16-byte chunk of the dim-major V slab.
//   5. The normalised output rows leave through LDS (the K buffers, free after the last
//      step), so that each 16-byte store covers whole rows.
// A key split (only for batches too small to fill the chip, see prefill_split_plan) cuts
// an item's keys at multiples of split_keys: split s covers the key tiles of
// [s * split_keys, (s + 1) * split_keys). A row whose keys all fall in split 0 is finished
// there; any other row leaves one partial result (unnormalised output, running maximum and
// weight sum) per split it reaches, merged afterwards by their log-sum-exp weights. The cut
// points depend on key positions only, so results are deterministic.
// Masking is by selection (scores to -inf), applied only to tiles that reach past some
// column's last visible key; V slots past the sequence end are zeroed in LDS before the last
// tile's value product, so stale bits (NaN included) never meet a zero weight inside the
// matrix core.
#pragma once

#include <math.h>

#include <type_traits>

#include "device_utils.h"

namespace pkv {
namespace pre {

constexpr int kWaves = 4;             // waves per workgroup
constexpr int kThreads = 64 * kWaves;
constexpr int kCols = 32 * kWaves;    // query columns per workgroup (32 per wave)
constexpr int kSlabWaves = kWaves / 4;  // waves staging each of a tile's four block slabs
constexpr int kKeys = 64;   // keys per tile (4 blocks)

// Wait until every global load this thread issued has completed (vmcnt = 0; the other
// counters left at their maxima), so its direct-to-LDS loads have been written.
__device__ __forceinline__ void wait_vmem() { __builtin_amdgcn_s_waitcnt(0x0F70); }

// The value held by the lane 32 apart (lanes l and l ^ 32 hold the two key halves of one
// column): v_permlane32_swap exchanges the upper half of one register with the lower half of
// another, so swapping a register with a copy of itself gives every lane its partner's value.
__device__ __forceinline__ float swap_halves(float x) {
  const uint32_t u = __float_as_uint(x);
  const auto r = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  // lanes < 32 find the partner in the second result, lanes >= 32 in the first
  return __uint_as_float((threadIdx.x & 32) ? r[0] : r[1]);
}

// sigma: swap bits 2 and 3 of a key index within a 16-key block (an involution)
__device__ __forceinline__ int swap23(int s) {
  return (s & ~0xC) | ((s & 8) >> 1) | ((s & 4) << 1);
}

template <int D>
struct PrefillSmem {
  static constexpr int SLAB = D * kBlockSize;  // elements per block slab
  uint16_t k[2][4 * SLAB];
  uint16_t v[2][4 * SLAB];
};

// The matrix-core block of a step (below): fragments read this many matrix-core ops ahead,
// fences every kSub ops, three vector ops scheduled after each matrix-core op. Measured against
// 5 or 6 reads ahead, fences every 2 or 8 ops, 4 vector ops and no fences: equal within 0.5%
// or slower (2 ops per fence 1-2%, 4 vector ops 2-4%).
constexpr int kAhead = 4, kSub = 4, kValu = 3;

// Rescale the running output only when a column's maximum grows by more than this many
// powers of two; otherwise keep the stale maximum (weights then stay below 2^8, exact in the
// normalisation). After the first tiles the maximum of N(0,1) scores hardly moves, so the
// 64 accumulator multiplies per tile are almost always skipped.
constexpr float kRescaleThreshold = 8.0f;
constexpr float kRescaleLimit = 256.0f;  // 2^kRescaleThreshold

// ---- staging: direct global -> LDS 16-byte loads. Wave w stages block w % 4 of every
// tile, sharing it with the other kWaves / 4 - 1 waves of that block: its load k fills LDS
// units 64 (part * WLOADS + k) + lane of that block's slab (with four waves, the whole 4 KB
// slab at head_dim 128 in four loads). The bank swizzle is applied on the global side: LDS K
// unit c*16 + t holds global unit c*16 + swap23(t), LDS V unit 2d + t holds global unit
// 2d + (t ^ ((d >> 3) & 1)); with these, the 16 lanes the LDS serves per cycle read 16
// distinct 16-byte bank groups. ----
template <int D>
struct Staging {
  static constexpr int SLAB = D * kBlockSize;          // elements per block slab
  static constexpr int UNITS = SLAB / 8;               // 16-byte units per block slab
  static constexpr int WLOADS = UNITS / 64 / kSlabWaves;  // loads per wave per block slab
  int slab, part;  // the block of a tile this wave stages; its share of it
  // Per-lane element offsets of load 0 within a block slab; load k reads 512 k elements
  // further on (the swizzles act within 64-unit groups), so two registers serve every load.
  int kofs, vofs;
  __device__ __forceinline__ Staging(int wave, int lane) : slab(wave & 3), part(wave >> 2) {
    const int pos = part * WLOADS * 64 + lane;
    const int c = pos >> 4;
    kofs = (c * 16 + swap23(pos & 15)) * 8;
    const int d = pos >> 1;
    vofs = (2 * d + ((pos & 1) ^ ((d >> 3) & 1))) * 8;
  }
  template <int K>
  __device__ __forceinline__ void issue_load(const uint16_t* src, uint16_t* dst, int ofs) const {
    lds_load16(src, SLAB * 2, (ofs + K * 512) * 2, dst + slab * SLAB + (part * WLOADS + K) * 512);
    if constexpr (K + 1 < WLOADS) issue_load<K + 1>(src, dst, ofs);
  }
  // This wave's share of block `blk` (kv head `kvh`) into the tile buffer `dst`, with offsets
  // `ofs` (kofs or vofs). One slab = one buffer resource (base = the slab, 4 KB,
  // bounds-checked by the hardware).
  __device__ __forceinline__ void issue(const uint16_t* cache, uint16_t* dst, int ofs, int blk,
                                        int hkv, int kvh) const {
    issue_load<0>(cache + ((size_t)blk * hkv + kvh) * SLAB, dst, ofs);
  }
};

// Q as the B operand of S^T = K Q^T: lane (lc, hh) of wave `wave` holds column
// qt * kCols + 32 wave + lc, dims 16 kk + 8 hh .. +7. A lane past the last column reads a
// valid row (token n - 1); the caller zeroes it before use.
template <int D>
__device__ __forceinline__ void load_q(const uint16_t* __restrict__ q, int hq, int hkv, int kvh,
                                       int qt, int row0, int n, int wave, int lane,
                                       bf16x8 (&qf)[D / 16]) {
  const int g = hq / hkv;
  const int gcol = qt * kCols + wave * 32 + (lane & 31);
  const int j = gcol < n * g ? gcol / g : n - 1;
  const int head = kvh * g + gcol % g;
  const uint16_t* qrow = q + ((size_t)(row0 + j) * hq + head) * D + (lane >> 5) * 8;
#pragma unroll
  for (int kk = 0; kk < D / 16; ++kk) qf[kk] = as_bf16x8(ld16(qrow + kk * 16));
}

// One work item: query tile qt (columns qt * kCols ..) of the (sequence i, kv head kvh)
// group, whose cached prefix is p tokens and whose n new tokens start at row row0 of q and
// out. t_first and t_lane are entry 0 and entry `lane` of the sequence's block-table row
// (-1 past the row).
template <int D>
__device__ __forceinline__ void prefill_item(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k_cache,
    const uint16_t* __restrict__ v_cache, const int32_t* __restrict__ block_tables,
    int32_t max_blocks, int32_t hq, int32_t hkv, int32_t num_blocks, float scale_log2,
    uint16_t* __restrict__ out, float* __restrict__ lse, const int i, const int kvh,
    const int qt, const int p, const int row0, const int n, const int32_t t_first,
    const int32_t t_lane, PrefillSmem<D>& sm, const int split_keys = 0, const int split = 0,
    const int nsplit = 1, float* __restrict__ ws_o = nullptr,
    float* __restrict__ ws_ml = nullptr) {
  constexpr int SLAB = D * kBlockSize;
  constexpr int UNITS = SLAB / 8;        // 16-byte units per block slab
  constexpr int LPT = 4 * UNITS / kThreads;  // 16-byte units per thread per tile (K or V)
  constexpr int KK = D / 16;             // k-steps of the score product
  constexpr int DB = D / 32;             // 32-dim blocks of the value product

  const int32_t* table = block_tables + (size_t)i * max_blocks;
  const int g = hq / hkv;
  const int ncols = n * g;
  const int col0 = qt * kCols;
  const int len = p + n;

  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform
  const int lane = tid & 63;
  const int lc = lane & 31;
  const int hh = lane >> 5;

  const int gcol = col0 + wave * 32 + lc;
  const bool col_ok = gcol < ncols;
  const int j = col_ok ? gcol / g : n - 1;
  const int lim = p + j;  // last key this column sees
  const int lim_h = lim - 8 * hh;  // the same, less the lane's key offset within a block

  const int jmax = min(n - 1, (col0 + kCols - 1) / g);
  const int nkeys = p + jmax + 1;
  const int ntiles = (nkeys + kKeys - 1) / kKeys;
  // this item's key tiles [kt0, kt_end): all of them, or one split (split_keys is a multiple
  // of 1024 keys, so a split starts at a table chunk and on an even tile)
  const int kt0 = split_keys > 0 ? split * (split_keys / kKeys) : 0;
  const int kt_end = split_keys > 0 ? min(ntiles, kt0 + split_keys / kKeys) : ntiles;
  if (split_keys > 0 && kt0 >= kt_end) return;  // (workgroup-uniform) an empty split
  const int nt = kt_end - kt0;
  const int wcol0 = col0 + wave * 32;
  const int wj_lo = min(wcol0 / g, n - 1);         // earliest token among the wave's columns
  const bool wave_live = wcol0 < ncols;            // the wave has at least one real column

  f32x16 o[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[db][r] = 0.f;
  float m = -INFINITY;
  float lpart = 0.f;
  bf16x8 qf[KK];  // Q fragments, loaded in the prologue

  // stand-in for blocks past the sequence: its first block (len >= 1, so it owns one)
  const int32_t blk_first = (t_first >= 0 && t_first < num_blocks) ? t_first : 0;
  const Staging<D> st(wave, lane);
  const int slab = st.slab;

  // Block-table entries through a per-wave register table: lane l of a chunk holds entry
  // 64 c + l, already checked (entries past the sequence, past the table or out of the pool
  // are replaced by the sequence's first block: finite data, masked or zeroed before use).
  // A chunk covers 16 tiles; the K and V streams keep one chunk each.
  auto load_chunk = [&](int c) {
    const int e = c * 64 + lane;
    int v = blk_first;
    if (e < max_blocks && e * kBlockSize < len) {
      const int t = table[e];
      v = (t >= 0 && t < num_blocks) ? t : blk_first;
    }
    return v;
  };
  int kchunk = (lane * kBlockSize < len && t_lane >= 0 && t_lane < num_blocks) ? t_lane
                                                                              : blk_first;
  int kchunk_id = 0;
  int vchunk = kchunk, vchunk_id = 0;
  auto block_of = [&](int& chunk, int& chunk_id, int kt) {
    const int e = kt * 4 + slab;  // the block of tile kt this wave stages
    const int c = e >> 6;
    if (c != chunk_id) {
      chunk = load_chunk(c);
      chunk_id = c;
    }
    return __builtin_amdgcn_readlane(chunk, e & 63);
  };
  // One slab = one buffer resource (base = the slab, 4 KB, bounds-checked by the hardware).
  auto issue_k = [&](int kt, int buf) {
    st.issue(k_cache, sm.k[buf], st.kofs, block_of(kchunk, kchunk_id, kt), hkv, kvh);
  };
  auto issue_v = [&](int kt, int buf) {
    st.issue(v_cache, sm.v[buf], st.vofs, block_of(vchunk, vchunk_id, kt), hkv, kvh);
  };

  // lane-constant LDS read offsets (elements)
  const int kread = (lc >> 4) * SLAB + (hh * 16 + (lc & 15)) * 8;
  const int vread = (2 * lc + (hh ^ ((lc >> 3) & 1))) * 8;

  // register r of half-tile beta holds the score of key
  // key0 + 32 beta + 16 (r/8) + 8 hh + 4 ((r/4) % 2) + r % 4
  // (compared as a compile-time offset against lim - key0 - 8 hh, so no per-register key
  // positions are kept live)
  auto mask_tile = [&](int key0, f32x16 (&sc)[2]) {
    const int d = lim_h - key0;
#pragma unroll
    for (int beta = 0; beta < 2; ++beta)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int c = 32 * beta + 16 * (r >> 3) + 4 * ((r >> 2) & 1) + (r & 3);
        sc[beta][r] = c <= d ? sc[beta][r] : -INFINITY;
      }
  };

  // weights of one tile outside the block (after a rescale, and on an item's first tile):
  // the same arithmetic as the block's softmax slices, in the same order
  auto weights = [&](f32x16 (&sc)[2], bf16x8 (&pw)[2][2]) {
    const float neg_m = -m;
    float sum[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int beta = 0; beta < 2; ++beta)
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        u32x4 w;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float a = fast_exp2(__builtin_fmaf(sc[beta][8 * u + 2 * e], scale_log2, neg_m));
          const float b = fast_exp2(__builtin_fmaf(sc[beta][8 * u + 2 * e + 1], scale_log2, neg_m));
          w[e] = pack_bf16x2(a, b);
          sum[2 * e] += a;
          sum[2 * e + 1] += b;
        }
        pw[beta][u] = as_bf16x8(w);
      }
    return ((sum[0] + sum[1]) + (sum[2] + sum[3])) + ((sum[4] + sum[5]) + (sum[6] + sum[7]));
  };
  // The matrix-core work of a step as fenced sub-blocks of kSub ops each: the score products
  // S^T = K Q^T of the K tile in buffer kbuf (when QK; op t < NQ reads K fragment (kk, beta) =
  // (t / 2, t % 2), both 32-key halves as two independent chains), then the value products
  // O^T += V^T P^T of the V tile in buffer vbuf with the weights pw (when PV; op NQ + f reads
  // V fragment f = (beta, u, db) in that nesting: step (beta, u) covers block 2 beta + u of
  // the tile, lane group hh supplying slots 8 hh .. 8 hh + 7 of V^T row 32 db + lc). 32 ops
  // in a steady-state step at head dim 128, 16 at 64. Fragments sit in an 8-entry register
  // ring and are read kAhead ops ahead (the first kAhead by the caller unless PRE), so every
  // op finds its operand landed; the fences keep the compiler from reordering ops against
  // their reads. With SM the sixteen slices of the softmax of the scores in cur are spread
  // evenly over the sub-blocks (kValu vector ops after each matrix-core op): weights
  // P = 2^(scale_log2 * S - m) rounded to bf16 into pcur, and the sums of the fp32 weights
  // before rounding in eight independent partial sums (each rounded weight is within a
  // relative 2^-9 of its fp32 value, unbiased; a single accumulator would chain dependent
  // adds through the block).
  using yes_t = std::true_type;
  using no_t = std::false_type;
  auto frag = [&](auto nq, int t, int kbuf, int vbuf) -> u32x4 {
    constexpr int NQ = decltype(nq)::value;
    if (t < NQ) {
      const int kk = t >> 1, beta = t & 1;
      return ld16(&sm.k[kbuf][kread + beta * 2 * SLAB + kk * 256]);
    }
    const int f = t - NQ;
    const int beta = f / (2 * DB), u = (f / DB) & 1, db = f % DB;
    return ld16(&sm.v[vbuf][(2 * beta + u) * SLAB + vread + db * 512]);
  };
  auto block = [&](auto qk, auto pv, auto smx, auto pre, int kbuf, int vbuf, u32x4 (&fr)[8],
                   f32x16 (&sc)[2], const bf16x8 (&pw)[2][2], const f32x16 (&cur)[2],
                   bf16x8 (&pcur)[2][2], float (&sum)[8]) {
    constexpr bool QK = decltype(qk)::value, PV = decltype(pv)::value;
    constexpr bool SM = decltype(smx)::value, PRE = decltype(pre)::value;
    constexpr int NQ = QK ? 2 * KK : 0;
    constexpr int NOPS = NQ + (PV ? 4 * DB : 0);
    constexpr int NSUB = NOPS / kSub;
    constexpr int SLICES = SM ? 16 / NSUB : 0;  // softmax slices per sub-block
    static_assert(NOPS % kSub == 0 && NOPS > kAhead && kAhead < 8 && (!SM || 16 % NSUB == 0),
                  "block shape");
    using nq_t = std::integral_constant<int, NQ>;
    if constexpr (PRE) {
#pragma unroll
      for (int t = 0; t < kAhead; ++t) fr[t] = frag(nq_t(), t, kbuf, vbuf);
    }
    const float neg_m = -m;
    u32x4 w[2][2];
#pragma unroll
    for (int s = 0; s < NSUB; ++s) {
#pragma unroll
      for (int k = 0; k < kSub; ++k) {
        const int t = kSub * s + k;
        if (t + kAhead < NOPS) fr[(t + kAhead) & 7] = frag(nq_t(), t + kAhead, kbuf, vbuf);
        if (t < NQ) {
          const int kk = t >> 1, beta = t & 1;
          sc[beta] = mfma32(as_bf16x8(fr[t & 7]), qf[kk], sc[beta]);
        } else {
          const int f = t - NQ;
          const int beta = f / (2 * DB), u = (f / DB) & 1, db = f % DB;
          o[db] = mfma32(as_bf16x8(fr[t & 7]), pw[beta][u], o[db]);
        }
      }
#pragma unroll
      for (int h = 0; h < SLICES; ++h) {
        const int it = SLICES * s + h;  // softmax slice (beta, u, e)
        const int beta = it >> 3, u = (it >> 2) & 1, e = it & 3;
        const float a = fast_exp2(__builtin_fmaf(cur[beta][8 * u + 2 * e], scale_log2, neg_m));
        const float b = fast_exp2(__builtin_fmaf(cur[beta][8 * u + 2 * e + 1], scale_log2, neg_m));
        w[beta][u][e] = pack_bf16x2(a, b);
        asm volatile("" ::"v"(w[beta][u][e]));  // the pack stays in this sub-block
        sum[2 * e] += a;
        sum[2 * e + 1] += b;
      }
#pragma unroll
      for (int k = 0; k < kSub; ++k) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // 1 MFMA
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // 1 LDS read
        if constexpr (SM) __builtin_amdgcn_sched_group_barrier(0x002, kValu, 0);  // vector ops
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    if constexpr (SM) {
#pragma unroll
      for (int beta = 0; beta < 2; ++beta)
#pragma unroll
        for (int u = 0; u < 2; ++u) pcur[beta][u] = as_bf16x8(w[beta][u]);
    }
  };
  auto zero_scores = [&](f32x16 (&sc)[2]) {
#pragma unroll
    for (int beta = 0; beta < 2; ++beta)
#pragma unroll
      for (int r = 0; r < 16; ++r) sc[beta][r] = 0.f;
  };

  // One step of the software pipeline, for tile kt. On entry cur holds the raw scores of
  // tile kt and pprev the weights of tile kt-1 (when has_prev). One straight-line block
  // then issues the score MFMAs of tile kt+1 (when has_next) and the value MFMAs of tile
  // kt-1 (when has_prev), interleaved with the softmax of tile kt, whose weights use the
  // running maximum m speculatively: with the lazy rescale m almost never moves, and when
  // some column's maximum does grow by more than the threshold a rare branch rescales the
  // accumulator and recomputes the weights. On the item's first tile (no has_prev) m is still
  // -inf: the block only issues the next tile's score products, and the weights follow the
  // maximum.
  // LDS: step kt reads K(kt+1) from K buffer (kt+1)&1 and V(kt-1) from V buffer (kt-1)&1,
  // and loads K(kt+2) into K buffer kt&1 and V(kt) into V buffer kt&1 -- the buffers whose
  // last readers were in step kt-1, which the barrier at the top of step kt has retired
  // (V(0) is loaded by the prologue, whose buffers are all free).
  auto step = [&](auto has_prev, auto has_next, int kt, f32x16 (&cur)[2], f32x16 (&nxt)[2],
                  bf16x8 (&pprev)[2][2], bf16x8 (&pcur)[2][2]) {
    wait_vmem();
    __syncthreads();  // K(kt+1) and V(kt-1) have landed; all waves are done with step kt-1
    constexpr bool HN = decltype(has_next)::value, HP = decltype(has_prev)::value;
    using nq_t = std::integral_constant<int, HN ? 2 * KK : 0>;
    u32x4 fr[8];
    if constexpr (HN || HP) {
      // the block's first fragments, ahead of the staging issue
      if (wave_live) {
#pragma unroll
        for (int t = 0; t < kAhead; ++t) fr[t] = frag(nq_t(), t, (kt + 1) & 1, (kt - 1) & 1);
      }
    }
    if (kt + 2 < kt_end) issue_k(kt + 2, kt & 1);
    if constexpr (HP) issue_v(kt, kt & 1);  // V(0): prologue
    if (!wave_live) return;
    const int key0 = kt * kKeys;
    if (key0 + kKeys - 1 > p + wj_lo) mask_tile(key0, cur);

    // ---- the straight-line block ----
    // (at a raised wave priority: when both waves on a SIMD can issue, the one in its block of
    // matrix-core work goes first; 1-1.6% faster on the Llama-3-8B and 70B-shaped layers)
    __builtin_amdgcn_s_setprio(2);
    float lnew = 0.f;
    float sum[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    if constexpr (HN) zero_scores(nxt);
    if constexpr (HP) {
      block(has_next, yes_t(), yes_t(), no_t(), (kt + 1) & 1, (kt - 1) & 1, fr, nxt, pprev,
            cur, pcur, sum);
      lnew = ((sum[0] + sum[1]) + (sum[2] + sum[3])) + ((sum[4] + sum[5]) + (sum[6] + sum[7]));
    } else {
      // the item's first tile: the running maximum is still -inf, so its weights are computed
      // below, after the maximum; until then they are zero
      if constexpr (HN)
        block(yes_t(), no_t(), no_t(), no_t(), (kt + 1) & 1, 0, fr, nxt, pprev, cur, pcur, sum);
      const u32x4 zero = {0u, 0u, 0u, 0u};
#pragma unroll
      for (int beta = 0; beta < 2; ++beta)
#pragma unroll
        for (int u = 0; u < 2; ++u) pcur[beta][u] = as_bf16x8(zero);
    }
    // keep the speculative weights in this block: without a use here the compiler would sink
    // their computation past the rare branch below (which overwrites them), out of reach of
    // the interleave
    asm volatile("" ::"v"(__builtin_bit_cast(u32x4, pcur[0][0])),
                 "v"(__builtin_bit_cast(u32x4, pcur[0][1])),
                 "v"(__builtin_bit_cast(u32x4, pcur[1][0])),
                 "v"(__builtin_bit_cast(u32x4, pcur[1][1])), "v"(lnew));
    __builtin_amdgcn_s_setprio(0);
    // The running maximum only has to move when some weight of the tile exceeds 2^threshold,
    // and then this lane's (non-negative) weight sum exceeds it too: test the sum, and only
    // then find the tile's exact maximum (the first tile, where m = -inf, always does).
    bool check = true;
    if constexpr (decltype(has_prev)::value)
      check = __builtin_amdgcn_ballot_w64(!(lnew <= kRescaleLimit)) != 0;
    if (check) {
      float mx = -INFINITY;
#pragma unroll
      for (int beta = 0; beta < 2; ++beta)
#pragma unroll
        for (int r = 0; r < 16; ++r) mx = fmaxf(mx, cur[beta][r]);
      mx = fmaxf(mx, swap_halves(mx)) * scale_log2;
      const bool grow = mx > m + kRescaleThreshold;
      if (__builtin_amdgcn_ballot_w64(grow)) {
        const float m_new = grow ? mx : m;
        const float alpha = fast_exp2(m - m_new);
        m = m_new;
        lpart *= alpha;
#pragma unroll
        for (int db = 0; db < DB; ++db)
#pragma unroll
          for (int r = 0; r < 16; ++r) o[db][r] *= alpha;
        lnew = weights(cur, pcur);
      }
    }
    lpart += lnew;
  };

  // prologue: K(kt0), K(kt0+1) and V(kt0) (every buffer is free; their blocks are entries
  // 0..7 of the item's first chunk), then Q, all under one wait; scores of tile kt0
  if (kt0 > 0) {
    kchunk_id = vchunk_id = kt0 / 16;
    kchunk = vchunk = load_chunk(kchunk_id);
  }
  st.issue(k_cache, sm.k[0], st.kofs, __builtin_amdgcn_readlane(kchunk, slab), hkv, kvh);
  if (nt > 1)
    st.issue(k_cache, sm.k[1], st.kofs, __builtin_amdgcn_readlane(kchunk, 4 + slab), hkv, kvh);
  st.issue(v_cache, sm.v[0], st.vofs, __builtin_amdgcn_readlane(kchunk, slab), hkv, kvh);
  // Q fragments; a lane past the last column computes with zeros
  load_q<D>(q, hq, hkv, kvh, qt, row0, n, wave, lane, qf);
#pragma unroll
  for (int kk = 0; kk < KK; ++kk) {
    const u32x4 zero = {0u, 0u, 0u, 0u};
    qf[kk] = col_ok ? qf[kk] : as_bf16x8(zero);
  }
  wait_vmem();
  __syncthreads();
  f32x16 sa[2], sb[2];
  bf16x8 pa[2][2], pb[2][2];
  if (wave_live) {
    u32x4 fr[8];
    float sum[8];
    zero_scores(sa);
    block(yes_t(), no_t(), no_t(), yes_t(), 0, 0, fr, sa, pa, sb, pb, sum);
  }
  using yes = std::true_type;
  using no = std::false_type;
  // step kt consumes scores sa/sb alternately and writes weights pa/pb alternately
  if (nt == 1) {
    step(no(), no(), kt0, sa, sb, pb, pa);
  } else {
    step(no(), yes(), kt0, sa, sb, pb, pa);
    int kt = kt0 + 1;
    for (; kt + 2 < kt_end; kt += 2) {
      step(yes(), yes(), kt, sb, sa, pa, pb);
      step(yes(), yes(), kt + 1, sa, sb, pb, pa);
    }
    if (kt + 1 < kt_end) {
      step(yes(), yes(), kt, sb, sa, pa, pb);
      step(yes(), no(), kt + 1, sa, sb, pb, pa);
      kt += 2;
    } else {
      step(yes(), no(), kt, sb, sa, pa, pb);
      kt += 1;
    }
    (void)kt;
  }
  // epilogue: V of the last tile (loaded by the last step) lands; where that tile reaches
  // past the sequence, zero the V slots >= len (they may hold any bits); then its value
  // product, with the weights in pa when nt is odd and in pb when it is even
  {
    const int kt = kt_end - 1;
    wait_vmem();
    __syncthreads();
    if ((kt + 1) * kKeys > len) {
      uint16_t* vt = sm.v[kt & 1];
#pragma unroll
      for (int k = 0; k < LPT; ++k) {
        const int P = tid + kThreads * k;
        const int bb = P / UNITS, pos = P % UNITS;
        const int d = pos >> 1;
        const int hf = (pos & 1) ^ ((d >> 3) & 1);
        const int first = kt * kKeys + bb * kBlockSize + hf * 8;
        const int keep = min(max(len - first, 0), 8);
        if (keep < 8) {
          u32x4 w = ld16(&vt[P * 8]);
          uint32_t words[4] = {w[0], w[1], w[2], w[3]};
#pragma unroll
          for (int e = 0; e < 8; ++e)
            if (e >= keep) words[e >> 1] &= (e & 1) ? 0x0000FFFFu : 0xFFFF0000u;
          st16(&vt[P * 8], u32x4{words[0], words[1], words[2], words[3]});
        }
      }
      __syncthreads();
    }
    if (wave_live) {
      u32x4 fr[8];
      float sum[8];
      if (nt & 1) block(no_t(), yes_t(), no_t(), yes_t(), 0, kt & 1, fr, sa, pa, sb, pb, sum);
      else block(no_t(), yes_t(), no_t(), yes_t(), 0, kt & 1, fr, sa, pb, sb, pa, sum);
    }
  }

  const float l = lpart + swap_halves(lpart);
  if (!wave_live) return;
  // The wave's 32 output rows go out through LDS as whole rows, with non-temporal stores (so
  // that no dirty lines of the output are left for later work to write back; a launch's output
  // is mostly larger than the memory-side cache anyway): a lane holds 8-byte pieces
  // of one row (column), so storing them directly would put 32 rows into every store
  // instruction; written to LDS first (the K buffers, free since the last step's barrier:
  // 32 rows x D per wave), each 16-byte store below covers 64 / (D / 8) complete rows.
  // 16-byte unit u of row r sits at unit u ^ (r % (D / 8)), so that both the 8-byte writes
  // (32 rows at once) and the 16-byte reads (whole rows) spread over all LDS banks.
  constexpr int CH = D / 8;    // 16-byte units per row
  constexpr int RPI = 64 / CH; // rows per store instruction
  uint16_t* tile = &sm.k[0][0] + wave * 32 * D;
  // the lane index afresh (an opaque copy), so that no value derived from it for this block
  // is computed ahead of the step loop and kept live through it
  int ln;
  asm volatile("v_and_b32 %0, 63, %1" : "=v"(ln) : "v"((int)threadIdx.x));
  const int lcl = ln & 31, hhl = ln >> 5;
  if (split_keys > 0) {
    // rows that reach past split 0 leave this split's partial result (when they reach into
    // it): the unnormalised output, the running maximum and the weight sum
    const int gcp = wcol0 + lcl;
    const int jp = gcp / g;
    if (gcp < ncols && p + jp >= split_keys && p + jp >= kt0 * kKeys) {
      const size_t slot =
          ((size_t)(row0 + jp) * hq + kvh * g + gcp % g) * (size_t)nsplit + (size_t)split;
      float* wo = ws_o + slot * D + 4 * hhl;
#pragma unroll
      for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int a = 0; a < 4; ++a)
          st16(wo + 32 * db + 8 * a,
               u32x4{__float_as_uint(o[db][4 * a + 0]), __float_as_uint(o[db][4 * a + 1]),
                     __float_as_uint(o[db][4 * a + 2]), __float_as_uint(o[db][4 * a + 3])});
      if (hhl == 0) {
        ws_ml[slot * 2 + 0] = m;
        ws_ml[slot * 2 + 1] = l;
      }
    }
    if (split > 0) return;  // only split 0 holds rows that end in it
  }
  // rows that end in this item: every row without a split, and the rows of split 0 whose
  // keys all fall in it (gc: a column of the item)
  auto row_ends_here = [&](int gc) { return split_keys == 0 || p + gc / g < split_keys; };
  {
    const float inv = 1.f / l;  // columns past the end: any value, never stored
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int a = 0; a < 4; ++a) {
        // registers 4a .. 4a+3 hold dims 32 db + 8 a + 4 hh + 0..3
        u32x2 w = {pack_bf16x2(o[db][4 * a + 0] * inv, o[db][4 * a + 1] * inv),
                   pack_bf16x2(o[db][4 * a + 2] * inv, o[db][4 * a + 3] * inv)};
        const int u = (4 * db + a) ^ (lcl % CH);
        st8(tile + lcl * D + u * 8 + 4 * hhl, w);
      }
  }
#pragma unroll
  for (int k = 0; k < 32 / RPI; ++k) {
    const int r = k * RPI + ln / CH;  // the row (wave column) this lane stores a unit of
    const int u = ln % CH;
    const u32x4 v = ld16(tile + r * D + ((u ^ (r % CH)) * 8));
    const int gc = wcol0 + r;
    if (gc < ncols && row_ends_here(gc)) {
      const int jr = gc / g;
      st16_nt(out + ((size_t)(row0 + jr) * hq + kvh * g + gc % g) * D + u * 8, v);
    }
  }
  const int gcl = wcol0 + lcl;  // this lane's column, recomputed like the lane index
  if (lse != nullptr && hhl == 0 && gcl < ncols && row_ends_here(gcl))
    lse[(size_t)(row0 + gcl / g) * hq + kvh * g + gcl % g] = (m + log2f(l)) * kLn2;
}

// The body of one prefill workgroup of a one-item-per-workgroup launch (the mixed launch);
// `wg` is its index in the launch's work list.
template <int D>
__device__ __forceinline__ void prefill_body(const uint16_t* __restrict__ q, const uint16_t* __restrict__ k_cache,
                    const uint16_t* __restrict__ v_cache, const int32_t* __restrict__ block_tables,
                    int32_t max_blocks, const int32_t* __restrict__ cached_lens,
                    const int32_t* __restrict__ cu_new_lens, int32_t num_seqs, int32_t hq,
                    int32_t hkv, int32_t num_blocks, int32_t qtiles, float scale_log2,
                    uint16_t* __restrict__ out, float* __restrict__ lse, const unsigned wg,
                    int32_t split_keys = 0, int32_t nsplit = 1, float* __restrict__ ws_o = nullptr,
                    float* __restrict__ ws_ml = nullptr,
                    const int32_t* __restrict__ order = nullptr) {
  __shared__ __align__(16) PrefillSmem<D> sm;
  // XCD-aware mapping: workgroup id b runs on XCD b % 8 (a mixed launch passes a `wg` with
  // the same residue mod 8 as its workgroup id). The unit that must stay on one XCD
  // is a (sequence, kv head) group -- its query tiles read the same K/V and share that XCD's
  // L2 when they run together -- so groups are dealt to XCDs round-robin (group index mod 8)
  // and each XCD walks its groups in order. With 8 kv heads every XCD receives one kv head of
  // every sequence: equal work per XCD, whatever the lengths.
  // Within a group the query tiles go longest (last) first, rotated by the group's place in
  // the XCD's list: an XCD hands its workgroups to its shader engines in a fixed rotation,
  // and without the rotation slot s of every group -- and with it the low tiles, the ones
  // every sequence has -- would always land on the same engine, which then fills first and
  // stalls the rotation while the others have free slots.
  // With a key split a group holds qtiles x nsplit items: each query tile's splits follow
  // one another in the list.
  const int per = qtiles * nsplit;         // items per group
  const int xcd = wg & 7;
  const int pos = wg >> 3;                 // position in this XCD's list
  const int gpos = pos / per;              // the group's place in this XCD's list
  const int group = gpos * 8 + xcd;        // (sequence, kv head) group index
  const int idx = (pos % per + gpos) % per;
  const int qt = qtiles - 1 - idx / nsplit;
  const int sp = idx % nsplit;
  if (group >= num_seqs * hkv) return;
  const int kvh = group % hkv;
  // with an order, group ranks map to sequences longest first
  const int i = order != nullptr ? order[group / hkv] : group / hkv;
  // The first table chunk (entry `lane` of the sequence's row, and entry 0) is fetched
  // before the lengths: its address depends on the sequence only, so the two loads overlap.
  const int32_t* table = block_tables + (size_t)i * max_blocks;
  const int32_t t_first = table[0];
  const int32_t t_lane = (int)(threadIdx.x & 63) < max_blocks ? table[threadIdx.x & 63] : -1;
  const int p = cached_lens[i];
  const int row0 = cu_new_lens[i];
  const int n = cu_new_lens[i + 1] - row0;
  if (qt * kCols >= n * (hq / hkv)) return;
  prefill_item<D>(q, k_cache, v_cache, block_tables, max_blocks, hq, hkv, num_blocks, scale_log2,
                  out, lse, i, kvh, qt, p, row0, n, t_first, t_lane, sm, split_keys, sp, nsplit,
                  ws_o, ws_ml);
}

// The work list of a prefill batch: query tiles per (sequence, kv head) group, and the
// number of workgroups (the groups dealt to 8 XCD lists of equal length, qtiles x nsplit
// each).
struct PrefillGrid {
  int64_t qtiles;
  int64_t items;
};
inline PrefillGrid prefill_grid(int32_t hq, int32_t hkv, int32_t num_seqs, int32_t max_new_len,
                                int32_t nsplit = 1) {
  const int32_t g = hq / hkv;
  const int64_t qtiles = ((int64_t)max_new_len * g + kCols - 1) / kCols;
  const int64_t groups = (int64_t)hkv * num_seqs;
  return PrefillGrid{qtiles, (groups + 7) / 8 * 8 * qtiles * nsplit};
}

}  // namespace pre
}  // namespace pkv
