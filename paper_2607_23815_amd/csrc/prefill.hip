// Prefix-reuse paged prefill attention for gfx950.
//
// A downstream operator's prefill computes attention only for its N new tokens; the keys are
// the sequence's cached prefix (left in the pool by the upstream operator) followed by the new
// tokens, all read through the block table. New token j sees keys 0 .. P + j.
//
// Work item = (sequence, kv head, tile of 128 query columns). A column is one (new token,
// query head) pair of the kv head's group, token-major, so the g = Hq/Hkv heads that share
// the kv head are packed into the matrix-core M dimension and every K/V byte staged in LDS
// serves all of them. The workgroup has four waves of 32 columns each and walks the keys in
// tiles of 64 (four 16-token blocks):
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
// Masking is by selection (scores to -inf), applied only to tiles that reach past some
// column's last visible key; V slots past the sequence end are zeroed while staging, so stale
// bits (NaN included) never meet a zero weight inside the matrix core.
#include <math.h>

#include "device_utils.h"
#include "launch.h"

namespace pkv {
namespace {

constexpr int kCols = 128;  // query columns per workgroup (4 waves x 32)
constexpr int kKeys = 64;   // keys per tile (4 blocks)

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

template <int D>
__global__ __launch_bounds__(256) void prefill_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k_cache,
    const uint16_t* __restrict__ v_cache, const int32_t* __restrict__ block_tables,
    int32_t max_blocks, const int32_t* __restrict__ cached_lens,
    const int32_t* __restrict__ cu_new_lens, int32_t hq, int32_t hkv, int32_t num_blocks,
    float scale_log2, uint16_t* __restrict__ out, float* __restrict__ lse) {
  constexpr int SLAB = D * kBlockSize;
  constexpr int UNITS = 4 * SLAB / 8;   // 16-byte units per K (or V) tile
  constexpr int LPT = UNITS / 256;      // units per thread per tile
  constexpr int KK = D / 16;            // k-steps of the score product
  constexpr int DB = D / 32;            // 32-dim blocks of the value product
  __shared__ __align__(16) PrefillSmem<D> sm;

  const int g = hq / hkv;
  const int qt = (int)(gridDim.x - 1 - blockIdx.x);  // last (longest) query tiles first
  const int kvh = blockIdx.y;
  const int i = blockIdx.z;
  const int p = cached_lens[i];
  const int row0 = cu_new_lens[i];
  const int n = cu_new_lens[i + 1] - row0;
  const int ncols = n * g;
  const int col0 = qt * kCols;
  if (col0 >= ncols) return;
  const int len = p + n;

  const int tid = threadIdx.x;
  const int wave = tid >> 6;
  const int lane = tid & 63;
  const int lc = lane & 31;
  const int hh = lane >> 5;

  const int gcol = col0 + wave * 32 + lc;
  const bool col_ok = gcol < ncols;
  const int j = col_ok ? gcol / g : n - 1;
  const int head = kvh * g + gcol % g;
  const int lim = p + j;  // last key this column sees

  const int jmax = min(n - 1, (col0 + kCols - 1) / g);
  const int nkeys = p + jmax + 1;
  const int ntiles = (nkeys + kKeys - 1) / kKeys;
  const int wcol0 = col0 + wave * 32;
  const int wj_lo = min(wcol0 / g, n - 1);        // earliest token among the wave's columns
  const int wj_hi = min((wcol0 + 31) / g, n - 1); // latest
  const bool wave_live = wcol0 < ncols;            // the wave has at least one real column

  // Q as the B operand of S^T = K Q^T: lane holds Q[column lc][16 kk + 8 hh .. +7]
  bf16x8 qf[KK];
  {
    const uint16_t* qrow = q + ((size_t)(row0 + j) * hq + head) * D + hh * 8;
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
      u32x4 v = {0u, 0u, 0u, 0u};
      if (col_ok) v = ld16(qrow + kk * 16);
      qf[kk] = as_bf16x8(v);
    }
  }

  f32x16 o[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[db][r] = 0.f;
  float m = -INFINITY;
  float lpart = 0.f;

  const int32_t* table = block_tables + (size_t)i * max_blocks;
  const size_t head_off = (size_t)kvh * SLAB;

  // ---- staging: thread tid moves units tid + 256 k of the K tile and of the V tile ----
  u32x4 kreg[LPT], vreg[LPT];
  auto load_tile = [&](int kt) {
#pragma unroll
    for (int k = 0; k < LPT; ++k) {
      const int u = tid + 256 * k;
      const int bb = u / (SLAB / 8);   // block within the tile
      const int w = u % (SLAB / 8);    // unit within the block slab
      const int b = kt * 4 + bb;       // logical block
      u32x4 kv = {0u, 0u, 0u, 0u}, vv = {0u, 0u, 0u, 0u};
      if (b * kBlockSize < len && b < max_blocks) {
        const int blk = table[b];
        if (blk >= 0 && blk < num_blocks) {
          const size_t base = (size_t)blk * hkv * SLAB + head_off + (size_t)w * 8;
          kv = ld16(k_cache + base);
          vv = ld16(v_cache + base);
          // V unit w = (dim d, half hf) holds slots 8 hf .. 8 hf + 7; zero slots >= len
          const int first = b * kBlockSize + (w & 1) * 8;
          if (first + 8 > len) {
            const int keep = max(len - first, 0);  // 0..7 slots stay
            uint32_t words[4] = {vv[0], vv[1], vv[2], vv[3]};
#pragma unroll
            for (int e = 0; e < 8; ++e) {
              if (e >= keep) words[e >> 1] &= (e & 1) ? 0x0000FFFFu : 0xFFFF0000u;
            }
            vv = u32x4{words[0], words[1], words[2], words[3]};
          }
        }
      }
      kreg[k] = kv;
      vreg[k] = vv;
    }
  };
  auto store_tile = [&](int buf) {
#pragma unroll
    for (int k = 0; k < LPT; ++k) {
      const int u = tid + 256 * k;
      const int bb = u / (SLAB / 8);
      const int w = u % (SLAB / 8);
      // K unit w = (chunk c, slot s): placed at c*16 + swap23(s)
      const int c = w >> 4, s = w & 15;
      const int kpos = bb * (SLAB / 8) + c * 16 + swap23(s);
      // V unit w = (dim d, half hf): placed at 2d + (hf ^ ((d >> 2) & 1))
      const int d = w >> 1, hf = w & 1;
      const int vpos = bb * (SLAB / 8) + 2 * d + (hf ^ ((d >> 2) & 1));
      st16(&sm.k[buf][kpos * 8], kreg[k]);
      st16(&sm.v[buf][vpos * 8], vreg[k]);
    }
  };

  load_tile(0);
  store_tile(0);
  __syncthreads();

  for (int kt = 0; kt < ntiles; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < ntiles) load_tile(kt + 1);

    const int key0 = kt * kKeys;
    if (wave_live && key0 <= p + wj_hi) {  // a key of the tile is visible to a wave column
      // ---- scores ----
      f32x16 s[2];
#pragma unroll
      for (int beta = 0; beta < 2; ++beta) {
#pragma unroll
        for (int r = 0; r < 16; ++r) s[beta][r] = 0.f;
        // A row lc <- key 32 beta + sigma(lc): block 2 beta + lc/16; LDS slot position lc%16
        const uint16_t* kb = &sm.k[buf][(2 * beta + (lc >> 4)) * SLAB];
#pragma unroll
        for (int kk = 0; kk < KK; ++kk) {
          const int c = 2 * kk + hh;
          const u32x4 a = ld16(kb + (c * 16 + (lc & 15)) * 8);
          s[beta] = mfma32(as_bf16x8(a), qf[kk], s[beta]);
        }
      }
      // register r of half-tile beta holds score row R = 8(r/4) + 4hh + r%4, i.e. key
      // key0 + 32 beta + sigma(R) = key0 + 32 beta + 8 hh + 4 (r/4 % 2) + 16 (r/8) + r%4
      const bool need_mask = key0 + kKeys - 1 > p + wj_lo;
      float mx = -INFINITY;
#pragma unroll
      for (int beta = 0; beta < 2; ++beta)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          float x = s[beta][r] * scale_log2;
          if (need_mask) {
            const int key = key0 + 32 * beta + 16 * (r >> 3) + 8 * hh + 4 * ((r >> 2) & 1) +
                            (r & 3);
            x = key <= lim ? x : -INFINITY;
          }
          s[beta][r] = x;
          mx = fmaxf(mx, x);
        }
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      const float m_new = fmaxf(m, mx);
      const float alpha = fast_exp2(m - m_new);
      m = m_new;
      float ps = 0.f;
      bf16x8 pf[2][2];
#pragma unroll
      for (int beta = 0; beta < 2; ++beta)
#pragma unroll
        for (int u = 0; u < 2; ++u) {
          u32x4 w;
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const float a = fast_exp2(s[beta][8 * u + 2 * e] - m_new);
            const float b = fast_exp2(s[beta][8 * u + 2 * e + 1] - m_new);
            ps += a + b;
            w[e] = pack_bf16x2(a, b);
          }
          pf[beta][u] = as_bf16x8(w);
        }
      lpart = lpart * alpha + ps;
#pragma unroll
      for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int r = 0; r < 16; ++r) o[db][r] *= alpha;
      // ---- values: step (beta, u) covers keys key0 + 32 beta + 16 u + 0..15 = block
      // 2 beta + u; lane group hh supplies slots 8 hh .. 8 hh + 7 of V^T row 32 db + lc ----
#pragma unroll
      for (int beta = 0; beta < 2; ++beta)
#pragma unroll
        for (int u = 0; u < 2; ++u) {
          const uint16_t* vb = &sm.v[buf][(2 * beta + u) * SLAB];
#pragma unroll
          for (int db = 0; db < DB; ++db) {
            const int d = db * 32 + lc;
            const int pos = 2 * d + (hh ^ ((d >> 2) & 1));
            const u32x4 a = ld16(vb + pos * 8);
            o[db] = mfma32(as_bf16x8(a), pf[beta][u], o[db]);
          }
        }
    }

    if (kt + 1 < ntiles) {
      store_tile(buf ^ 1);
    }
    __syncthreads();
  }

  const float l = lpart + __shfl_xor(lpart, 32);
  if (!col_ok) return;
  const float inv = 1.f / l;
  uint16_t* orow = out + ((size_t)(row0 + j) * hq + head) * D;
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int a = 0; a < 4; ++a) {
      // registers 4a .. 4a+3 hold dims 32 db + 8 a + 4 hh + 0..3
      u32x2 w = {pack_bf16x2(o[db][4 * a + 0] * inv, o[db][4 * a + 1] * inv),
                 pack_bf16x2(o[db][4 * a + 2] * inv, o[db][4 * a + 3] * inv)};
      st8(orow + db * 32 + 8 * a + 4 * hh, w);
    }
  if (lse != nullptr && hh == 0) lse[(size_t)(row0 + j) * hq + head] = (m + log2f(l)) * kLn2;
}

}  // namespace

hipError_t launch_prefill(const KvView& kv, const uint16_t* q, int32_t hq,
                          const int32_t* block_tables, int32_t max_blocks,
                          const int32_t* cached_lens, const int32_t* cu_new_lens,
                          int32_t num_seqs, int32_t max_new_len, float scale, uint16_t* out,
                          float* lse, hipStream_t stream) {
  const int32_t g = hq / kv.hkv;
  const int64_t qtiles = ((int64_t)max_new_len * g + kCols - 1) / kCols;
  const dim3 grid((unsigned)qtiles, kv.hkv, num_seqs);
  const float scale_log2 = scale * kLog2e;
  if (kv.head_dim == 128)
    hipLaunchKernelGGL(prefill_kernel<128>, grid, dim3(256), 0, stream, q, kv.k, kv.v,
                       block_tables, max_blocks, cached_lens, cu_new_lens, hq, kv.hkv,
                       kv.num_blocks, scale_log2, out, lse);
  else
    hipLaunchKernelGGL(prefill_kernel<64>, grid, dim3(256), 0, stream, q, kv.k, kv.v,
                       block_tables, max_blocks, cached_lens, cu_new_lens, hq, kv.hkv,
                       kv.num_blocks, scale_log2, out, lse);
  return hipGetLastError();
}

}  // namespace pkv
