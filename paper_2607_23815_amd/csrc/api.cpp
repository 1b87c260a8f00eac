// The C ABI's device calls: host-side argument validation, then the gfx950 kernel launches.
// Every check happens before any launch, so a refused call has enqueued nothing.
#include <hip/hip_runtime.h>

#include <atomic>
#include <cstdlib>
#include <cstring>
#include <string>

#include "internal.h"
#include "launch.h"

namespace pkv {

namespace {
thread_local std::string g_last_error;
}

pkv_status fail(pkv_status status, const std::string& message) {
  g_last_error = message;
  return status;
}

pkv_status ok() {
  g_last_error.clear();
  return PKV_OK;
}

namespace {

constexpr int kMaxGridZ = 65535;
constexpr int kMaxGridX = 1 << 30;

pkv_status check_kv(const pkv_paged_kv* kv, const char* fn, KvView* view) {
  const std::string f(fn);
  if (kv == nullptr) return fail(PKV_ERR_INVALID_ARG, f + ": kv is NULL");
  if (kv->k_cache == nullptr || kv->v_cache == nullptr)
    return fail(PKV_ERR_INVALID_ARG, f + ": k_cache / v_cache is NULL");
  if (kv->num_blocks <= 0 || kv->num_kv_heads <= 0)
    return fail(PKV_ERR_INVALID_ARG, f + ": num_blocks and num_kv_heads must be positive");
  if (kv->block_size != kSupportedBlockSize)
    return fail(PKV_ERR_UNSUPPORTED_SHAPE, f + ": block_size must be 16");
  if (kv->head_dim != 64 && kv->head_dim != 128)
    return fail(PKV_ERR_UNSUPPORTED_SHAPE, f + ": head_dim must be 64 or 128");
  if ((reinterpret_cast<uintptr_t>(kv->k_cache) | reinterpret_cast<uintptr_t>(kv->v_cache)) & 15)
    return fail(PKV_ERR_INVALID_ARG, f + ": k_cache / v_cache must be 16-byte aligned");
  view->k = static_cast<uint16_t*>(kv->k_cache);
  view->v = static_cast<uint16_t*>(kv->v_cache);
  view->num_blocks = kv->num_blocks;
  view->hkv = kv->num_kv_heads;
  view->head_dim = kv->head_dim;
  return PKV_OK;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

pkv_status launched(hipError_t err, const char* fn) {
  if (err != hipSuccess)
    return fail(PKV_ERR_HIP, std::string(fn) + ": " + hipGetErrorString(err));
  return ok();
}

// Opt-in validation of device metadata: off unless PKV_DEBUG_VALIDATE is set (and not "0")
// in the environment when the library first needs the setting, or pkv_set_debug_validate
// turns it on.
std::atomic<int> g_debug_validate{-1};

bool debug_validate() {
  int v = g_debug_validate.load(std::memory_order_relaxed);
  if (v < 0) {
    const char* e = std::getenv("PKV_DEBUG_VALIDATE");
    v = (e != nullptr && e[0] != '\0' && std::strcmp(e, "0") != 0) ? 1 : 0;
    int expected = -1;
    g_debug_validate.compare_exchange_strong(expected, v);
    v = g_debug_validate.load(std::memory_order_relaxed);
  }
  return v == 1;
}

// With validation on: run the checks (waiting for the stream) and refuse the call if any
// fails; with it off: nothing.
pkv_status check_metadata(const char* fn, const MetaCheck* checks, int n, hipStream_t stream) {
  if (!debug_validate()) return PKV_OK;
  uint32_t bad = 0u;
  int32_t seq = -1, which = -1;
  const hipError_t err = validate_metadata(checks, n, stream, &bad, &seq, &which);
  if (err != hipSuccess) return fail(PKV_ERR_HIP, std::string(fn) + ": " + hipGetErrorString(err));
  if (bad == 0u) return PKV_OK;
  std::string what;
  if (bad & kMetaBadBlockId) what += " a block id outside the pool;";
  if (bad & kMetaBadLength) what += " a length outside its host maximum or the table;";
  if (bad & kMetaBadOffsets) what += " token offsets not starting at 0, decreasing or not ending at the total;";
  std::string batch;
  if (n > 1) batch = which == 0 ? " of the prefill batch" : " of the decode batch";
  return fail(PKV_ERR_BAD_METADATA, std::string(fn) + ": PKV_DEBUG_VALIDATE refused the call:" +
                                        what + " first offending sequence " +
                                        std::to_string(seq) + batch);
}

MetaCheck meta(int32_t mode, const KvView& view, const int32_t* tables, int32_t max_blocks,
               const int32_t* lens, const int32_t* cu, int32_t num_seqs, int64_t total,
               int64_t max_len, int64_t max_total) {
  MetaCheck c;
  c.mode = mode;
  c.tables = tables;
  c.max_blocks = max_blocks;
  c.num_blocks = view.num_blocks;
  c.lens = lens;
  c.cu = cu;
  c.num_seqs = num_seqs;
  c.total = total;
  c.max_len = max_len;
  c.max_total = max_total;
  return c;
}

// Argument checks of a prefill batch (prefill and mixed calls); *empty when there is nothing
// to compute.
pkv_status check_prefill(const KvView& view, const char* fn, const void* q, int32_t num_q_heads,
                         const int32_t* block_tables, int32_t max_blocks,
                         const int32_t* cached_lens, const int32_t* cu_new_lens,
                         int32_t num_seqs, int32_t total_new, int32_t max_new_len,
                         int32_t max_total_len, float scale, const void* out,
                         const void* workspace, size_t workspace_bytes, bool* empty) {
  const std::string f(fn);
  *empty = false;
  if (num_q_heads <= 0 || num_q_heads % view.hkv != 0)
    return fail(PKV_ERR_UNSUPPORTED_SHAPE,
                f + ": num_q_heads must be a positive multiple of num_kv_heads");
  if (num_seqs < 0 || total_new < 0 || max_new_len < 0 || max_total_len < 0 || max_blocks < 0)
    return fail(PKV_ERR_INVALID_ARG, f + ": negative size");
  if (num_seqs == 0 || total_new == 0) {
    *empty = true;
    return ok();
  }
  if (q == nullptr || out == nullptr || block_tables == nullptr || cached_lens == nullptr ||
      cu_new_lens == nullptr)
    return fail(PKV_ERR_INVALID_ARG, f + ": NULL pointer");
  if (!aligned16(q) || !aligned16(out))
    return fail(PKV_ERR_INVALID_ARG, f + ": q / out must be 16-byte aligned");
  if (max_new_len == 0 || max_total_len < max_new_len || max_blocks == 0)
    return fail(PKV_ERR_INVALID_ARG,
                f + ": need 0 < max_new_len <= max_total_len, max_blocks > 0");
  if ((int64_t)max_blocks * kSupportedBlockSize < max_total_len)
    return fail(PKV_ERR_INVALID_ARG, f + ": max_total_len exceeds max_blocks * block_size");
  if (!(scale > 0.f)) return fail(PKV_ERR_INVALID_ARG, f + ": scale <= 0");
  if (num_seqs > kMaxGridZ)
    return fail(PKV_ERR_INVALID_ARG, f + ": more than 65535 sequences");
  // A workspace enables the key split of batches too small to fill the chip; without one
  // (NULL) the launch does not split. One that is given must hold what the split needs.
  const size_t need = prefill_workspace_bytes(num_seqs, total_new, num_q_heads, view.hkv,
                                              view.head_dim, max_new_len, max_total_len);
  if (need > 0 && workspace != nullptr && (workspace_bytes < need || !aligned16(workspace)))
    return fail(PKV_ERR_INVALID_ARG,
                f + ": workspace too small or not 16-byte aligned (see "
                    "pkv_prefill_workspace_bytes; NULL runs without the key split)");
  return ok();
}

// Argument checks of a decode batch (decode and mixed calls). With scratch set the call
// brings no workspace: the fixed scratch array must hold what it needs.
pkv_status check_decode(const KvView& view, const char* fn, const void* q, int32_t num_q_heads,
                        const int32_t* block_tables, int32_t max_blocks,
                        const int32_t* seq_lens, int32_t num_seqs, int32_t max_seq_len,
                        float scale, const void* out, const void* workspace,
                        size_t workspace_bytes, bool* empty, bool scratch = false) {
  const std::string f(fn);
  *empty = false;
  if (num_q_heads <= 0 || num_q_heads % view.hkv != 0 || num_q_heads / view.hkv > 16)
    return fail(PKV_ERR_UNSUPPORTED_SHAPE,
                f + ": num_q_heads must be a multiple of num_kv_heads, with at most 16 query "
                    "heads per kv head");
  if (num_seqs < 0 || max_seq_len < 0 || max_blocks < 0)
    return fail(PKV_ERR_INVALID_ARG, f + ": negative size");
  if (num_seqs == 0) {
    *empty = true;
    return ok();
  }
  if (q == nullptr || out == nullptr || block_tables == nullptr || seq_lens == nullptr)
    return fail(PKV_ERR_INVALID_ARG, f + ": NULL pointer");
  if (!aligned16(q) || !aligned16(out))
    return fail(PKV_ERR_INVALID_ARG, f + ": q / out must be 16-byte aligned");
  if (max_seq_len == 0 || max_blocks == 0)
    return fail(PKV_ERR_INVALID_ARG, f + ": max_seq_len, max_blocks must be > 0");
  if ((int64_t)max_blocks * kSupportedBlockSize < max_seq_len)
    return fail(PKV_ERR_INVALID_ARG, f + ": max_seq_len exceeds max_blocks * block_size");
  if (!(scale > 0.f)) return fail(PKV_ERR_INVALID_ARG, f + ": scale <= 0");
  const size_t need = decode_workspace_bytes(num_seqs, num_q_heads, view.hkv, view.head_dim,
                                             max_seq_len);
  if (scratch) {
    if (need > kDecodeScratchBytes)
      return fail(PKV_ERR_INVALID_ARG,
                  f + ": the call needs " + std::to_string(need) +
                      " bytes of workspace, above the fixed scratch of " +
                      std::to_string(kDecodeScratchBytes) +
                      " bytes (pkv_decode_attention takes a caller-owned workspace)");
    return ok();
  }
  if (need > 0 && (workspace == nullptr || workspace_bytes < need || !aligned16(workspace)))
    return fail(PKV_ERR_INVALID_ARG,
                f + ": workspace missing, too small or not 16-byte aligned "
                    "(see pkv_decode_workspace_bytes)");
  return ok();
}

}  // namespace
}  // namespace pkv

using namespace pkv;

extern "C" {

const char* pkv_last_error(void) { return pkv::g_last_error.c_str(); }

int32_t pkv_abi_version(void) { return 2; }

pkv_status pkv_set_debug_validate(int32_t on) {
  g_debug_validate.store(on != 0 ? 1 : 0, std::memory_order_relaxed);
  return ok();
}

int32_t pkv_get_debug_validate(void) { return debug_validate() ? 1 : 0; }

pkv_status pkv_kv_append(const pkv_paged_kv* kv, const void* k_new, const void* v_new,
                         const int32_t* block_tables, int32_t max_blocks,
                         const int32_t* cached_lens, const int32_t* cu_new_lens,
                         int32_t num_seqs, int32_t total_new, int32_t max_new_len,
                         void* stream) {
  const char* fn = "pkv_kv_append";
  KvView view;
  pkv_status st = check_kv(kv, fn, &view);
  if (st != PKV_OK) return st;
  if (num_seqs < 0 || total_new < 0 || max_new_len < 0 || max_blocks < 0)
    return fail(PKV_ERR_INVALID_ARG, "pkv_kv_append: negative size");
  if (num_seqs == 0 || total_new == 0) return ok();
  if (k_new == nullptr || v_new == nullptr || block_tables == nullptr ||
      cached_lens == nullptr || cu_new_lens == nullptr)
    return fail(PKV_ERR_INVALID_ARG, "pkv_kv_append: NULL pointer");
  if (!aligned16(k_new) || !aligned16(v_new))
    return fail(PKV_ERR_INVALID_ARG, "pkv_kv_append: k_new / v_new must be 16-byte aligned");
  if (max_new_len == 0 || max_blocks == 0)
    return fail(PKV_ERR_INVALID_ARG, "pkv_kv_append: max_new_len and max_blocks must be > 0");
  if (num_seqs > kMaxGridZ)
    return fail(PKV_ERR_INVALID_ARG, "pkv_kv_append: more than 65535 sequences per call");
  {
    const MetaCheck c = meta(kMetaAppend, view, block_tables, max_blocks, cached_lens,
                             cu_new_lens, num_seqs, total_new, max_new_len,
                             (int64_t)max_blocks * kSupportedBlockSize);
    if ((st = check_metadata(fn, &c, 1, static_cast<hipStream_t>(stream))) != PKV_OK) return st;
  }
  return launched(launch_kv_append(view, static_cast<const uint16_t*>(k_new),
                                   static_cast<const uint16_t*>(v_new), block_tables,
                                   max_blocks, cached_lens, cu_new_lens, num_seqs, max_new_len,
                                   static_cast<hipStream_t>(stream)),
                  fn);
}

size_t pkv_prefill_workspace_bytes(int32_t num_seqs, int32_t total_new, int32_t num_q_heads,
                                   int32_t num_kv_heads, int32_t head_dim, int32_t max_new_len,
                                   int32_t max_total_len) {
  if (num_seqs <= 0 || total_new <= 0 || num_q_heads <= 0 || num_kv_heads <= 0 ||
      head_dim <= 0 || max_new_len <= 0 || max_total_len <= 0 ||
      num_q_heads % num_kv_heads != 0)
    return 0;
  return prefill_workspace_bytes(num_seqs, total_new, num_q_heads, num_kv_heads, head_dim,
                                 max_new_len, max_total_len);
}

pkv_status pkv_prefill_attention(const pkv_paged_kv* kv, const void* q, int32_t num_q_heads,
                                 const int32_t* block_tables, int32_t max_blocks,
                                 const int32_t* cached_lens, const int32_t* cu_new_lens,
                                 int32_t num_seqs, int32_t total_new, int32_t max_new_len,
                                 int32_t max_total_len, float scale, void* out, float* lse,
                                 void* workspace, size_t workspace_bytes, void* stream) {
  const char* fn = "pkv_prefill_attention";
  KvView view;
  pkv_status st = check_kv(kv, fn, &view);
  if (st != PKV_OK) return st;
  bool empty = false;
  st = check_prefill(view, fn, q, num_q_heads, block_tables, max_blocks, cached_lens,
                     cu_new_lens, num_seqs, total_new, max_new_len, max_total_len, scale, out,
                     workspace, workspace_bytes, &empty);
  if (st != PKV_OK || empty) return st;
  {
    const MetaCheck c = meta(kMetaPrefill, view, block_tables, max_blocks, cached_lens,
                             cu_new_lens, num_seqs, total_new, max_new_len, max_total_len);
    if ((st = check_metadata(fn, &c, 1, static_cast<hipStream_t>(stream))) != PKV_OK) return st;
  }
  const bool split = workspace != nullptr &&
                     prefill_workspace_bytes(num_seqs, total_new, num_q_heads, view.hkv,
                                             view.head_dim, max_new_len, max_total_len) > 0;
  return launched(launch_prefill(view, static_cast<const uint16_t*>(q), num_q_heads,
                                 block_tables, max_blocks, cached_lens, cu_new_lens, num_seqs,
                                 total_new, max_new_len, max_total_len, scale,
                                 static_cast<uint16_t*>(out), lse, split ? workspace : nullptr,
                                 static_cast<hipStream_t>(stream)),
                  fn);
}

size_t pkv_decode_workspace_bytes(int32_t num_seqs, int32_t num_q_heads, int32_t num_kv_heads,
                                  int32_t head_dim, int32_t max_seq_len) {
  if (num_seqs <= 0 || num_q_heads <= 0 || num_kv_heads <= 0 || head_dim <= 0 ||
      max_seq_len <= 0)
    return 0;
  return decode_workspace_bytes(num_seqs, num_q_heads, num_kv_heads, head_dim, max_seq_len);
}

pkv_status pkv_decode_attention(const pkv_paged_kv* kv, const void* q, int32_t num_q_heads,
                                const int32_t* block_tables, int32_t max_blocks,
                                const int32_t* seq_lens, int32_t num_seqs, int32_t max_seq_len,
                                float scale, void* out, float* lse, void* workspace,
                                size_t workspace_bytes, void* stream) {
  const char* fn = "pkv_decode_attention";
  KvView view;
  pkv_status st = check_kv(kv, fn, &view);
  if (st != PKV_OK) return st;
  bool empty = false;
  st = check_decode(view, fn, q, num_q_heads, block_tables, max_blocks, seq_lens, num_seqs,
                    max_seq_len, scale, out, workspace, workspace_bytes, &empty);
  if (st != PKV_OK || empty) return st;
  {
    const MetaCheck c = meta(kMetaDecode, view, block_tables, max_blocks, seq_lens, nullptr,
                             num_seqs, -1, max_seq_len, 0);
    if ((st = check_metadata(fn, &c, 1, static_cast<hipStream_t>(stream))) != PKV_OK) return st;
  }
  return launched(launch_decode(view, static_cast<const uint16_t*>(q), num_q_heads,
                                block_tables, max_blocks, seq_lens, num_seqs, max_seq_len, scale,
                                static_cast<uint16_t*>(out), lse, workspace,
                                static_cast<hipStream_t>(stream)),
                  fn);
}

pkv_status pkv_decode_attention_noalloc(const pkv_paged_kv* kv, const void* q,
                                        int32_t num_q_heads, const int32_t* block_tables,
                                        int32_t max_blocks, const int32_t* seq_lens,
                                        int32_t num_seqs, int32_t max_seq_len, float scale,
                                        void* out, float* lse, void* stream) {
  const char* fn = "pkv_decode_attention_noalloc";
  static_assert(PKV_DECODE_NOALLOC_MAX_BYTES == kDecodeScratchBytes,
                "the header's limit is the scratch array's size");
  KvView view;
  pkv_status st = check_kv(kv, fn, &view);
  if (st != PKV_OK) return st;
  bool empty = false;
  st = check_decode(view, fn, q, num_q_heads, block_tables, max_blocks, seq_lens, num_seqs,
                    max_seq_len, scale, out, nullptr, 0, &empty, /*scratch=*/true);
  if (st != PKV_OK || empty) return st;
  {
    const MetaCheck c = meta(kMetaDecode, view, block_tables, max_blocks, seq_lens, nullptr,
                             num_seqs, -1, max_seq_len, 0);
    if ((st = check_metadata(fn, &c, 1, static_cast<hipStream_t>(stream))) != PKV_OK) return st;
  }
  void* ws = nullptr;
  const hipError_t err = decode_scratch(&ws);
  if (err != hipSuccess) return launched(err, fn);
  return launched(launch_decode(view, static_cast<const uint16_t*>(q), num_q_heads,
                                block_tables, max_blocks, seq_lens, num_seqs, max_seq_len, scale,
                                static_cast<uint16_t*>(out), lse, ws,
                                static_cast<hipStream_t>(stream)),
                  fn);
}

pkv_status pkv_mixed_attention(const pkv_paged_kv* kv, int32_t num_q_heads, float scale,
                               const void* q, const int32_t* block_tables, int32_t max_blocks,
                               const int32_t* cached_lens, const int32_t* cu_new_lens,
                               int32_t num_seqs, int32_t total_new, int32_t max_new_len,
                               int32_t max_total_len, void* out, float* lse, const void* dq,
                               const int32_t* d_block_tables, int32_t d_max_blocks,
                               const int32_t* seq_lens, int32_t d_num_seqs,
                               int32_t max_seq_len, void* d_out, float* d_lse,
                               void* workspace, size_t workspace_bytes, void* stream) {
  const char* fn = "pkv_mixed_attention";
  KvView view;
  pkv_status st = check_kv(kv, fn, &view);
  if (st != PKV_OK) return st;
  bool no_prefill = false, no_decode = false;
  st = check_prefill(view, fn, q, num_q_heads, block_tables, max_blocks, cached_lens,
                     cu_new_lens, num_seqs, total_new, max_new_len, max_total_len, scale, out,
                     nullptr, 0, &no_prefill);
  if (st != PKV_OK) return st;
  st = check_decode(view, fn, dq, num_q_heads, d_block_tables, d_max_blocks, seq_lens,
                    d_num_seqs, max_seq_len, scale, d_out, workspace, workspace_bytes,
                    &no_decode);
  if (st != PKV_OK) return st;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  if (no_prefill && no_decode) return ok();
  {
    MetaCheck c[2];
    c[0] = meta(kMetaPrefill, view, block_tables, max_blocks, cached_lens, cu_new_lens,
                no_prefill ? 0 : num_seqs, total_new, max_new_len, max_total_len);
    c[1] = meta(kMetaDecode, view, d_block_tables, d_max_blocks, seq_lens, nullptr,
                no_decode ? 0 : d_num_seqs, -1, max_seq_len, 0);
    if ((st = check_metadata(fn, c, 2, s)) != PKV_OK) return st;
  }
  if (no_decode)
    return launched(launch_prefill(view, static_cast<const uint16_t*>(q), num_q_heads,
                                   block_tables, max_blocks, cached_lens, cu_new_lens, num_seqs,
                                   total_new, max_new_len, max_total_len, scale,
                                   static_cast<uint16_t*>(out), lse, nullptr, s),
                    fn);
  if (no_prefill)
    return launched(launch_decode(view, static_cast<const uint16_t*>(dq), num_q_heads,
                                  d_block_tables, d_max_blocks, seq_lens, d_num_seqs,
                                  max_seq_len, scale, static_cast<uint16_t*>(d_out), d_lse,
                                  workspace, s),
                    fn);
  return launched(launch_mixed(view, num_q_heads, scale, static_cast<const uint16_t*>(q),
                               block_tables, max_blocks, cached_lens, cu_new_lens, num_seqs,
                               max_new_len, static_cast<uint16_t*>(out), lse,
                               static_cast<const uint16_t*>(dq), d_block_tables, d_max_blocks,
                               seq_lens, d_num_seqs, max_seq_len, static_cast<uint16_t*>(d_out),
                               d_lse, workspace, s),
                  fn);
}

pkv_status pkv_gather_kv(const pkv_paged_kv* kv, const int32_t* block_tables,
                         int32_t max_blocks, const int32_t* lens, const int32_t* cu_lens,
                         int32_t num_seqs, int32_t max_len, void* k_out, void* v_out,
                         void* stream) {
  const char* fn = "pkv_gather_kv";
  KvView view;
  pkv_status st = check_kv(kv, fn, &view);
  if (st != PKV_OK) return st;
  if (num_seqs < 0 || max_len < 0 || max_blocks < 0)
    return fail(PKV_ERR_INVALID_ARG, "pkv_gather_kv: negative size");
  if (num_seqs == 0 || max_len == 0) return ok();
  if (block_tables == nullptr || lens == nullptr || cu_lens == nullptr || k_out == nullptr ||
      v_out == nullptr)
    return fail(PKV_ERR_INVALID_ARG, "pkv_gather_kv: NULL pointer");
  if (!aligned16(k_out) || !aligned16(v_out))
    return fail(PKV_ERR_INVALID_ARG, "pkv_gather_kv: outputs must be 16-byte aligned");
  if (num_seqs > kMaxGridZ)
    return fail(PKV_ERR_INVALID_ARG, "pkv_gather_kv: more than 65535 sequences per call");
  {
    const MetaCheck c = meta(kMetaGather, view, block_tables, max_blocks, lens, cu_lens,
                             num_seqs, -1, max_len, 0);
    if ((st = check_metadata(fn, &c, 1, static_cast<hipStream_t>(stream))) != PKV_OK) return st;
  }
  return launched(launch_gather_kv(view, block_tables, max_blocks, lens, cu_lens, num_seqs,
                                   max_len, static_cast<uint16_t*>(k_out),
                                   static_cast<uint16_t*>(v_out),
                                   static_cast<hipStream_t>(stream)),
                  fn);
}

pkv_status pkv_copy_blocks(const pkv_paged_kv* kv, const int32_t* pairs, int32_t num_pairs,
                           void* stream) {
  const char* fn = "pkv_copy_blocks";
  KvView view;
  pkv_status st = check_kv(kv, fn, &view);
  if (st != PKV_OK) return st;
  if (num_pairs < 0) return fail(PKV_ERR_INVALID_ARG, "pkv_copy_blocks: negative size");
  if (num_pairs == 0) return ok();
  if (pairs == nullptr) return fail(PKV_ERR_INVALID_ARG, "pkv_copy_blocks: NULL pointer");
  if (num_pairs > kMaxGridX)
    return fail(PKV_ERR_INVALID_ARG, "pkv_copy_blocks: too many pairs per call");
  return launched(launch_copy_blocks(view, pairs, num_pairs, static_cast<hipStream_t>(stream)),
                  fn);
}

}  // extern "C"
