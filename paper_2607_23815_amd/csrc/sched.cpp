// Pipelined semantic-operator scheduler (Section 5, Algorithm 1; Section 6 memory management)
// over the KV block pool, with a step-synchronous engine that, in device mode, runs every
// engine step's attention work through this library's kernels.
//
// Pipeline: stage s runs one operator per task; task t of stage s+1 is right-side row
// t % fanout[s] joined (Cartesian product) with task t / fanout[s] of stage s and reuses that
// task's cached KV as its prefix. Per task the inputs fix the tokens it appends, the tokens its
// request generates and whether its predicate drops the tuple.
//
// Algorithm 1: each iteration launches what the memory manager admits (per stage in order,
// head of the waiting queue first), advances the engine one step, completes finished tasks
// (retry at the token bound with a doubled bound; children enqueued with the dependency
// tracked; final results output; memory released, cascading to parents whose children are all
// released) and rebalances budgets (saturated middle stages give Delta to the last stage,
// from themselves or else from the first stage with Delta unused; from the last stage down,
// a starving stage gives Delta to the one before it). Thresholds high = alpha * budget /
// minBudget and low = beta * budget / minBudget on the waiting-queue length.
//
// Readings where the paper is silent (the oracle's model takes the same ones): memory is
// counted in 16-token blocks; a task reusing its parent's P cached tokens is charged
// ceil((P + suffix + bound) / 16) - floor(P / 16) blocks (the partly filled last prefix block
// is copied on write), a task recomputing them ceil((P + suffix + bound) / 16) (blocking
// execution always charges that, since no parent keeps a charge); minBudget_s is the largest
// such charge at the largest bound; a step advances the first max_batch admitted tasks, the
// first step prefilling the prompt and yielding one token, each later step appending the
// previous token's KV and yielding one more; bounds are fixed at admission, estimated as the
// nearest-rank 99th percentile of the output/input ratio (double precision, rounded up) once
// min_obs requests have completed; a retried task's bound doubles, at most max_out.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <chrono>
#include <cmath>
#include <deque>
#include <set>
#include <string>
#include <vector>

#include "internal.h"

namespace {

constexpr int32_t kBS = 16;

int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }
uint64_t key_of(int32_t stage, int64_t idx) { return ((uint64_t)stage << 40) | (uint64_t)idx; }

struct Task {
  int32_t stage = 0;
  int64_t idx = 0;
  int64_t parent = -1;  // index into Sched::tasks
  int32_t bound = 0;
  bool fixed_bound = false;
  int64_t charge = 0;
  bool hit = true;
  int64_t seq = 0;
  int64_t cached = 0;  // prefix tokens reused from the cache
  int64_t prompt = 0;  // prompt tokens to prefill
  int64_t prefilled = 0;  // of which done
  int32_t generated = 0;
  int32_t children_left = 0;
};

// One engine step's attention work for one task.
struct StepItem {
  int64_t seq;
  int32_t cached;  // KV tokens already in the pool
  int32_t n_new;   // tokens this step appends (the prompt, or 1)
};

// Device mode: per step, block copies (copy-on-write), KV append, prefill attention over the
// tasks in their first step, decode attention over the others, timed with HIP events.
class DeviceRunner {
 public:
  ~DeviceRunner() { release(); }

  pkv_status init(const pkv_sched_device* dev, int32_t max_batch, int64_t max_kv_len,
                  int32_t max_table) {
    dev_ = *dev;
    const pkv_paged_kv& kv = dev_.kv;
    if (dev_.src_rows < max_batch)
      return pkv::fail(PKV_ERR_INVALID_ARG, "pkv_sched_run: src_rows < max_batch");
    max_table_ = max_table;
    max_batch_ = max_batch;
    // room for two groups' metadata (a step's last prefill group and its decode group go out
    // together), or for max_batch copy-on-write pairs
    const size_t meta_ints = 2 * ((size_t)max_batch * max_table + 4 * (size_t)max_batch + 8);
    meta_bytes_ = meta_ints * sizeof(int32_t);
    // The decode workspace depends on the batch and the longest sequence, and not
    // monotonically in the latter (shorter sequences may split into more pieces). Size it for
    // the most pieces any call can have: sequences of up to max_kv_len keys cut into splits of
    // at least 64 keys, on top of the space the sequence order takes.
    size_t ws = 0;
    for (int32_t n = 1; n <= max_batch; ++n) {
      const size_t order = pkv_decode_workspace_bytes(n, dev_.num_q_heads, kv.num_kv_heads,
                                                      kv.head_dim, 1);
      const size_t parts = (size_t)n * dev_.num_q_heads * (size_t)((max_kv_len + 63) / 64) *
                           (size_t)(kv.head_dim + 2) * sizeof(float);
      ws = std::max(ws, order + parts);
    }
    ws_bytes_ = ws;
    // prefill rows (at most src_rows), then a decode group's rows (at most max_batch)
    out_dec_off_ = (size_t)dev_.src_rows * dev_.num_q_heads * kv.head_dim * 2;
    const size_t out_bytes =
        out_dec_off_ + (size_t)max_batch * dev_.num_q_heads * kv.head_dim * 2;
    hipError_t e = hipMalloc(&meta_dev_, meta_bytes_);
    if (e == hipSuccess) e = hipHostMalloc(&meta_host_, meta_bytes_, hipHostMallocDefault);
    if (e == hipSuccess) e = hipMalloc(&out_, out_bytes);
    if (e == hipSuccess && ws_bytes_ > 0) e = hipMalloc(&ws_, ws_bytes_);
    if (e == hipSuccess) e = hipEventCreate(&ev0_);
    if (e == hipSuccess) e = hipEventCreate(&ev1_);
    if (e != hipSuccess) {
      release();
      return pkv::fail(PKV_ERR_HIP, std::string("pkv_sched_run: ") + hipGetErrorString(e));
    }
    return PKV_OK;
  }

  // Runs one step; adds the GPU time of its launches (block copies, appends, attention; not
  // the metadata uploads or the host's work between them) to *ms.
  pkv_status step(pkv_pool* pool, int64_t step_no, const std::vector<int32_t>& copies,
                  const std::vector<StepItem>& pre, const std::vector<StepItem>& dec,
                  double* ms) {
    hipStream_t stream = static_cast<hipStream_t>(dev_.stream);
    hipError_t e = hipSuccess;
    int32_t* h = static_cast<int32_t*>(meta_host_);
    int32_t* d = static_cast<int32_t*>(meta_dev_);
    pkv_status st = PKV_OK;
    step_no_ = step_no;
    ms_ = ms;
    // copy-on-write copies (one pair per admitted task that continues a partly filled
    // block), in groups of at most max_batch pairs, which the staging area holds
    for (size_t c0 = 0; c0 < copies.size(); c0 += 2 * (size_t)max_batch_) {
      const size_t cn = std::min(copies.size() - c0, 2 * (size_t)max_batch_);
      std::copy(copies.begin() + c0, copies.begin() + c0 + cn, h);
      if ((e = upload(h, d, cn, stream)) != hipSuccess) return hip_fail(e);
      if ((e = hipEventRecord(ev0_, stream)) != hipSuccess) return hip_fail(e);
      st = pkv_copy_blocks(&dev_.kv, d, (int32_t)(cn / 2), dev_.stream);
      if (st != PKV_OK) return st;
      if ((st = end_segment()) != PKV_OK) return st;
    }
    // prefill: groups of at most src_rows new tokens; the last one goes out with the decode
    // group in one fused launch (pkv_mixed_attention) when the step has both
    size_t a = 0;
    while (a < pre.size()) {
      size_t b = a;
      int64_t rows = 0;
      while (b < pre.size() && rows + pre[b].n_new <= dev_.src_rows) rows += pre[b++].n_new;
      if (b == a) return pkv::fail(PKV_ERR_INVALID_ARG, "pkv_sched_run: a prompt exceeds src_rows");
      if (b == pre.size() && !dec.empty()) return run_fused(pool, pre, a, b, dec);
      if ((st = run_group(pool, pre, a, b, false)) != PKV_OK) return st;
      a = b;
    }
    if (!dec.empty() && (st = run_group(pool, dec, 0, dec.size(), true)) != PKV_OK) return st;
    return PKV_OK;
  }

 private:
  pkv_status hip_fail(hipError_t e) {
    return pkv::fail(PKV_ERR_HIP, std::string("pkv_sched_run: ") + hipGetErrorString(e));
  }

  // End of a timed segment that began with ev0_: wait for it and add its time.
  pkv_status end_segment() {
    hipError_t e = hipEventRecord(ev1_, static_cast<hipStream_t>(dev_.stream));
    if (e == hipSuccess) e = hipEventSynchronize(ev1_);
    float t = 0.f;
    if (e == hipSuccess) e = hipEventElapsedTime(&t, ev0_, ev1_);
    if (e != hipSuccess) return hip_fail(e);
    *ms_ += t;
    return PKV_OK;
  }

  void call_hook(int32_t phase, bool decode, int32_t n, const int32_t* tab, const int32_t* cached,
                 const int32_t* cu, const void* out) {
    if (dev_.group_hook == nullptr) return;
    pkv_sched_group g;
    g.step = step_no_;
    g.phase = phase;
    g.decode = decode ? 1 : 0;
    g.num_seqs = n;
    g.max_blocks = max_table_;
    g.tables = tab;
    g.cached = cached;
    g.cu_new = cu;
    g.out = out;
    dev_.group_hook(dev_.hook_user, &g);
  }

  hipError_t upload(const int32_t* h, int32_t* d, size_t n, hipStream_t stream) {
    return hipMemcpyAsync(d, h, n * sizeof(int32_t), hipMemcpyHostToDevice, stream);
  }

  // One group's launch metadata, laid out at `h` (host, pinned) and mirrored at `d` (device):
  // tables [n][max_table], cached [n], cu_new [n + 1], lens [n].
  struct Group {
    int32_t n = 0, rows = 0, max_new = 0, max_total = 0;
    int32_t *h_tab = nullptr, *h_cached = nullptr, *h_cu = nullptr, *h_lens = nullptr;
    const int32_t *d_tab = nullptr, *d_cached = nullptr, *d_cu = nullptr, *d_lens = nullptr;
    size_t ints = 0;  // metadata size
  };
  pkv_status fill_group(pkv_pool* pool, const std::vector<StepItem>& items, size_t a, size_t b,
                        int32_t* h, const int32_t* d, Group* g) {
    const int32_t n = (int32_t)(b - a);
    g->n = n;
    g->h_tab = h;
    g->h_cached = h + (size_t)n * max_table_;
    g->h_cu = g->h_cached + n;
    g->h_lens = g->h_cu + n + 1;
    g->d_tab = d;
    g->d_cached = d + (size_t)n * max_table_;
    g->d_cu = g->d_cached + n;
    g->d_lens = g->d_cu + n + 1;
    g->ints = (size_t)n * max_table_ + 3 * (size_t)n + 1;
    std::vector<int64_t> ids((size_t)n);
    g->max_new = g->max_total = 0;
    for (int32_t k = 0; k < n; ++k) {
      const StepItem& it = items[a + k];
      ids[k] = it.seq;
      g->h_cached[k] = it.cached;
      g->h_cu[k] = k == 0 ? 0 : g->h_cu[k - 1] + items[a + k - 1].n_new;
      g->h_lens[k] = it.cached + it.n_new;
      g->max_new = std::max(g->max_new, it.n_new);
      g->max_total = std::max(g->max_total, it.cached + it.n_new);
    }
    g->h_cu[n] = g->h_cu[n - 1] + items[b - 1].n_new;
    g->rows = g->h_cu[n];
    return pkv_fill_block_tables(pool, ids.data(), n, max_table_, g->h_tab, nullptr);
  }

  // The group's KV append (rows cu_new[k].. of the K/V sources)
  pkv_status append(const Group& g) {
    return pkv_kv_append(&dev_.kv, dev_.k_src, dev_.v_src, g.d_tab, max_table_, g.d_cached,
                         g.d_cu, g.n, g.rows, g.max_new, dev_.stream);
  }

  // Metadata of items [a, b) into the pinned staging area and the device copy, then the
  // append and the attention launch. The staging area is reused only after the previous
  // group's launches have consumed it (synchronised below).
  pkv_status run_group(pkv_pool* pool, const std::vector<StepItem>& items, size_t a, size_t b,
                       bool decode) {
    hipStream_t stream = static_cast<hipStream_t>(dev_.stream);
    int32_t* h = static_cast<int32_t*>(meta_host_);
    int32_t* d = static_cast<int32_t*>(meta_dev_);
    Group g;
    pkv_status st = fill_group(pool, items, a, b, h, d, &g);
    if (st != PKV_OK) return st;
    hipError_t e = upload(h, d, g.ints, stream);
    if (e != hipSuccess) return hip_fail(e);
    if (dev_.group_hook != nullptr) {  // the pool and the metadata settle before the hook
      if ((e = hipStreamSynchronize(stream)) != hipSuccess) return hip_fail(e);
      call_hook(0, decode, g.n, g.h_tab, g.h_cached, g.h_cu, out_);
    }
    if ((e = hipEventRecord(ev0_, stream)) != hipSuccess) return hip_fail(e);
    if ((st = append(g)) != PKV_OK) return st;
    const float scale = 1.0f / std::sqrt((float)dev_.kv.head_dim);
    if (decode)
      st = pkv_decode_attention(&dev_.kv, dev_.q_src, dev_.num_q_heads, g.d_tab, max_table_,
                                g.d_lens, g.n, g.max_total, scale, out_, nullptr, ws_,
                                ws_bytes_, dev_.stream);
    else
      st = pkv_prefill_attention(&dev_.kv, dev_.q_src, dev_.num_q_heads, g.d_tab, max_table_,
                                 g.d_cached, g.d_cu, g.n, g.rows, g.max_new, g.max_total, scale,
                                 out_, nullptr, nullptr, 0, dev_.stream);
    if (st != PKV_OK) return st;
    if ((st = end_segment()) != PKV_OK) return st;
    call_hook(1, decode, g.n, g.h_tab, g.h_cached, g.h_cu, out_);
    return PKV_OK;
  }

  // The prefill group of items pre[a, b) and the decode group dec together: one metadata
  // upload, both appends, then one fused launch (pkv_mixed_attention, bit-identical to the
  // prefill call followed by the decode call). The prefill output goes to the start of the
  // output buffer, the decode output after the src_rows rows a prefill group can fill.
  pkv_status run_fused(pkv_pool* pool, const std::vector<StepItem>& pre, size_t a, size_t b,
                       const std::vector<StepItem>& dec) {
    hipStream_t stream = static_cast<hipStream_t>(dev_.stream);
    int32_t* h = static_cast<int32_t*>(meta_host_);
    int32_t* d = static_cast<int32_t*>(meta_dev_);
    Group gp, gd;
    pkv_status st = fill_group(pool, pre, a, b, h, d, &gp);
    if (st != PKV_OK) return st;
    st = fill_group(pool, dec, 0, dec.size(), h + gp.ints, d + gp.ints, &gd);
    if (st != PKV_OK) return st;
    hipError_t e = upload(h, d, gp.ints + gd.ints, stream);
    if (e != hipSuccess) return hip_fail(e);
    void* out_dec = static_cast<char*>(out_) + out_dec_off_;
    if (dev_.group_hook != nullptr) {  // both groups' pool blocks and metadata, before the appends
      if ((e = hipStreamSynchronize(stream)) != hipSuccess) return hip_fail(e);
      call_hook(0, false, gp.n, gp.h_tab, gp.h_cached, gp.h_cu, out_);
      call_hook(0, true, gd.n, gd.h_tab, gd.h_cached, gd.h_cu, out_dec);
    }
    if ((e = hipEventRecord(ev0_, stream)) != hipSuccess) return hip_fail(e);
    if ((st = append(gp)) != PKV_OK) return st;
    if ((st = append(gd)) != PKV_OK) return st;
    const float scale = 1.0f / std::sqrt((float)dev_.kv.head_dim);
    st = pkv_mixed_attention(&dev_.kv, dev_.num_q_heads, scale, dev_.q_src, gp.d_tab, max_table_,
                             gp.d_cached, gp.d_cu, gp.n, gp.rows, gp.max_new, gp.max_total,
                             out_, nullptr, dev_.q_src, gd.d_tab, max_table_, gd.d_lens, gd.n,
                             gd.max_total, out_dec, nullptr, ws_, ws_bytes_, dev_.stream);
    if (st != PKV_OK) return st;
    if ((st = end_segment()) != PKV_OK) return st;
    call_hook(1, false, gp.n, gp.h_tab, gp.h_cached, gp.h_cu, out_);
    call_hook(1, true, gd.n, gd.h_tab, gd.h_cached, gd.h_cu, out_dec);
    return PKV_OK;
  }

  void release() {
    if (dev_.stream != nullptr || meta_dev_ != nullptr)
      (void)hipStreamSynchronize(static_cast<hipStream_t>(dev_.stream));
    if (meta_dev_) (void)hipFree(meta_dev_);
    if (meta_host_) (void)hipHostFree(meta_host_);
    if (out_) (void)hipFree(out_);
    if (ws_) (void)hipFree(ws_);
    if (ev0_) (void)hipEventDestroy(ev0_);
    if (ev1_) (void)hipEventDestroy(ev1_);
    meta_dev_ = meta_host_ = out_ = ws_ = nullptr;
    ev0_ = ev1_ = nullptr;
  }

  pkv_sched_device dev_{};
  int64_t step_no_ = 0;
  double* ms_ = nullptr;
  int32_t max_table_ = 0, max_batch_ = 0;
  size_t meta_bytes_ = 0, ws_bytes_ = 0, out_dec_off_ = 0;
  void* meta_dev_ = nullptr;
  void* meta_host_ = nullptr;
  void* out_ = nullptr;
  void* ws_ = nullptr;
  hipEvent_t ev0_ = nullptr, ev1_ = nullptr;
};

class Sched {
 public:
  Sched(const pkv_sched_config& c, int32_t S, const int32_t* fanout) : c_(c), S_(S) {
    fanout_.assign(fanout, fanout + S);
    fanout_[S - 1] = 1;
  }

  pkv_status setup(int32_t num_tuples, int64_t num_tasks, const int32_t* suffix,
                   const int32_t* out_len, const uint8_t* filtered) {
    int64_t count = num_tuples, base = 0;
    for (int32_t s = 0; s < S_; ++s) {
      base_.push_back(base);
      count_.push_back(count);
      base += count;
      if (s + 1 < S_) {
        if (fanout_[s] < 1) return pkv::fail(PKV_ERR_INVALID_ARG, "pkv_sched_run: fanout < 1");
        count *= fanout_[s];
        if (count > ((int64_t)1 << 32))
          return pkv::fail(PKV_ERR_INVALID_ARG, "pkv_sched_run: too many tasks");
      }
    }
    if (base != num_tasks)
      return pkv::fail(PKV_ERR_INVALID_ARG,
                       "pkv_sched_run: num_tasks is not the sum of the stages' task counts");
    suffix_.assign(suffix, suffix + base);
    out_.assign(out_len, out_len + base);
    filt_.assign(filtered, filtered + base);
    prefix_.assign((size_t)base, 0);
    for (int64_t k = 0; k < base; ++k) {
      if (suffix_[k] < 0 || suffix_[k] > INT32_MAX / 4 || out_[k] < 1 || out_[k] > c_.max_out)
        return pkv::fail(PKV_ERR_INVALID_ARG,
                         "pkv_sched_run: suffix must be >= 0 and out_len in 1..max_out");
    }
    for (int32_t s = 1; s < S_; ++s)
      for (int64_t t = 0; t < count_[s]; ++t) {
        prefix_[base_[s] + t] = kv_len(s - 1, t / fanout_[s - 1]);
        if (prefix_[base_[s] + t] > INT32_MAX / 4)
          return pkv::fail(PKV_ERR_INVALID_ARG, "pkv_sched_run: a task's prefix is too long");
      }
    if (max_kv_len() > INT32_MAX / 2)
      return pkv::fail(PKV_ERR_INVALID_ARG, "pkv_sched_run: a task's sequence is too long");
    for (int32_t s = 0; s < S_; ++s) {
      int64_t mb = 0;
      for (int64_t t = 0; t < count_[s]; ++t)
        mb = std::max(mb, cdiv(P(s, t) + Suf(s, t) + c_.max_out, kBS));
      min_budget_.push_back(mb);
    }
    delta_ = c_.delta > 0 ? c_.delta : *std::max_element(min_budget_.begin(), min_budget_.end());
    // budgets
    budget_.assign(S_, 0);
    if (c_.policy == PKV_SCHED_SEQUENTIAL || c_.policy == PKV_SCHED_BLOCKING) {
      budget_[0] = c_.num_blocks;
    } else {
      for (int32_t s = 0; s + 1 < S_; ++s) budget_[s] = min_budget_[s];
      if (c_.policy == PKV_SCHED_BREADTH_FIRST && S_ > 1)
        budget_[0] = std::max(min_budget_[0], (int64_t)(c_.breadth_share * c_.num_blocks));
      int64_t rest = c_.num_blocks;
      for (int32_t s = 0; s + 1 < S_; ++s) rest -= budget_[s];
      budget_[S_ - 1] = rest;
      if (rest < min_budget_[S_ - 1])
        return pkv::fail(PKV_ERR_INVALID_ARG,
                         "pkv_sched_run: the pool is smaller than the stages' minimum budgets");
    }
    used_.assign(S_, 0);
    waiting_.assign(S_, {});
    ratios_.assign(S_, {});
    pkv_status st = pkv_pool_create(c_.num_blocks, kBS, nullptr, &pool_);
    if (st != PKV_OK) return st;
    if ((st = pkv_pool_set_eviction(pool_, c_.eviction)) != PKV_OK) return st;
    if ((st = pkv_pool_set_pinning(pool_, c_.pinning)) != PKV_OK) return st;
    return PKV_OK;
  }

  ~Sched() { pkv_pool_destroy(pool_); }

  int64_t max_prompt() const {
    int64_t m = 0;
    for (size_t k = 0; k < prefix_.size(); ++k) m = std::max(m, prefix_[k] + suffix_[k]);
    return m;
  }

  int64_t max_kv_len() const {
    int64_t m = 0;
    for (size_t k = 0; k < prefix_.size(); ++k) m = std::max(m, prefix_[k] + suffix_[k] + c_.max_out);
    return m;
  }

  pkv_status run(DeviceRunner* dev, int32_t* trace, int64_t max_events, int64_t* num_events,
                 pkv_sched_stats* stats) {
    trace_ = trace;
    max_events_ = max_events;
    for (int64_t t = 0; t < count_[0]; ++t) waiting_[0].push_back(new_task(0, t, -1));
    const auto w0 = std::chrono::steady_clock::now();
    pkv_status st = PKV_OK;
    while (any_waiting() || !running_.empty()) {
      if (step_ >= c_.max_steps) return pkv::fail(PKV_ERR_INVALID_ARG, "pkv_sched_run: step limit reached");
      copies_.clear();
      if ((st = admit_waiting()) != PKV_OK) return st;
      if (running_.empty())
        return pkv::fail(PKV_ERR_INVALID_ARG,
                         "pkv_sched_run: no task can be admitted and none is running");
      std::vector<std::pair<int64_t, int>> done;
      if ((st = engine_step(dev, &done)) != PKV_OK) return st;
      for (const auto& d : done)
        if ((st = on_finished(d.first, d.second == 1)) != PKV_OK) return st;
      if (c_.policy == PKV_SCHED_ADAPTIVE) adapt_budgets();
      ++step_;
    }
    const auto w1 = std::chrono::steady_clock::now();
    stats_.steps = step_;
    pkv_pool_stats ps;
    pkv_pool_get_stats(pool_, &ps);
    stats_.evictions = ps.evictions;
    stats_.wall_ms = std::chrono::duration<double, std::milli>(w1 - w0).count();
    *stats = stats_;
    *num_events = n_events_;
    return PKV_OK;
  }

  const std::vector<int64_t>& budgets() const { return budget_; }

 private:
  int64_t P(int32_t s, int64_t t) const { return prefix_[base_[s] + t]; }
  int64_t Suf(int32_t s, int64_t t) const { return suffix_[base_[s] + t]; }
  int32_t Out(int32_t s, int64_t t) const { return out_[base_[s] + t]; }
  bool Filtered(int32_t s, int64_t t) const { return filt_[base_[s] + t] != 0; }
  int64_t kv_len(int32_t s, int64_t t) const { return P(s, t) + Suf(s, t) + Out(s, t) - 1; }

  int64_t new_task(int32_t stage, int64_t idx, int64_t parent) {
    Task t;
    t.stage = stage;
    t.idx = idx;
    t.parent = parent;
    tasks_.push_back(t);
    return (int64_t)tasks_.size() - 1;
  }

  bool any_waiting() const {
    for (const auto& w : waiting_)
      if (!w.empty()) return true;
    return false;
  }

  void event(int32_t kind, int32_t stage, int64_t task, int64_t value) {
    if (trace_ != nullptr && n_events_ < max_events_) {
      int32_t* e = trace_ + 5 * n_events_;
      e[0] = (int32_t)step_;
      e[1] = kind;
      e[2] = stage;
      e[3] = (int32_t)task;
      e[4] = (int32_t)value;
    }
    ++n_events_;
  }

  int32_t charged_stage(const Task& t) const {
    return (c_.policy == PKV_SCHED_SEQUENTIAL || c_.policy == PKV_SCHED_BLOCKING) ? 0 : t.stage;
  }

  int32_t bound_of(const Task& t) const {
    if (t.fixed_bound) return t.bound;
    const int32_t s = t.stage;
    if (c_.static_bound[s] > 0) return std::min(c_.static_bound[s], c_.max_out);
    const std::multiset<double>& r = ratios_[s];
    if ((int64_t)r.size() >= c_.min_obs) {
      const int64_t k = (99 * (int64_t)r.size() + 99) / 100 - 1;  // nearest rank
      auto it = r.begin();
      std::advance(it, k);
      const double prompt = (double)(P(s, t.idx) + Suf(s, t.idx));
      const double b = std::ceil(*it * prompt);
      return (int32_t)std::max(1.0, std::min(b, (double)c_.max_out));
    }
    return std::max(1, std::min(c_.initial_bound[s] > 0 ? c_.initial_bound[s] : c_.max_out,
                                c_.max_out));
  }

  // (charge, hit, bound) of admitting task ti now
  void size_of(const Task& t, int64_t* charge, bool* hit, int32_t* bound) const {
    const int32_t s = t.stage;
    const int64_t p = P(s, t.idx), suf = Suf(s, t.idx);
    *bound = bound_of(t);
    int32_t tok = 0;
    if (s == 0) {
      *hit = true;
    } else {
      pkv_prefix_lookup(pool_, key_of(s - 1, t.idx / fanout_[s - 1]), &tok);
      *hit = tok > 0;
    }
    const int64_t whole = cdiv(p + suf + *bound, kBS);
    *charge = (c_.policy == PKV_SCHED_BLOCKING || !*hit) ? whole : whole - p / kBS;
  }

  // Whether task t's reservation fits now: in its stage's budget, or (one shared budget for
  // the sequential and blocking policies) in the whole pool.
  bool fits(int32_t stage, const Task& t) const {
    int64_t charge;
    bool hit;
    int32_t bound;
    size_of(t, &charge, &hit, &bound);
    if (shared_budget()) {
      int64_t u = 0;
      for (int64_t x : used_) u += x;
      return u + charge <= c_.num_blocks;
    }
    return used_[stage] + charge <= budget_[stage];
  }
  bool shared_budget() const {
    return c_.policy == PKV_SCHED_BLOCKING || c_.policy == PKV_SCHED_SEQUENTIAL;
  }

  pkv_status allocate(int32_t stage, int64_t ti) {
    Task& t = tasks_[ti];
    int64_t charge;
    bool hit;
    int32_t bound;
    size_of(t, &charge, &hit, &bound);
    const int32_t s = t.stage;
    const int64_t p = P(s, t.idx), suf = Suf(s, t.idx);
    t.bound = bound;
    t.charge = charge;
    t.hit = hit;
    pkv_status st;
    if (s == 0) {
      if ((st = pkv_seq_create(pool_, &t.seq)) != PKV_OK) return st;
      if ((st = pkv_seq_reserve(pool_, t.seq, (int32_t)(suf + bound))) != PKV_OK) return st;
      t.cached = 0;
      t.prompt = suf;
    } else if (hit) {
      int32_t tok = 0;
      if ((st = pkv_prefix_attach(pool_, key_of(s - 1, t.idx / fanout_[s - 1]), &t.seq, &tok)) != PKV_OK)
        return st;
      int32_t pair[2] = {0, 0};
      int32_t ncp = 0;
      if ((st = pkv_seq_reserve_cow(pool_, t.seq, (int32_t)(suf + bound), pair, 1, &ncp)) != PKV_OK)
        return st;
      if (ncp == 1) {
        copies_.push_back(pair[0]);
        copies_.push_back(pair[1]);
      }
      stats_.cow_copies += ncp;
      t.cached = p;
      t.prompt = suf;
      stats_.hits += 1;
    } else {
      if ((st = pkv_seq_create(pool_, &t.seq)) != PKV_OK) return st;
      if ((st = pkv_seq_reserve(pool_, t.seq, (int32_t)(p + suf + bound))) != PKV_OK) return st;
      t.cached = 0;
      t.prompt = p + suf;
      stats_.misses += 1;
    }
    used_[charged_stage(t)] += charge;
    t.generated = 0;
    t.prefilled = 0;
    stats_.launches += 1;
    event(PKV_EV_LAUNCH, s, t.idx, 2 * charge + (hit ? 1 : 0));
    running_.push_back(ti);
    return PKV_OK;
  }

  // The stages whose queues may admit this iteration, [lo, hi): every stage; under blocking
  // execution only the first stage with unfinished work; under sequential execution the
  // deepest stage with a waiting task, and only while nothing runs (one task at a time).
  void admission_window(int32_t* lo, int32_t* hi) const {
    *lo = 0;
    *hi = S_;
    if (c_.policy == PKV_SCHED_SEQUENTIAL) {
      *hi = 0;
      if (!running_.empty()) return;
      for (int32_t s = S_ - 1; s >= 0; --s)
        if (!waiting_[s].empty()) {
          *lo = s;
          *hi = s + 1;
          return;
        }
      return;
    }
    if (c_.policy == PKV_SCHED_BLOCKING) {
      int32_t s = 0;
      for (; s < S_; ++s) {
        bool open = !waiting_[s].empty();
        for (int64_t ti : running_) open = open || tasks_[ti].stage == s;
        if (open) break;
      }
      *lo = s;
      *hi = s + 1;
    }
  }

  // Admission pass: each stage in the window hands over its queue in order while the head's
  // reservation fits; a head that does not fit stops that stage (first come, first served).
  pkv_status admit_waiting() {
    int32_t lo, hi;
    admission_window(&lo, &hi);
    const bool one_task = c_.policy == PKV_SCHED_SEQUENTIAL;
    for (int32_t s = lo; s < hi; ++s) {
      while (!waiting_[s].empty() && fits(s, tasks_[waiting_[s].front()])) {
        const int64_t ti = waiting_[s].front();
        waiting_[s].pop_front();
        pkv_status st = allocate(s, ti);
        if (st != PKV_OK) return st;
        if (one_task) return PKV_OK;
      }
    }
    return PKV_OK;
  }

  pkv_status engine_step(DeviceRunner* dev, std::vector<std::pair<int64_t, int>>* done) {
    const size_t nb = std::min(running_.size(), (size_t)c_.max_batch);
    stats_.max_batch = std::max(stats_.max_batch, (int32_t)nb);
    // tokens each batch task takes this step (-1: not scheduled)
    std::vector<int64_t> take(nb, -1);
    if (c_.max_step_tokens <= 0) {
      for (size_t k = 0; k < nb; ++k) {
        const Task& t = tasks_[running_[k]];
        take[k] = t.generated == 0 ? t.prompt - t.prefilled : 1;
      }
    } else {  // chunked prefill: decodes first, then prompt chunks, in queue order
      int64_t left = c_.max_step_tokens;
      for (size_t k = 0; k < nb; ++k)
        if (tasks_[running_[k]].generated > 0 && left > 0) {
          take[k] = 1;
          left -= 1;
        }
      for (size_t k = 0; k < nb; ++k) {
        const Task& t = tasks_[running_[k]];
        if (t.generated != 0) continue;
        const int64_t rest = t.prompt - t.prefilled;
        if (rest == 0 || left > 0) {
          take[k] = std::min(rest, left);
          left -= take[k];
        }
      }
    }
    std::vector<StepItem> pre, dec;
    for (size_t k = 0; k < nb; ++k) {
      if (take[k] < 0) continue;
      Task& t = tasks_[running_[k]];
      pkv_status st;
      if (t.generated == 0) {
        pre.push_back({t.seq, (int32_t)(t.cached + t.prefilled), (int32_t)take[k]});
        if ((st = pkv_seq_commit(pool_, t.seq, (int32_t)take[k])) != PKV_OK) return st;
        stats_.prefill_tokens += take[k];
        if (t.prefilled == 0) stats_.reused_tokens += t.cached;
        stats_.prefill_chunks += 1;
        t.prefilled += take[k];
        if (t.prefilled < t.prompt) continue;
      } else {
        dec.push_back({t.seq, (int32_t)(t.cached + t.prompt + t.generated - 1), 1});
        if ((st = pkv_seq_commit(pool_, t.seq, 1)) != PKV_OK) return st;
        stats_.decode_tokens += 1;
      }
      t.generated += 1;
      if (t.generated == Out(t.stage, t.idx))
        done->push_back({running_[k], 0});
      else if (t.generated == t.bound)
        done->push_back({running_[k], 1});
    }
    if (dev != nullptr) {
      pkv_status st = dev->step(pool_, step_, copies_, pre, dec, &stats_.gpu_ms);
      if (st != PKV_OK) return st;
    }
    return PKV_OK;
  }

  // Give back a finished task's charge, and with it the charge of every ancestor whose last
  // outstanding child this was (explicitly pinned prefixes are unpinned as they go, and stay
  // cached until evicted). Blocking execution tracks no children.
  pkv_status return_charges(int64_t ti) {
    for (int64_t cur = ti;;) {
      Task& t = tasks_[cur];
      used_[charged_stage(t)] -= t.charge;
      event(PKV_EV_RELEASE, t.stage, t.idx, t.charge);
      if (t.parent < 0 || c_.policy == PKV_SCHED_BLOCKING) return PKV_OK;
      Task& par = tasks_[t.parent];
      if (--par.children_left > 0) return PKV_OK;
      if (c_.pinning == PKV_PIN_EXPLICIT) {
        const pkv_status st = pkv_prefix_unpin(pool_, key_of(par.stage, par.idx));
        if (st != PKV_OK) return st;
      }
      cur = t.parent;
    }
  }

  // An interrupted request (it reached its token bound first): drop its sequence and charge,
  // double the bound (up to max_out) and queue the task again at the back of its stage.
  pkv_status requeue(int64_t ti) {
    Task& t = tasks_[ti];
    pkv_status st = pkv_seq_free(pool_, t.seq);
    if (st != PKV_OK) return st;
    used_[charged_stage(t)] -= t.charge;
    t.bound = std::min(2 * t.bound, c_.max_out);
    t.fixed_bound = true;
    stats_.retries += 1;
    event(PKV_EV_RETRY, t.stage, t.idx, t.bound);
    waiting_[t.stage].push_back(ti);
    return PKV_OK;
  }

  // A surviving task of a non-final stage: its join with the next stage's rows becomes that
  // stage's new tasks, all reusing its prefix, which is published in the prefix cache (pinned
  // under explicit pinning) before the task's own sequence goes. Its charge stays until the
  // last child returns its own (blocking execution returns it now).
  pkv_status spawn_children(int64_t ti) {
    const int32_t s = tasks_[ti].stage;
    const int64_t idx = tasks_[ti].idx;
    const int32_t f = fanout_[s];
    for (int32_t r = 0; r < f; ++r) waiting_[s + 1].push_back(new_task(s + 1, idx * f + r, ti));
    Task& t = tasks_[ti];  // new_task may have moved the vector
    t.children_left = f;
    const uint64_t key = key_of(s, idx);
    pkv_status st = pkv_prefix_publish(pool_, t.seq, key, (int32_t)kv_len(s, idx));
    if (st != PKV_OK) return st;
    if (c_.pinning == PKV_PIN_EXPLICIT && c_.policy != PKV_SCHED_BLOCKING &&
        (st = pkv_prefix_pin(pool_, key)) != PKV_OK)
      return st;
    if ((st = pkv_seq_free(pool_, t.seq)) != PKV_OK) return st;
    event(PKV_EV_DONE, s, idx, Out(s, idx));
    if (c_.policy == PKV_SCHED_BLOCKING) {
      used_[0] -= t.charge;
      event(PKV_EV_RELEASE, s, idx, t.charge);
    }
    return PKV_OK;
  }

  // A task the engine reports finished (interrupted: it hit its bound). A finished request
  // records its output/input ratio for the bound estimate; then it feeds the next stage, is a
  // result of the pipeline, or ends its branch (filtered); the last two free everything.
  pkv_status on_finished(int64_t ti, bool interrupted) {
    running_.erase(std::find(running_.begin(), running_.end(), ti));
    if (interrupted) return requeue(ti);
    const Task& t = tasks_[ti];
    const int32_t s = t.stage;
    ratios_[s].insert((double)Out(s, t.idx) / (double)(P(s, t.idx) + Suf(s, t.idx)));
    if (Filtered(s, t.idx)) {
      event(PKV_EV_FILTERED, s, t.idx, Out(s, t.idx));
    } else if (s + 1 < S_) {
      return spawn_children(ti);
    } else {
      stats_.outputs += 1;
      event(PKV_EV_OUTPUT, s, t.idx, Out(s, t.idx));
    }
    const pkv_status st = pkv_seq_free(pool_, tasks_[ti].seq);
    if (st != PKV_OK) return st;
    return return_charges(ti);
  }

  // Queue pressure of a stage against its budget, counted in tasks of its largest footprint
  // (minBudget): a backlog above alpha * budget / minBudget means the stage holds more
  // admitted work than the pipeline behind it can absorb (saturation); below beta * ... it
  // has too little queued work to keep its budget busy (starvation).
  double capacity_in_tasks(int32_t s) const {
    return (double)budget_[s] / (double)min_budget_[s];
  }
  bool backlog_high(int32_t s) const {
    return (double)waiting_[s].size() > c_.alpha * capacity_in_tasks(s);
  }
  bool backlog_low(int32_t s) const {
    return (double)waiting_[s].size() < c_.beta * capacity_in_tasks(s);
  }
  // A stage can spare delta blocks when that much of its budget is unused and what remains
  // still covers one task of its largest footprint.
  bool can_spare(int32_t u) const {
    return budget_[u] - used_[u] >= delta_ && budget_[u] - delta_ >= min_budget_[u];
  }
  void shift(int32_t from, int32_t to) {
    budget_[from] -= delta_;
    budget_[to] += delta_;
    event(PKV_EV_TRANSFER, from, to, delta_);
  }

  // Budget adaptation after each engine step (the adaptive policy). First, every middle
  // stage with a high backlog moves delta to the last stage, which is what drains it: from its
  // own spare budget, else from the first stage that can spare it. Then, walking from the
  // last stage back to the second, a stage with a low backlog hands delta of its spare budget
  // to the stage feeding it.
  void adapt_budgets() {
    const int32_t last = S_ - 1;
    for (int32_t s = 1; s < last; ++s) {
      if (!backlog_high(s)) continue;
      int32_t donor = can_spare(s) ? s : -1;
      for (int32_t u = 0; donor < 0 && u < last; ++u)
        if (can_spare(u)) donor = u;
      if (donor >= 0) shift(donor, last);
    }
    for (int32_t s = last; s >= 1; --s)
      if (backlog_low(s) && can_spare(s)) shift(s, s - 1);
  }

  pkv_sched_config c_;
  int32_t S_;
  std::vector<int32_t> fanout_;
  std::vector<int64_t> base_, count_;
  std::vector<int64_t> suffix_, prefix_;
  std::vector<int32_t> out_;
  std::vector<uint8_t> filt_;
  std::vector<int64_t> min_budget_, budget_, used_;
  int64_t delta_ = 0;
  std::vector<std::deque<int64_t>> waiting_;
  std::vector<int64_t> running_;
  std::vector<std::multiset<double>> ratios_;
  std::vector<Task> tasks_;
  std::vector<int32_t> copies_;
  pkv_pool* pool_ = nullptr;
  int32_t* trace_ = nullptr;
  int64_t max_events_ = 0, n_events_ = 0;
  int64_t step_ = 0;
  pkv_sched_stats stats_{};
};

}  // namespace

using pkv::fail;

extern "C" {

pkv_status pkv_sched_run(const pkv_sched_config* cfg, int32_t num_stages, int32_t num_tuples,
                         const int32_t* fanout, int64_t num_tasks, const int32_t* suffix,
                         const int32_t* out_len, const uint8_t* filtered,
                         const pkv_sched_device* dev, int32_t* trace,
                         int64_t max_events, int64_t* num_events, int64_t* final_budgets,
                         pkv_sched_stats* stats) {
  if (cfg == nullptr || fanout == nullptr || suffix == nullptr || out_len == nullptr ||
      filtered == nullptr || num_events == nullptr || stats == nullptr)
    return fail(PKV_ERR_INVALID_ARG, "pkv_sched_run: NULL argument");
  if (num_stages < 1 || num_stages > PKV_MAX_STAGES || num_tuples < 1)
    return fail(PKV_ERR_INVALID_ARG, "pkv_sched_run: need 1..8 stages and at least one tuple");
  if (cfg->policy < PKV_SCHED_ADAPTIVE || cfg->policy > PKV_SCHED_BLOCKING ||
      cfg->num_blocks < 1 || cfg->max_out < 1 || cfg->max_batch < 1 || cfg->min_obs < 1 ||
      cfg->delta < 0 || cfg->max_step_tokens < 0 || !(cfg->alpha > 0.0) || !(cfg->beta >= 0.0) ||
      !(cfg->breadth_share >= 0.0 && cfg->breadth_share <= 1.0) ||
      (trace == nullptr && max_events > 0) || max_events < 0)
    return fail(PKV_ERR_INVALID_ARG, "pkv_sched_run: bad configuration");
  Sched sched(*cfg, num_stages, fanout);
  pkv_status st = sched.setup(num_tuples, num_tasks, suffix, out_len, filtered);
  if (st != PKV_OK) return st;
  DeviceRunner runner;
  DeviceRunner* dp = nullptr;
  if (dev != nullptr) {
    if (dev->kv.num_blocks < cfg->num_blocks)
      return fail(PKV_ERR_INVALID_ARG, "pkv_sched_run: the device pool has fewer blocks than "
                                       "num_blocks");
    if (sched.max_prompt() > dev->src_rows)
      return fail(PKV_ERR_INVALID_ARG, "pkv_sched_run: src_rows is smaller than the longest "
                                       "prompt (prefix and suffix)");
    const int64_t max_len = sched.max_kv_len();
    if (max_len > INT32_MAX / 2) return fail(PKV_ERR_INVALID_ARG, "pkv_sched_run: too long");
    if ((st = runner.init(dev, cfg->max_batch, max_len, (int32_t)cdiv(max_len, kBS))) != PKV_OK)
      return st;
    dp = &runner;
  }
  *stats = pkv_sched_stats{};
  st = sched.run(dp, trace, max_events, num_events, stats);
  if (st != PKV_OK) return st;
  if (final_budgets != nullptr)
    for (int32_t s = 0; s < num_stages; ++s) final_budgets[s] = sched.budgets()[s];
  return pkv::ok();
}

}  // extern "C"
