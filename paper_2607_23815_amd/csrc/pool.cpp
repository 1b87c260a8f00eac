// KV block pool: host bookkeeping of which physical blocks each sequence holds.
//
// Follows the block-pool semantics of Section 2.1 ("vLLM memory model"): blocks are taken
// from a global pool when a request is admitted and returned when it completes, and a request
// that does not fit is deferred -- here `reserve` is all-or-nothing and a refusal changes no
// state, so the caller can defer and retry. Section 4's predicate contract (a dropped tuple
// frees its prefix) is `seq_free`; Section 5.3's rule that a parent's memory outlives its
// children (Algorithm 1, Complete) is `seq_fork` with per-block reference counts.
// Only whole blocks are shared; a write into a block held by another sequence is refused
// (or, through pkv_seq_reserve_cow, redirected to a private copy).
//
// Prefix cache (Section 2.1, automatic prefix caching, and Section 6, explicit and virtual
// pinning): a sequence's leading tokens can be published under a key. The entry holds one
// reference on each of its blocks, so they stay resident after the sequence is freed and a
// later sequence can attach to them (a hit) instead of recomputing them (a miss). Resident
// entries are evicted -- their references dropped -- when a reservation finds too few free
// blocks, least recently used first (or most recently used, the alternative the paper
// discusses); an entry pinned explicitly is not evicted while pinning is explicit. The
// deadlock check of Section 6 (requests waiting, none running) unpins every entry and
// switches to virtual pinning, under which pins no longer protect anything.
#include <algorithm>
#include <deque>
#include <map>
#include <string>
#include <unordered_map>
#include <vector>

#include "internal.h"

struct pkv_pool {
  int32_t num_blocks = 0;
  int32_t block_size = 0;
  std::deque<int32_t> free_list;  // front = next block handed out
  std::vector<int32_t> refcount;  // holders of each block: sequences plus cache entries
  std::vector<int32_t> seq_refs;  // the sequences among them
  struct Seq {
    std::vector<int32_t> blocks;
    int32_t length = 0;   // committed tokens
    int32_t pending = 0;  // reserved, not yet committed
  };
  std::unordered_map<int64_t, Seq> seqs;
  int64_t next_id = 1;
  // prefix cache
  struct Entry {
    std::vector<int32_t> blocks;
    int32_t tokens = 0;
    int32_t pins = 0;
    int64_t last_use = 0;  // logical clock of the last publish or attach
  };
  std::map<uint64_t, Entry> entries;
  int64_t clock = 0;
  int32_t eviction = PKV_EVICT_LRU;
  int32_t pinning = PKV_PIN_EXPLICIT;
  int64_t hits = 0, misses = 0, evictions = 0, cow_copies = 0;
};

namespace {

// An entry may be evicted when no pin protects it. Dropping it releases its references only:
// blocks that a sequence or another entry still holds stay with them.
bool evictable(const pkv_pool* pool, const pkv_pool::Entry& e) {
  return e.pins == 0 || pool->pinning == PKV_PIN_VIRTUAL;
}

// Evictable entries in eviction order: by last use, oldest first (LRU) or newest first (MRU).
// Every publish and hit takes its own clock tick, so last-use values are distinct.
std::vector<uint64_t> eviction_order(const pkv_pool* pool) {
  std::vector<std::pair<int64_t, uint64_t>> v;
  for (const auto& kv : pool->entries)
    if (evictable(pool, kv.second))
      v.push_back({pool->eviction == PKV_EVICT_LRU ? kv.second.last_use : -kv.second.last_use,
                   kv.first});
  std::sort(v.begin(), v.end());
  std::vector<uint64_t> out;
  for (const auto& x : v) out.push_back(x.second);
  return out;
}

void drop_entry(pkv_pool* pool, std::map<uint64_t, pkv_pool::Entry>::iterator it) {
  for (int32_t b : it->second.blocks)
    if (--pool->refcount[b] == 0) pool->free_list.push_back(b);
  pool->entries.erase(it);
}

// Make `need` blocks free by evicting entries in policy order, all or nothing: first count
// what evicting the prefix of the order would free (a block returns to the free list when
// its last reference goes), and evict only if that reaches `need`.
bool make_room(pkv_pool* pool, int64_t need) {
  if (need <= (int64_t)pool->free_list.size()) return true;
  const std::vector<uint64_t> order = eviction_order(pool);
  std::unordered_map<int32_t, int32_t> dec;
  int64_t freed = 0;
  size_t n_evict = 0;
  while ((int64_t)pool->free_list.size() + freed < need && n_evict < order.size()) {
    for (int32_t b : pool->entries.at(order[n_evict]).blocks)
      if (pool->refcount[b] - ++dec[b] == 0) ++freed;
    ++n_evict;
  }
  if ((int64_t)pool->free_list.size() + freed < need) return false;
  for (size_t k = 0; k < n_evict; ++k) drop_entry(pool, pool->entries.find(order[k]));
  pool->evictions += (int64_t)n_evict;
  return true;
}

// A free block handed to a sequence.
int32_t take_block(pkv_pool* pool) {
  const int32_t b = pool->free_list.front();
  pool->free_list.pop_front();
  pool->refcount[b] = 1;
  pool->seq_refs[b] = 1;
  return b;
}

// Shared body of pkv_seq_reserve (cow == false: a shared block in the write range is refused)
// and pkv_seq_reserve_cow (each such block is replaced by a private copy; the (source, copy)
// pairs go to `copies`).
pkv_status reserve_impl(pkv_pool* pool, int64_t seq, int32_t new_tokens, bool cow,
                        int32_t* copies, int32_t max_copies, int32_t* num_copies,
                        const char* fn) {
  const std::string name(fn);
  if (pool == nullptr) return pkv::fail(PKV_ERR_INVALID_ARG, name + ": NULL pool");
  if (num_copies != nullptr) *num_copies = 0;
  auto it = pool->seqs.find(seq);
  if (it == pool->seqs.end()) return pkv::fail(PKV_ERR_NOT_FOUND, name + ": unknown seq");
  if (new_tokens < 0) return pkv::fail(PKV_ERR_INVALID_ARG, name + ": new_tokens < 0");
  if (new_tokens == 0) return pkv::ok();
  pkv_pool::Seq& s = it->second;
  const int64_t start = (int64_t)s.length + s.pending;
  const int64_t end = start + new_tokens;
  if (end > INT32_MAX) return pkv::fail(PKV_ERR_INVALID_ARG, name + ": length overflow");
  std::vector<size_t> shared;
  for (size_t k = (size_t)(start / pool->block_size); k < s.blocks.size(); ++k)
    if (pool->refcount[s.blocks[k]] > 1) shared.push_back(k);
  if (!shared.empty() && !cow)
    return pkv::fail(PKV_ERR_SHARED_BLOCK_WRITE,
                     name + ": the new tokens would land in a block shared with another "
                            "holder");
  if ((int64_t)shared.size() > max_copies)
    return pkv::fail(PKV_ERR_INVALID_ARG, name + ": " + std::to_string(shared.size()) +
                                              " copies needed, room for " +
                                              std::to_string(max_copies));
  const int64_t grow = (end + pool->block_size - 1) / pool->block_size - (int64_t)s.blocks.size();
  const int64_t need = grow + (int64_t)shared.size();
  if (!make_room(pool, need))
    return pkv::fail(PKV_ERR_OUT_OF_BLOCKS, name + ": " + std::to_string(need) +
                                                " blocks needed, " +
                                                std::to_string(pool->free_list.size()) +
                                                " free after eviction");
  // an eviction above may have dropped a block's other holders: such a block is now private
  // and is written in place
  shared.erase(std::remove_if(shared.begin(), shared.end(),
                              [&](size_t k) { return pool->refcount[s.blocks[k]] <= 1; }),
               shared.end());
  for (size_t c = 0; c < shared.size(); ++c) {
    const int32_t old = s.blocks[shared[c]];
    const int32_t fresh = take_block(pool);
    pool->refcount[old] -= 1;  // was > 1: the block stays with its other holders
    pool->seq_refs[old] -= 1;
    s.blocks[shared[c]] = fresh;
    copies[2 * c] = old;
    copies[2 * c + 1] = fresh;
  }
  pool->cow_copies += (int64_t)shared.size();
  if (num_copies != nullptr) *num_copies = (int32_t)shared.size();
  for (int64_t k = 0; k < grow; ++k) s.blocks.push_back(take_block(pool));
  s.pending += new_tokens;
  return pkv::ok();
}

}  // namespace

using pkv::fail;
using pkv::ok;

extern "C" {

pkv_status pkv_pool_create(int32_t num_blocks, int32_t block_size, const int32_t* free_order,
                           pkv_pool** out) {
  if (out == nullptr) return fail(PKV_ERR_INVALID_ARG, "pkv_pool_create: out is NULL");
  *out = nullptr;
  if (num_blocks <= 0) return fail(PKV_ERR_INVALID_ARG, "pkv_pool_create: num_blocks <= 0");
  if (block_size != pkv::kSupportedBlockSize)
    return fail(PKV_ERR_UNSUPPORTED_SHAPE, "pkv_pool_create: block_size must be 16");
  auto* pool = new pkv_pool();
  pool->num_blocks = num_blocks;
  pool->block_size = block_size;
  pool->refcount.assign(num_blocks, 0);
  pool->seq_refs.assign(num_blocks, 0);
  if (free_order != nullptr) {
    std::vector<char> seen(num_blocks, 0);
    for (int32_t k = 0; k < num_blocks; ++k) {
      const int32_t b = free_order[k];
      if (b < 0 || b >= num_blocks || seen[b]) {
        delete pool;
        return fail(PKV_ERR_INVALID_ARG,
                    "pkv_pool_create: free_order is not a permutation of 0..num_blocks-1");
      }
      seen[b] = 1;
      pool->free_list.push_back(b);
    }
  } else {
    for (int32_t b = 0; b < num_blocks; ++b) pool->free_list.push_back(b);
  }
  *out = pool;
  return ok();
}

void pkv_pool_destroy(pkv_pool* pool) { delete pool; }

int32_t pkv_pool_num_free(const pkv_pool* pool) {
  return pool == nullptr ? -1 : (int32_t)pool->free_list.size();
}

pkv_status pkv_seq_create(pkv_pool* pool, int64_t* seq_id) {
  if (pool == nullptr || seq_id == nullptr)
    return fail(PKV_ERR_INVALID_ARG, "pkv_seq_create: NULL argument");
  const int64_t id = pool->next_id++;
  pool->seqs.emplace(id, pkv_pool::Seq());
  *seq_id = id;
  return ok();
}

pkv_status pkv_seq_fork(pkv_pool* pool, int64_t parent, int32_t shared_tokens, int64_t* child) {
  if (pool == nullptr || child == nullptr)
    return fail(PKV_ERR_INVALID_ARG, "pkv_seq_fork: NULL argument");
  auto it = pool->seqs.find(parent);
  if (it == pool->seqs.end()) return fail(PKV_ERR_NOT_FOUND, "pkv_seq_fork: unknown parent");
  const pkv_pool::Seq& p = it->second;
  if (shared_tokens < 0 || shared_tokens % pool->block_size != 0 || shared_tokens > p.length)
    return fail(PKV_ERR_INVALID_ARG,
                "pkv_seq_fork: shared_tokens must be a multiple of block_size within the "
                "parent's committed length");
  pkv_pool::Seq c;
  c.blocks.assign(p.blocks.begin(), p.blocks.begin() + shared_tokens / pool->block_size);
  c.length = shared_tokens;
  for (int32_t b : c.blocks) {
    pool->refcount[b] += 1;
    pool->seq_refs[b] += 1;
  }
  const int64_t id = pool->next_id++;
  pool->seqs.emplace(id, std::move(c));
  *child = id;
  return ok();
}

pkv_status pkv_seq_reserve(pkv_pool* pool, int64_t seq, int32_t new_tokens) {
  return reserve_impl(pool, seq, new_tokens, false, nullptr, 0, nullptr, "pkv_seq_reserve");
}

pkv_status pkv_seq_reserve_cow(pkv_pool* pool, int64_t seq, int32_t new_tokens, int32_t* copies,
                               int32_t max_copies, int32_t* num_copies) {
  if (num_copies == nullptr || max_copies < 0 || (max_copies > 0 && copies == nullptr))
    return fail(PKV_ERR_INVALID_ARG, "pkv_seq_reserve_cow: bad copies argument");
  return reserve_impl(pool, seq, new_tokens, true, copies, max_copies, num_copies,
                      "pkv_seq_reserve_cow");
}

pkv_status pkv_seq_commit(pkv_pool* pool, int64_t seq, int32_t new_tokens) {
  if (pool == nullptr) return fail(PKV_ERR_INVALID_ARG, "pkv_seq_commit: NULL pool");
  auto it = pool->seqs.find(seq);
  if (it == pool->seqs.end()) return fail(PKV_ERR_NOT_FOUND, "pkv_seq_commit: unknown seq");
  pkv_pool::Seq& s = it->second;
  if (new_tokens < 0 || new_tokens > s.pending)
    return fail(PKV_ERR_INVALID_ARG, "pkv_seq_commit: more tokens than reserved");
  s.length += new_tokens;
  s.pending -= new_tokens;
  return ok();
}

pkv_status pkv_seq_free(pkv_pool* pool, int64_t seq) {
  if (pool == nullptr) return fail(PKV_ERR_INVALID_ARG, "pkv_seq_free: NULL pool");
  auto it = pool->seqs.find(seq);
  if (it == pool->seqs.end()) return fail(PKV_ERR_NOT_FOUND, "pkv_seq_free: unknown seq");
  for (int32_t b : it->second.blocks) {
    pool->seq_refs[b] -= 1;
    if (--pool->refcount[b] == 0) pool->free_list.push_back(b);
  }
  pool->seqs.erase(it);
  return ok();
}

pkv_status pkv_seq_len(const pkv_pool* pool, int64_t seq, int32_t* len) {
  if (pool == nullptr || len == nullptr)
    return fail(PKV_ERR_INVALID_ARG, "pkv_seq_len: NULL argument");
  auto it = pool->seqs.find(seq);
  if (it == pool->seqs.end()) return fail(PKV_ERR_NOT_FOUND, "pkv_seq_len: unknown seq");
  *len = it->second.length;
  return ok();
}

pkv_status pkv_fill_block_tables(const pkv_pool* pool, const int64_t* seq_ids, int32_t n,
                                 int32_t max_blocks, int32_t* host_tables, int32_t* host_lens) {
  if (pool == nullptr || n < 0 || max_blocks < 0 ||
      (n > 0 && (seq_ids == nullptr || host_tables == nullptr)))
    return fail(PKV_ERR_INVALID_ARG, "pkv_fill_block_tables: bad argument");
  std::vector<const pkv_pool::Seq*> rows((size_t)n);
  for (int32_t k = 0; k < n; ++k) {
    auto it = pool->seqs.find(seq_ids[k]);
    if (it == pool->seqs.end())
      return fail(PKV_ERR_NOT_FOUND, "pkv_fill_block_tables: unknown seq");
    if ((int64_t)it->second.blocks.size() > max_blocks)
      return fail(PKV_ERR_INVALID_ARG, "pkv_fill_block_tables: a sequence holds more than "
                                       "max_blocks blocks");
    rows[k] = &it->second;
  }
  for (int32_t k = 0; k < n; ++k) {
    int32_t* row = host_tables + (size_t)k * max_blocks;
    const auto& blocks = rows[k]->blocks;
    std::copy(blocks.begin(), blocks.end(), row);
    std::fill(row + blocks.size(), row + max_blocks, -1);
    if (host_lens != nullptr) host_lens[k] = rows[k]->length;
  }
  return ok();
}

pkv_status pkv_pool_set_eviction(pkv_pool* pool, int32_t policy) {
  if (pool == nullptr || (policy != PKV_EVICT_LRU && policy != PKV_EVICT_MRU))
    return fail(PKV_ERR_INVALID_ARG, "pkv_pool_set_eviction: bad argument");
  pool->eviction = policy;
  return ok();
}

pkv_status pkv_pool_set_pinning(pkv_pool* pool, int32_t mode) {
  if (pool == nullptr || (mode != PKV_PIN_EXPLICIT && mode != PKV_PIN_VIRTUAL))
    return fail(PKV_ERR_INVALID_ARG, "pkv_pool_set_pinning: bad argument");
  pool->pinning = mode;
  return ok();
}

pkv_status pkv_pool_check_deadlock(pkv_pool* pool, int32_t waiting, int32_t running,
                                   int32_t* recovered) {
  if (pool == nullptr || recovered == nullptr || waiting < 0 || running < 0)
    return fail(PKV_ERR_INVALID_ARG, "pkv_pool_check_deadlock: bad argument");
  *recovered = 0;
  if (waiting > 0 && running == 0) {
    for (auto& kv : pool->entries) kv.second.pins = 0;
    pool->pinning = PKV_PIN_VIRTUAL;
    *recovered = 1;
  }
  return ok();
}

pkv_status pkv_prefix_publish(pkv_pool* pool, int64_t seq, uint64_t key, int32_t tokens) {
  if (pool == nullptr) return fail(PKV_ERR_INVALID_ARG, "pkv_prefix_publish: NULL pool");
  auto it = pool->seqs.find(seq);
  if (it == pool->seqs.end()) return fail(PKV_ERR_NOT_FOUND, "pkv_prefix_publish: unknown seq");
  const pkv_pool::Seq& s = it->second;
  if (tokens <= 0 || tokens > s.length)
    return fail(PKV_ERR_INVALID_ARG,
                "pkv_prefix_publish: tokens must be in 1..the sequence's committed length");
  if (pool->entries.count(key) != 0)
    return fail(PKV_ERR_KEY_EXISTS, "pkv_prefix_publish: key already published");
  pkv_pool::Entry e;
  e.blocks.assign(s.blocks.begin(),
                  s.blocks.begin() + (tokens + pool->block_size - 1) / pool->block_size);
  e.tokens = tokens;
  e.last_use = ++pool->clock;
  for (int32_t b : e.blocks) pool->refcount[b] += 1;
  pool->entries.emplace(key, std::move(e));
  return ok();
}

pkv_status pkv_prefix_attach(pkv_pool* pool, uint64_t key, int64_t* seq, int32_t* tokens) {
  if (pool == nullptr || seq == nullptr || tokens == nullptr)
    return fail(PKV_ERR_INVALID_ARG, "pkv_prefix_attach: NULL argument");
  auto it = pool->entries.find(key);
  if (it == pool->entries.end()) {
    pool->misses += 1;
    return fail(PKV_ERR_NOT_FOUND, "pkv_prefix_attach: no entry under this key");
  }
  pkv_pool::Entry& e = it->second;
  pkv_pool::Seq c;
  c.blocks = e.blocks;
  c.length = e.tokens;
  for (int32_t b : c.blocks) {
    pool->refcount[b] += 1;
    pool->seq_refs[b] += 1;
  }
  e.last_use = ++pool->clock;
  pool->hits += 1;
  const int64_t id = pool->next_id++;
  pool->seqs.emplace(id, std::move(c));
  *seq = id;
  *tokens = e.tokens;
  return ok();
}

pkv_status pkv_prefix_lookup(const pkv_pool* pool, uint64_t key, int32_t* tokens) {
  if (pool == nullptr || tokens == nullptr)
    return fail(PKV_ERR_INVALID_ARG, "pkv_prefix_lookup: NULL argument");
  auto it = pool->entries.find(key);
  *tokens = it == pool->entries.end() ? 0 : it->second.tokens;
  return ok();
}

pkv_status pkv_prefix_pin(pkv_pool* pool, uint64_t key) {
  if (pool == nullptr) return fail(PKV_ERR_INVALID_ARG, "pkv_prefix_pin: NULL pool");
  auto it = pool->entries.find(key);
  if (it == pool->entries.end()) return fail(PKV_ERR_NOT_FOUND, "pkv_prefix_pin: unknown key");
  it->second.pins += 1;
  return ok();
}

pkv_status pkv_prefix_unpin(pkv_pool* pool, uint64_t key) {
  if (pool == nullptr) return fail(PKV_ERR_INVALID_ARG, "pkv_prefix_unpin: NULL pool");
  auto it = pool->entries.find(key);
  if (it == pool->entries.end())
    return fail(PKV_ERR_NOT_FOUND, "pkv_prefix_unpin: unknown key");
  if (it->second.pins == 0) return fail(PKV_ERR_INVALID_ARG, "pkv_prefix_unpin: not pinned");
  it->second.pins -= 1;
  return ok();
}

pkv_status pkv_prefix_release(pkv_pool* pool, uint64_t key) {
  if (pool == nullptr) return fail(PKV_ERR_INVALID_ARG, "pkv_prefix_release: NULL pool");
  auto it = pool->entries.find(key);
  if (it == pool->entries.end())
    return fail(PKV_ERR_NOT_FOUND, "pkv_prefix_release: unknown key");
  drop_entry(pool, it);
  return ok();
}

pkv_status pkv_pool_get_stats(const pkv_pool* pool, pkv_pool_stats* out) {
  if (pool == nullptr || out == nullptr)
    return fail(PKV_ERR_INVALID_ARG, "pkv_pool_get_stats: NULL argument");
  out->num_free = (int32_t)pool->free_list.size();
  out->num_entries = (int32_t)pool->entries.size();
  out->cached_blocks = 0;
  for (int32_t b = 0; b < pool->num_blocks; ++b)
    if (pool->seq_refs[b] == 0 && pool->refcount[b] > 0) out->cached_blocks += 1;
  out->pinned_entries = 0;
  for (const auto& kv : pool->entries)
    if (kv.second.pins > 0) out->pinned_entries += 1;
  out->eviction = pool->eviction;
  out->pinning = pool->pinning;
  out->hits = pool->hits;
  out->misses = pool->misses;
  out->evictions = pool->evictions;
  out->cow_copies = pool->cow_copies;
  return ok();
}

}  // extern "C"
