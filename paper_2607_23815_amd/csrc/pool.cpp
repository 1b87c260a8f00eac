// KV block pool: host bookkeeping of which physical blocks each sequence holds.
//
// Follows the block-pool semantics of Section 2.1 ("vLLM memory model"): blocks are taken
// from a global pool when a request is admitted and returned when it completes, and a request
// that does not fit is deferred -- here `reserve` is all-or-nothing and a refusal changes no
// state, so the caller can defer and retry. Section 4's predicate contract (a dropped tuple
// frees its prefix) is `seq_free`; Section 5.3's rule that a parent's memory outlives its
// children (Algorithm 1, Complete) is `seq_fork` with per-block reference counts.
// Only whole blocks are shared; a write into a block held by another sequence is refused.
#include <algorithm>
#include <deque>
#include <string>
#include <unordered_map>
#include <vector>

#include "internal.h"

struct pkv_pool {
  int32_t num_blocks = 0;
  int32_t block_size = 0;
  std::deque<int32_t> free_list;  // front = next block handed out
  std::vector<int32_t> refcount;
  struct Seq {
    std::vector<int32_t> blocks;
    int32_t length = 0;   // committed tokens
    int32_t pending = 0;  // reserved, not yet committed
  };
  std::unordered_map<int64_t, Seq> seqs;
  int64_t next_id = 1;
};

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
  for (int32_t b : c.blocks) pool->refcount[b] += 1;
  const int64_t id = pool->next_id++;
  pool->seqs.emplace(id, std::move(c));
  *child = id;
  return ok();
}

pkv_status pkv_seq_reserve(pkv_pool* pool, int64_t seq, int32_t new_tokens) {
  if (pool == nullptr) return fail(PKV_ERR_INVALID_ARG, "pkv_seq_reserve: NULL pool");
  auto it = pool->seqs.find(seq);
  if (it == pool->seqs.end()) return fail(PKV_ERR_NOT_FOUND, "pkv_seq_reserve: unknown seq");
  if (new_tokens < 0) return fail(PKV_ERR_INVALID_ARG, "pkv_seq_reserve: new_tokens < 0");
  if (new_tokens == 0) return ok();
  pkv_pool::Seq& s = it->second;
  const int64_t start = (int64_t)s.length + s.pending;
  const int64_t end = start + new_tokens;
  if (end > INT32_MAX) return fail(PKV_ERR_INVALID_ARG, "pkv_seq_reserve: length overflow");
  const int64_t first_blk = start / pool->block_size;
  for (size_t k = (size_t)first_blk; k < s.blocks.size(); ++k)
    if (pool->refcount[s.blocks[k]] > 1)
      return fail(PKV_ERR_SHARED_BLOCK_WRITE,
                  "pkv_seq_reserve: the new tokens would land in a block shared with another "
                  "sequence");
  const int64_t need = (end + pool->block_size - 1) / pool->block_size - (int64_t)s.blocks.size();
  if (need > (int64_t)pool->free_list.size())
    return fail(PKV_ERR_OUT_OF_BLOCKS, "pkv_seq_reserve: " + std::to_string(need) +
                                           " blocks needed, " +
                                           std::to_string(pool->free_list.size()) + " free");
  for (int64_t k = 0; k < need; ++k) {
    const int32_t b = pool->free_list.front();
    pool->free_list.pop_front();
    pool->refcount[b] = 1;
    s.blocks.push_back(b);
  }
  s.pending += new_tokens;
  return ok();
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

}  // extern "C"
