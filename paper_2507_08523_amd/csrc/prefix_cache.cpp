// Host side of the prefix cache: chained 64-bit keys of 16-token blocks, an
// open-addressing key -> block-id table, and a bump block allocator.
//
// Block reuse follows InferLog section 2.1.2 ("KV Cache and Prefix Caching"):
// a block's KV is reusable only when the block and every block before it carry
// the same tokens, which a key chained over all preceding blocks captures.
// A batch is matched against the table as it stood before the batch (frozen
// snapshot), then its new full blocks are registered, first writer winning.
//
// Caches made by ilpc_cache_create_lru also give blocks a lifecycle (section
// 2.1.2: bounded memory, least-recently-used eviction): a block is in use
// (reference count > 0), cached (count 0 but still registered; on the LRU
// list), or free (on the free queue).  New blocks come from the free queue,
// else from the LRU head, whose key is then removed from the table.
#include <algorithm>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <new>
#include <string>
#include <vector>

#include "../../include/ilpc.h"
#include "ilpc_internal.h"

namespace ilpc {

namespace {
// A fixed buffer: recording an error allocates nothing, so it also works
// when the error is running out of memory.
thread_local char g_last_error[512];
}

int set_error(int code, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
  va_end(ap);
  return code;
}

namespace {

constexpr int kBlock = 16;
constexpr uint64_t kWordKey = 0x9E3779B97F4A7C15ull;  // golden-ratio word
constexpr uint64_t kChainSeed = 0x243F6A8885A308D3ull;  // fractional digits of pi

// MurmurHash3 64-bit finaliser (Appleby, public domain).
inline uint64_t fmix64(uint64_t x) {
  x ^= x >> 33;
  x *= 0xFF51AFD7ED558CCDull;
  x ^= x >> 33;
  x *= 0xC4CEB9FE1A85EC53ull;
  x ^= x >> 33;
  return x;
}

// Digest of one block: eight 64-bit words, each position-keyed and mixed
// independently (so the eight mixes overlap), summed, mixed once more.
inline uint64_t block_digest(const int32_t* t) {
  uint64_t acc = 0;
  for (int i = 0; i < kBlock / 2; ++i) {
    const uint64_t w = uint64_t(uint32_t(t[2 * i])) | (uint64_t(uint32_t(t[2 * i + 1])) << 32);
    acc += fmix64(w ^ (uint64_t(i + 1) * kWordKey));
  }
  return fmix64(acc);
}

}  // namespace
}  // namespace ilpc

struct ilpc_cache {
  int32_t num_blocks = 0;
  int32_t next_block = 0;
  uint64_t mask = 0;          // slots - 1
  int64_t max_entries = 0;    // 7/8 of the slots
  int64_t count = 0;
  std::vector<uint64_t> keys;  // 0 marks an empty slot
  std::vector<int32_t> vals;
  std::vector<uint64_t> journal;  // slot of every registration, oldest first

  // Block lifecycle (lru caches only).
  bool lru = false;
  std::vector<int32_t> ref;       // holders of each block
  std::vector<uint64_t> bkey;     // key registered for each block, 0 if none
  std::vector<int32_t> prv, nxt;  // LRU list of cached blocks, head = least recent
  int32_t lru_head = -1, lru_tail = -1;
  int64_t n_cached = 0, in_use = 0, evictions = 0;
  std::vector<int32_t> fq;        // free queue, a ring of num_blocks entries
  int64_t fq_head = 0, fq_size = 0;
  std::vector<int32_t> mark;      // per-block scratch counts, all zero between calls

  // Slot holding `key`, or the empty slot where it would go.
  uint64_t probe(uint64_t key) const {
    uint64_t s = key & mask;
    while (keys[s] != 0 && keys[s] != key) s = (s + 1) & mask;
    return s;
  }

  // Remove the key in slot s, shifting later members of its probe run back so
  // that every remaining key stays reachable from its home slot (linear
  // probing deletion without tombstones).
  void erase_slot(uint64_t s) {
    uint64_t hole = s;
    uint64_t j = s;
    for (;;) {
      j = (j + 1) & mask;
      if (keys[j] == 0) break;
      const uint64_t home = keys[j] & mask;
      // the key at j may move into the hole unless its home lies cyclically in (hole, j]
      const bool stays = hole <= j ? (hole < home && home <= j) : (hole < home || home <= j);
      if (stays) continue;
      keys[hole] = keys[j];
      vals[hole] = vals[j];
      hole = j;
    }
    keys[hole] = 0;
    vals[hole] = -1;
    --count;
  }

  void lru_unlink(int32_t b) {
    if (prv[b] >= 0) nxt[prv[b]] = nxt[b]; else lru_head = nxt[b];
    if (nxt[b] >= 0) prv[nxt[b]] = prv[b]; else lru_tail = prv[b];
    prv[b] = nxt[b] = -1;
    --n_cached;
  }

  void lru_push_tail(int32_t b) {
    prv[b] = lru_tail;
    nxt[b] = -1;
    if (lru_tail >= 0) nxt[lru_tail] = b; else lru_head = b;
    lru_tail = b;
    ++n_cached;
  }

  void fq_push(int32_t b) {
    fq[size_t((fq_head + fq_size) % num_blocks)] = b;
    ++fq_size;
  }

  // A block for a new logical block: the free queue's front, else the least
  // recently used cached block, whose key leaves the table.
  int32_t take() {
    int32_t b;
    if (fq_size > 0) {
      b = fq[size_t(fq_head)];
      fq_head = (fq_head + 1) % num_blocks;
      --fq_size;
    } else {
      b = lru_head;
      lru_unlink(b);
      erase_slot(probe(bkey[b]));
      bkey[b] = 0;
      ++evictions;
    }
    ref[b] = 1;
    ++in_use;
    return b;
  }

  void lifecycle_reset() {
    std::fill(ref.begin(), ref.end(), 0);
    std::fill(bkey.begin(), bkey.end(), 0);
    std::fill(prv.begin(), prv.end(), -1);
    std::fill(nxt.begin(), nxt.end(), -1);
    for (int32_t b = 0; b < num_blocks; ++b) fq[size_t(b)] = b;
    lru_head = lru_tail = -1;
    n_cached = in_use = evictions = 0;
    fq_head = 0;
    fq_size = num_blocks;
  }
};

using ilpc::set_error;

extern "C" const char* ilpc_last_error(void) { return ilpc::g_last_error; }

namespace {

int create_cache(const char* fn, int32_t num_blocks, int32_t block_size, int32_t table_log2_cap,
                 bool lru, ilpc_cache** out) {
  if (!out) return set_error(ILPC_EINVAL, "%s: out is NULL", fn);
  *out = nullptr;
  if (block_size != ilpc::kBlock)
    return set_error(ILPC_EUNSUP, "%s: block_size %d unsupported (16)", fn, block_size);
  if (num_blocks < 0) return set_error(ILPC_EINVAL, "%s: num_blocks < 0", fn);
  if (table_log2_cap < 1 || table_log2_cap > 30)
    return set_error(ILPC_EINVAL, "%s: table_log2_cap %d not in [1, 30]", fn, table_log2_cap);
  const uint64_t slots = uint64_t(1) << table_log2_cap;
  const int64_t max_entries = int64_t(slots - slots / 8);
  if (lru && max_entries < num_blocks)
    return set_error(ILPC_EINVAL, "%s: key capacity %lld < num_blocks %d (raise table_log2_cap)",
                     fn, (long long)max_entries, num_blocks);
  ilpc_cache* c = new (std::nothrow) ilpc_cache();
  if (!c) return set_error(ILPC_ENOSPC, "%s: out of host memory", fn);
  try {
    c->keys.assign(slots, 0);
    c->vals.assign(slots, -1);
    if (lru) {
      const size_t n = size_t(num_blocks);
      c->ref.assign(n, 0);
      c->bkey.assign(n, 0);
      c->prv.assign(n, -1);
      c->nxt.assign(n, -1);
      c->fq.assign(n, 0);
      c->mark.assign(n, 0);
    }
  } catch (...) {
    delete c;
    return set_error(ILPC_ENOSPC, "%s: out of host memory", fn);
  }
  c->num_blocks = num_blocks;
  c->mask = slots - 1;
  c->max_entries = max_entries;
  c->lru = lru;
  if (lru) c->lifecycle_reset();
  *out = c;
  return ILPC_OK;
}

}  // namespace

extern "C" int ilpc_cache_create(int32_t num_blocks, int32_t block_size, int32_t table_log2_cap,
                                 ilpc_cache** out) {
  return create_cache("ilpc_cache_create", num_blocks, block_size, table_log2_cap, false, out);
}

extern "C" int ilpc_cache_create_lru(int32_t num_blocks, int32_t block_size,
                                     int32_t table_log2_cap, ilpc_cache** out) {
  return create_cache("ilpc_cache_create_lru", num_blocks, block_size, table_log2_cap, true, out);
}

extern "C" void ilpc_cache_destroy(ilpc_cache* cache) { delete cache; }

extern "C" int ilpc_cache_reset(ilpc_cache* cache) {
  if (!cache) return set_error(ILPC_EINVAL, "ilpc_cache_reset: cache is NULL");
  std::fill(cache->keys.begin(), cache->keys.end(), 0);
  std::fill(cache->vals.begin(), cache->vals.end(), -1);
  cache->count = 0;
  cache->next_block = 0;
  cache->journal.clear();
  if (cache->lru) cache->lifecycle_reset();
  return ILPC_OK;
}

extern "C" int ilpc_cache_stats(const ilpc_cache* cache, int64_t stats[4]) {
  if (!cache || !stats) return set_error(ILPC_EINVAL, "ilpc_cache_stats: NULL argument");
  stats[0] = cache->count;
  stats[1] = cache->lru ? cache->num_blocks - cache->fq_size : cache->next_block;
  stats[2] = cache->max_entries;
  stats[3] = cache->num_blocks;
  return ILPC_OK;
}

extern "C" int ilpc_cache_checkpoint(const ilpc_cache* cache, int64_t mark[2]) {
  if (!cache || !mark) return set_error(ILPC_EINVAL, "ilpc_cache_checkpoint: NULL argument");
  if (cache->lru)
    return set_error(ILPC_EUNSUP, "ilpc_cache_checkpoint: not available on an LRU cache");
  mark[0] = int64_t(cache->journal.size());
  mark[1] = cache->next_block;
  return ILPC_OK;
}

extern "C" int ilpc_cache_rollback(ilpc_cache* cache, const int64_t mark[2]) {
  if (!cache || !mark) return set_error(ILPC_EINVAL, "ilpc_cache_rollback: NULL argument");
  if (cache->lru)
    return set_error(ILPC_EUNSUP, "ilpc_cache_rollback: not available on an LRU cache");
  if (mark[0] < 0 || mark[0] > int64_t(cache->journal.size()) || mark[1] < 0 ||
      mark[1] > cache->next_block)
    return set_error(ILPC_EINVAL, "ilpc_cache_rollback: mark is not from this cache's history");
  // Removing the newest registrations first keeps every remaining key's probe
  // run intact: each survivor was inserted before them, past older keys only.
  while (int64_t(cache->journal.size()) > mark[0]) {
    const uint64_t s = cache->journal.back();
    cache->journal.pop_back();
    cache->keys[s] = 0;
    cache->vals[s] = -1;
    --cache->count;
  }
  cache->next_block = int32_t(mark[1]);
  return ILPC_OK;
}

extern "C" int ilpc_prefix_match(ilpc_cache* cache, const int32_t* tokens,
                                 const int32_t* cu_seqlens, int32_t B, const int32_t* reserve,
                                 int32_t max_blocks, uint32_t flags, int32_t* cached_len,
                                 int32_t* block_tables, uint64_t* block_keys) {
  using namespace ilpc;
  if (!cache) return set_error(ILPC_EINVAL, "ilpc_prefix_match: cache is NULL");
  if (B < 0) return set_error(ILPC_EINVAL, "ilpc_prefix_match: B < 0");
  if (B == 0) return ILPC_OK;
  if (!cu_seqlens || !cached_len || !block_tables)
    return set_error(ILPC_EINVAL, "ilpc_prefix_match: NULL argument");
  if (flags & ~(ILPC_NO_LOOKUP | ILPC_NO_REGISTER))
    return set_error(ILPC_EINVAL, "ilpc_prefix_match: unknown flags 0x%x", flags);
  if (max_blocks < 1) return set_error(ILPC_EINVAL, "ilpc_prefix_match: max_blocks < 1");
  if (cu_seqlens[0] != 0) return set_error(ILPC_EINVAL, "ilpc_prefix_match: cu_seqlens[0] != 0");
  if (!tokens) return set_error(ILPC_EINVAL, "ilpc_prefix_match: tokens is NULL");
  const bool lookup = !(flags & ILPC_NO_LOOKUP);
  const bool reg = !(flags & ILPC_NO_REGISTER);

  // Validate every request before touching anything.
  int64_t total_keys = 0;
  for (int32_t r = 0; r < B; ++r) {
    const int64_t L = int64_t(cu_seqlens[r + 1]) - cu_seqlens[r];
    if (L < 1) return set_error(ILPC_EINVAL, "ilpc_prefix_match: request %d has length %lld", r,
                                (long long)L);
    const int64_t res = reserve ? reserve[r] : 0;
    if (res < 0) return set_error(ILPC_EINVAL, "ilpc_prefix_match: request %d reserve < 0", r);
    const int64_t n_total = (L + res + kBlock - 1) / kBlock;
    if (n_total > max_blocks)
      return set_error(ILPC_EINVAL, "ilpc_prefix_match: request %d needs %lld blocks > max_blocks %d",
                       r, (long long)n_total, max_blocks);
    total_keys += L / kBlock;
  }

  // Keys of every full block, and the matched run of each request (read-only pass).
  // Every allocation of the call happens here, before any state changes
  // (the bump cache's registration journal is grown to hold this batch's
  // keys too), so a call that runs out of host memory changes nothing.
  std::vector<uint64_t> keys;
  std::vector<int64_t> key_off, hit_off;
  std::vector<int32_t> matched, hit_ids;
  try {
    keys.resize(size_t(total_keys));
    key_off.resize(size_t(B) + 1);
    hit_off.resize(size_t(B) + 1);
    matched.resize(size_t(B));
    hit_ids.reserve(size_t(total_keys));
    const size_t jneed = cache->journal.size() + size_t(total_keys);
    if (reg && !cache->lru && jneed > cache->journal.capacity())
      cache->journal.reserve(std::max(jneed, 2 * cache->journal.capacity()));
  } catch (...) {
    return set_error(ILPC_ENOSPC, "ilpc_prefix_match: out of host memory");
  }
  int64_t ko = 0;
  for (int32_t r = 0; r < B; ++r) {
    const int32_t* t = tokens + cu_seqlens[r];
    const int64_t L = int64_t(cu_seqlens[r + 1]) - cu_seqlens[r];
    const int64_t n_full = L / kBlock, cap = (L - 1) / kBlock;
    key_off[r] = ko;
    uint64_t c = kChainSeed;
    for (int64_t b = 0; b < n_full; ++b) {
      c = fmix64(c ^ block_digest(t + b * kBlock));
      if (c == 0) c = 1;
      keys[size_t(ko + b)] = c;
    }
    hit_off[r] = int64_t(hit_ids.size());
    int32_t m = 0;
    if (lookup) {
      while (m < cap) {
        const uint64_t s = cache->probe(keys[size_t(ko + m)]);
        if (cache->keys[s] == 0) break;
        hit_ids.push_back(cache->vals[s]);
        ++m;
      }
    }
    matched[r] = m;
    ko += n_full;
  }
  key_off[B] = ko;
  hit_off[B] = int64_t(hit_ids.size());

  // Capacity checks (pool, then key table) before any state change.
  int64_t next = cache->next_block;
  int64_t new_keys = 0, need = 0;
  for (int32_t r = 0; r < B; ++r) {
    const int64_t L = int64_t(cu_seqlens[r + 1]) - cu_seqlens[r];
    const int64_t res = reserve ? reserve[r] : 0;
    need += (L + res + kBlock - 1) / kBlock - matched[r];
    new_keys += L / kBlock - matched[r];
  }
  next += need;
  if (cache->lru) {
    // Cached blocks this batch hits are pinned before any is taken, so they
    // do not count as available.
    int64_t revived = 0;
    for (const int32_t b : hit_ids) {
      if (cache->ref[b] == 0 && cache->mark[b] == 0) ++revived;
      cache->mark[b] = 1;
    }
    for (const int32_t b : hit_ids) cache->mark[b] = 0;
    const int64_t avail = cache->fq_size + cache->n_cached - revived;
    if (need > avail)
      return set_error(ILPC_ENOSPC,
                       "ilpc_prefix_match: batch needs %lld new blocks, %lld free or evictable",
                       (long long)need, (long long)avail);
    for (const int32_t b : hit_ids) {
      if (cache->ref[b] == 0) {
        cache->lru_unlink(b);
        ++cache->in_use;
      }
      ++cache->ref[b];
    }
  } else {
    if (next > cache->num_blocks)
      return set_error(ILPC_ENOSPC, "ilpc_prefix_match: batch needs %lld blocks, pool has %d",
                       (long long)next, cache->num_blocks);
    if (reg && cache->count + new_keys > cache->max_entries)
      return set_error(ILPC_ETABLE, "ilpc_prefix_match: %lld held + %lld new keys > capacity %lld",
                       (long long)cache->count, (long long)new_keys, (long long)cache->max_entries);
  }

  // Outputs: cached length, block table (hits, then fresh ids), keys.
  int32_t alloc = cache->next_block;
  for (int32_t r = 0; r < B; ++r) {
    const int64_t L = int64_t(cu_seqlens[r + 1]) - cu_seqlens[r];
    const int64_t res = reserve ? reserve[r] : 0;
    const int32_t n_total = int32_t((L + res + kBlock - 1) / kBlock);
    const int32_t n_full = int32_t(L / kBlock);
    const int32_t m = matched[r];
    int32_t* row = block_tables + int64_t(r) * max_blocks;
    for (int32_t b = 0; b < m; ++b) row[b] = hit_ids[size_t(hit_off[r] + b)];
    if (cache->lru) {
      for (int32_t b = m; b < n_total; ++b) row[b] = cache->take();
    } else {
      for (int32_t b = m; b < n_total; ++b) row[b] = alloc++;
    }
    for (int32_t b = n_total; b < max_blocks; ++b) row[b] = -1;
    cached_len[r] = kBlock * m;
    if (block_keys) {
      uint64_t* krow = block_keys + int64_t(r) * max_blocks;
      for (int32_t b = 0; b < n_full; ++b) krow[b] = keys[size_t(key_off[r] + b)];
      for (int32_t b = n_full; b < max_blocks; ++b) krow[b] = 0;
    }
  }

  // Commit: register new full blocks in request order, first writer wins.
  if (reg) {
    for (int32_t r = 0; r < B; ++r) {
      const int32_t n_full = int32_t(key_off[r + 1] - key_off[r]);
      const int32_t* row = block_tables + int64_t(r) * max_blocks;
      for (int32_t b = matched[r]; b < n_full; ++b) {
        const uint64_t key = keys[size_t(key_off[r] + b)];
        const uint64_t s = cache->probe(key);
        if (cache->keys[s] != 0) continue;
        cache->keys[s] = key;
        cache->vals[s] = row[b];
        ++cache->count;
        if (cache->lru)
          cache->bkey[row[b]] = key;
        else
          cache->journal.push_back(s);
      }
    }
  }
  cache->next_block = alloc;
  return ILPC_OK;
}

extern "C" int ilpc_cache_release(ilpc_cache* cache, const int32_t* block_tables, int32_t B,
                                  int32_t max_blocks) {
  if (!cache) return set_error(ILPC_EINVAL, "ilpc_cache_release: cache is NULL");
  if (!cache->lru)
    return set_error(ILPC_EUNSUP, "ilpc_cache_release: the cache was not made by ilpc_cache_create_lru");
  if (B < 0) return set_error(ILPC_EINVAL, "ilpc_cache_release: B < 0");
  if (B == 0) return ILPC_OK;
  if (!block_tables || max_blocks < 1)
    return set_error(ILPC_EINVAL, "ilpc_cache_release: NULL block_tables or max_blocks < 1");
  // Validate: ids in range, and no block released more often than it is held.
  // mark[] counts this call's releases per block; it is cleared again below.
  int rc = ILPC_OK;
  int32_t rows_seen = 0;
  for (; rows_seen < B && rc == ILPC_OK; ++rows_seen) {
    const int32_t* row = block_tables + int64_t(rows_seen) * max_blocks;
    for (int32_t k = 0; k < max_blocks && row[k] != -1; ++k) {
      const int32_t b = row[k];
      if (b < 0 || b >= cache->num_blocks) {
        rc = set_error(ILPC_EINVAL, "ilpc_cache_release: block id %d out of range", b);
        break;
      }
      if (++cache->mark[b] > cache->ref[b]) {
        rc = set_error(ILPC_EINVAL, "ilpc_cache_release: block %d released more often than held", b);
        break;
      }
    }
  }
  for (int32_t r = 0; r < rows_seen; ++r) {
    const int32_t* row = block_tables + int64_t(r) * max_blocks;
    for (int32_t k = 0; k < max_blocks && row[k] != -1; ++k)
      if (row[k] >= 0 && row[k] < cache->num_blocks) cache->mark[row[k]] = 0;
  }
  if (rc != ILPC_OK) return rc;
  // Release each row from its last block to its first.
  for (int32_t r = 0; r < B; ++r) {
    const int32_t* row = block_tables + int64_t(r) * max_blocks;
    int32_t len = 0;
    while (len < max_blocks && row[len] != -1) ++len;
    for (int32_t k = len - 1; k >= 0; --k) {
      const int32_t b = row[k];
      if (--cache->ref[b] > 0) continue;
      --cache->in_use;
      if (cache->bkey[b] != 0)
        cache->lru_push_tail(b);
      else
        cache->fq_push(b);
    }
  }
  return ILPC_OK;
}

extern "C" int ilpc_cache_touch(ilpc_cache* cache, const int32_t* block_ids, int32_t n) {
  if (!cache) return set_error(ILPC_EINVAL, "ilpc_cache_touch: cache is NULL");
  if (!cache->lru)
    return set_error(ILPC_EUNSUP, "ilpc_cache_touch: the cache was not made by ilpc_cache_create_lru");
  if (n < 0) return set_error(ILPC_EINVAL, "ilpc_cache_touch: n < 0");
  if (n > 0 && !block_ids) return set_error(ILPC_EINVAL, "ilpc_cache_touch: block_ids is NULL");
  for (int32_t i = 0; i < n; ++i) {
    const int32_t b = block_ids[i];
    if (b != -1 && (b < 0 || b >= cache->num_blocks))
      return set_error(ILPC_EINVAL, "ilpc_cache_touch: block id %d out of range", b);
  }
  for (int32_t i = 0; i < n; ++i) {
    const int32_t b = block_ids[i];
    if (b == -1 || cache->ref[b] != 0 || cache->bkey[b] == 0) continue;
    cache->lru_unlink(b);
    cache->lru_push_tail(b);
  }
  return ILPC_OK;
}

extern "C" int ilpc_cache_usage(const ilpc_cache* cache, int64_t usage[4]) {
  if (!cache || !usage) return set_error(ILPC_EINVAL, "ilpc_cache_usage: NULL argument");
  if (cache->lru) {
    usage[0] = cache->in_use;
    usage[1] = cache->n_cached;
    usage[2] = cache->fq_size;
    usage[3] = cache->evictions;
  } else {
    usage[0] = cache->next_block;
    usage[1] = 0;
    usage[2] = cache->num_blocks - cache->next_block;
    usage[3] = 0;
  }
  return ILPC_OK;
}

extern "C" int ilpc_cache_lru_order(const ilpc_cache* cache, int32_t* block_ids, int32_t max_ids,
                                    int32_t* n_cached) {
  if (!cache || !n_cached) return set_error(ILPC_EINVAL, "ilpc_cache_lru_order: NULL argument");
  if (max_ids < 0 || (max_ids > 0 && !block_ids))
    return set_error(ILPC_EINVAL, "ilpc_cache_lru_order: bad output buffer");
  *n_cached = cache->lru ? int32_t(cache->n_cached) : 0;
  int32_t k = 0;
  if (cache->lru)
    for (int32_t b = cache->lru_head; b >= 0 && k < max_ids; b = cache->nxt[b]) block_ids[k++] = b;
  return ILPC_OK;
}
