// Prefix-aware refinement of in-context demonstrations (InferLog section 3.2,
// "Prefix-Aware ICL Refinement" and "ICL Table Management"), host side.
//
// A demonstration is a (template id, demonstration id) pair; the
// demonstration id stands for the concrete log text and so for its tokens.
// The ICL table holds the demonstration sets of past requests in
// least-recently-used order.  For a new request:
//   matching:   the past set with the largest prefix-matching count (PMC:
//               the number of its leading demonstrations whose templates all
//               occur in the current set, each current demonstration serving
//               at most one of them) is the target; ties go to the most
//               recently used set, and a PMC of 0 means no target;
//   modifying:  each of the target's first PMC demonstrations replaces the
//               first not yet replaced current demonstration of its template;
//   reordering: the final set is the target's first PMC demonstrations in the
//               target's order, then the remaining current demonstrations in
//               their order.
// Table update (the paper's three rules): PMC = N reuses the target and moves
// it to the most-recent end; PMC = 0 appends the current set unchanged;
// otherwise the refined set is appended and the target keeps its place.  A
// set already in the table is stored once (appending it again refreshes it).
// Beyond the capacity, the least recently used set is evicted.
//
// Only past sets whose first template occurs in the current set can have a
// PMC above 0, so the table keeps an index from first template to sets, and a
// request looks at those sets only.
//
// Every structure the table uses (the slot arrays, both hash indexes and the
// per-request scratch) is sized when the table is created, so refinement
// allocates nothing: a call either is refused before it changes anything or
// completes.
#include <algorithm>
#include <cstdint>
#include <cstring>
#include <new>
#include <vector>

#include "../../include/ilpc.h"
#include "ilpc_internal.h"

namespace {

constexpr int32_t kMaxDemos = 4096;      // demonstrations per set accepted
constexpr int32_t kMaxCapacity = 1 << 24;  // sets per table accepted

inline uint64_t mix64(uint64_t x) {  // MurmurHash3 64-bit finaliser (Appleby, public domain)
  x ^= x >> 33;
  x *= 0xFF51AFD7ED558CCDull;
  x ^= x >> 33;
  x *= 0xC4CEB9FE1A85EC53ull;
  x ^= x >> 33;
  return x;
}

uint64_t set_key(const int32_t* tmpl, const int32_t* demo, int32_t n) {
  uint64_t h = 0x6A09E667F3BCC908ull;
  for (int32_t i = 0; i < n; ++i)
    h = mix64(h ^ (uint64_t(uint32_t(tmpl[i])) | (uint64_t(uint32_t(demo[i])) << 32)) ^ uint64_t(i));
  return h;
}

// A hash index over the table's slots: buckets of doubly linked slot chains,
// all arrays sized for the capacity at creation.
struct SlotIndex {
  uint64_t mask = 0;
  std::vector<int32_t> bucket, nxt, prv;  // bucket heads; per-slot chain links (-1: none)

  void init(int32_t cap) {
    uint64_t nb = 1;
    while (nb < 2 * uint64_t(cap)) nb <<= 1;
    mask = nb - 1;
    bucket.assign(size_t(nb), -1);
    nxt.assign(size_t(cap), -1);
    prv.assign(size_t(cap), -1);
  }
  void clear() { std::fill(bucket.begin(), bucket.end(), -1); }
  int32_t head(uint64_t h) const { return bucket[size_t(h & mask)]; }
  void insert(uint64_t h, int32_t s) {
    int32_t& b = bucket[size_t(h & mask)];
    prv[s] = -1;
    nxt[s] = b;
    if (b >= 0) prv[b] = s;
    b = s;
  }
  void erase(uint64_t h, int32_t s) {
    if (prv[s] >= 0) nxt[prv[s]] = nxt[s];
    else bucket[size_t(h & mask)] = nxt[s];
    if (nxt[s] >= 0) prv[nxt[s]] = prv[s];
    prv[s] = nxt[s] = -1;
  }
};

inline uint64_t first_hash(int32_t t) { return mix64(uint64_t(uint32_t(t)) ^ 0x3C6EF372FE94F82Bull); }

}  // namespace

struct ilpc_pair_table {
  int32_t capacity = 0, n = 0;
  // Slot s holds one set: tmpl/demo [s*n, s*n+n), its recency stamp, its key,
  // and its neighbours in LRU order (-1: none).  Free slots are chained on `free_head`.
  std::vector<int32_t> tmpl, demo, prev, next;
  std::vector<uint64_t> stamp, key;
  std::vector<uint8_t> live;
  int32_t head = -1, tail = -1, size = 0, free_head = -1;
  uint64_t clock = 0;
  SlotIndex by_key;    // set key -> slots (contents compared on a hit)
  SlotIndex by_first;  // first template -> slots (first template compared on a hit)
  // Per-request scratch: distinct templates of the current set and their
  // counts, the counts left while matching, replaced flags, the final set.
  std::vector<int32_t> w_tk, w_tc, w_avail, w_used, w_ft, w_fd;

  void init(int32_t cap, int32_t n_demos) {
    capacity = cap;
    n = n_demos;
    tmpl.assign(size_t(cap) * n, 0);
    demo.assign(size_t(cap) * n, 0);
    prev.assign(cap, -1);
    next.assign(cap, -1);
    stamp.assign(cap, 0);
    key.assign(cap, 0);
    live.assign(cap, 0);
    by_key.init(cap);
    by_first.init(cap);
    for (auto* v : {&w_tk, &w_tc, &w_avail, &w_used, &w_ft, &w_fd}) v->assign(size_t(n), 0);
    clear();
  }
  void clear() {
    head = tail = -1;
    size = 0;
    clock = 0;
    by_key.clear();
    by_first.clear();
    std::fill(live.begin(), live.end(), 0);
    free_head = capacity > 0 ? 0 : -1;
    for (int32_t s = 0; s < capacity; ++s) next[s] = s + 1 < capacity ? s + 1 : -1;
  }
  void unlink(int32_t s) {
    if (prev[s] >= 0) next[prev[s]] = next[s];
    else head = next[s];
    if (next[s] >= 0) prev[next[s]] = prev[s];
    else tail = prev[s];
    prev[s] = next[s] = -1;
  }
  void link_tail(int32_t s) {
    prev[s] = tail;
    next[s] = -1;
    if (tail >= 0) next[tail] = s;
    else head = s;
    tail = s;
    stamp[s] = ++clock;
  }
  void touch(int32_t s) {  // move to the most-recent end
    unlink(s);
    link_tail(s);
  }
  void evict_head() {
    const int32_t s = head;
    unlink(s);
    by_key.erase(key[s], s);
    by_first.erase(first_hash(tmpl[size_t(s) * n]), s);
    live[s] = 0;
    next[s] = free_head;
    free_head = s;
    --size;
  }
  int32_t find(const int32_t* t, const int32_t* d, uint64_t k) const {
    for (int32_t s = by_key.head(k); s >= 0; s = by_key.nxt[s])
      if (key[s] == k && !memcmp(&tmpl[size_t(s) * n], t, sizeof(int32_t) * n) &&
          !memcmp(&demo[size_t(s) * n], d, sizeof(int32_t) * n))
        return s;
    return -1;
  }
  // Append a set at the most-recent end (refresh it if already stored), then
  // evict from the least-recent end beyond the capacity.
  void append(const int32_t* t, const int32_t* d) {
    const uint64_t k = set_key(t, d, n);
    const int32_t found = find(t, d, k);
    if (found >= 0) {
      touch(found);
      return;
    }
    if (free_head < 0) evict_head();  // full: the new set's place frees the oldest
    const int32_t s = free_head;
    free_head = next[s];
    memcpy(&tmpl[size_t(s) * n], t, sizeof(int32_t) * n);
    memcpy(&demo[size_t(s) * n], d, sizeof(int32_t) * n);
    key[s] = k;
    live[s] = 1;
    link_tail(s);
    by_key.insert(k, s);
    by_first.insert(first_hash(t[0]), s);
    ++size;
  }
};

extern "C" int ilpc_pair_create(int32_t capacity, int32_t n_demos, ilpc_pair_table** out) {
  using ilpc::set_error;
  if (!out) return set_error(ILPC_EINVAL, "ilpc_pair_create: out is NULL");
  *out = nullptr;
  if (capacity < 1 || capacity > kMaxCapacity)
    return set_error(ILPC_EINVAL, "ilpc_pair_create: capacity %d outside [1, %d]", capacity, kMaxCapacity);
  if (n_demos < 1 || n_demos > kMaxDemos)
    return set_error(ILPC_EINVAL, "ilpc_pair_create: n_demos %d outside [1, %d]", n_demos, kMaxDemos);
  ilpc_pair_table* t = new (std::nothrow) ilpc_pair_table();
  if (!t) return set_error(ILPC_ENOSPC, "ilpc_pair_create: out of host memory");
  try {
    t->init(capacity, n_demos);
  } catch (...) {
    delete t;
    return set_error(ILPC_ENOSPC, "ilpc_pair_create: out of host memory");
  }
  *out = t;
  return ILPC_OK;
}

extern "C" void ilpc_pair_destroy(ilpc_pair_table* table) { delete table; }

extern "C" int ilpc_pair_reset(ilpc_pair_table* table) {
  if (!table) return ilpc::set_error(ILPC_EINVAL, "ilpc_pair_reset: table is NULL");
  table->clear();
  return ILPC_OK;
}

extern "C" int ilpc_pair_refine(ilpc_pair_table* table, const int32_t* templates, const int32_t* demos,
                                int32_t B, int32_t* out_templates, int32_t* out_demos, int32_t* pmc) {
  using ilpc::set_error;
  if (!table) return set_error(ILPC_EINVAL, "ilpc_pair_refine: table is NULL");
  if (B < 0) return set_error(ILPC_EINVAL, "ilpc_pair_refine: negative batch size");
  if (B == 0) return ILPC_OK;
  if (!templates || !demos || !out_templates || !out_demos || !pmc)
    return set_error(ILPC_EINVAL, "ilpc_pair_refine: NULL pointer");
  ilpc_pair_table& T = *table;
  const int32_t n = T.n;
  int32_t* tk = T.w_tk.data();  // distinct templates of the current set
  int32_t* tc = T.w_tc.data();  // their multiplicities
  int32_t* avail = T.w_avail.data();
  int32_t* used = T.w_used.data();
  int32_t* final_t = T.w_ft.data();
  int32_t* final_d = T.w_fd.data();
  for (int32_t b = 0; b < B; ++b) {
    const int32_t* ct = templates + size_t(b) * n;
    const int32_t* cd = demos + size_t(b) * n;
    int32_t nt = 0;
    for (int32_t i = 0; i < n; ++i) {
      int32_t j = 0;
      while (j < nt && tk[j] != ct[i]) ++j;
      if (j == nt) {
        tk[nt] = ct[i];
        tc[nt++] = 0;
      }
      ++tc[j];
    }
    // matching: candidates are the sets starting with a template of the current set
    int32_t best = -1, best_k = 0;
    for (int32_t u = 0; u < nt; ++u) {
      for (int32_t s = T.by_first.head(first_hash(tk[u])); s >= 0; s = T.by_first.nxt[s]) {
        const int32_t* ht = &T.tmpl[size_t(s) * n];
        if (ht[0] != tk[u]) continue;  // another template in the same bucket
        std::copy(tc, tc + nt, avail);
        int32_t k = 0;
        for (; k < n; ++k) {
          int32_t j = 0;
          while (j < nt && tk[j] != ht[k]) ++j;
          if (j == nt || avail[j] == 0) break;
          --avail[j];
        }
        if (k > best_k || (k == best_k && k > 0 && T.stamp[s] > T.stamp[best])) {
          best = s;
          best_k = k;
        }
      }
    }
    if (best_k == n) {  // rule (1): the target set as it is, refreshed
      memcpy(final_t, &T.tmpl[size_t(best) * n], sizeof(int32_t) * n);
      memcpy(final_d, &T.demo[size_t(best) * n], sizeof(int32_t) * n);
      T.touch(best);
    } else if (best_k == 0) {  // rule (2): unchanged, appended
      memcpy(final_t, ct, sizeof(int32_t) * n);
      memcpy(final_d, cd, sizeof(int32_t) * n);
      T.append(final_t, final_d);
    } else {  // rule (3): modified and reordered, appended
      std::fill(used, used + n, 0);
      const int32_t* ht = &T.tmpl[size_t(best) * n];
      const int32_t* hd = &T.demo[size_t(best) * n];
      for (int32_t k = 0; k < best_k; ++k) {
        for (int32_t i = 0; i < n; ++i)
          if (!used[i] && ct[i] == ht[k]) {
            used[i] = 1;
            break;
          }
        final_t[k] = ht[k];
        final_d[k] = hd[k];
      }
      int32_t m = best_k;
      for (int32_t i = 0; i < n; ++i)
        if (!used[i]) {
          final_t[m] = ct[i];
          final_d[m] = cd[i];
          ++m;
        }
      T.append(final_t, final_d);
    }
    memcpy(out_templates + size_t(b) * n, final_t, sizeof(int32_t) * n);
    memcpy(out_demos + size_t(b) * n, final_d, sizeof(int32_t) * n);
    pmc[b] = best_k;
  }
  return ILPC_OK;
}

extern "C" int ilpc_pair_entries(const ilpc_pair_table* table, int32_t* templates, int32_t* demos,
                                 int32_t max_entries, int32_t* n_entries) {
  using ilpc::set_error;
  if (!table || !n_entries) return set_error(ILPC_EINVAL, "ilpc_pair_entries: NULL pointer");
  if (max_entries < 0) return set_error(ILPC_EINVAL, "ilpc_pair_entries: negative max_entries");
  *n_entries = table->size;
  if (table->size > max_entries)
    return set_error(ILPC_EINVAL, "ilpc_pair_entries: %d entries do not fit in %d", table->size, max_entries);
  if (table->size > 0 && (!templates || !demos)) return set_error(ILPC_EINVAL, "ilpc_pair_entries: NULL pointer");
  const int32_t n = table->n;
  int32_t e = 0;
  for (int32_t s = table->head; s >= 0; s = table->next[s], ++e) {
    memcpy(templates + size_t(e) * n, &table->tmpl[size_t(s) * n], sizeof(int32_t) * n);
    memcpy(demos + size_t(e) * n, &table->demo[size_t(s) * n], sizeof(int32_t) * n);
  }
  return ILPC_OK;
}
