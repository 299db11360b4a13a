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
#include <cstdint>
#include <cstring>
#include <new>
#include <unordered_map>
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
  std::unordered_map<uint64_t, std::vector<int32_t>> by_key;    // set key -> slots
  std::unordered_map<int32_t, std::vector<int32_t>> by_first;   // first template -> slots

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
  static void erase_from(std::vector<int32_t>& v, int32_t s) {
    for (size_t i = 0; i < v.size(); ++i)
      if (v[i] == s) {
        v[i] = v.back();
        v.pop_back();
        return;
      }
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
    auto it = by_key.find(key[s]);
    erase_from(it->second, s);
    if (it->second.empty()) by_key.erase(it);
    auto jt = by_first.find(tmpl[size_t(s) * n]);
    erase_from(jt->second, s);
    if (jt->second.empty()) by_first.erase(jt);
    live[s] = 0;
    next[s] = free_head;
    free_head = s;
    --size;
  }
  int32_t find(const int32_t* t, const int32_t* d, uint64_t k) const {
    auto it = by_key.find(k);
    if (it == by_key.end()) return -1;
    for (int32_t s : it->second)
      if (!memcmp(&tmpl[size_t(s) * n], t, sizeof(int32_t) * n) &&
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
    by_key[k].push_back(s);
    by_first[t[0]].push_back(s);
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
  if (!t) return set_error(ILPC_EINVAL, "ilpc_pair_create: out of host memory");
  try {
    t->init(capacity, n_demos);
  } catch (...) {
    delete t;
    return set_error(ILPC_EINVAL, "ilpc_pair_create: out of host memory");
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
  try {
    // distinct templates of the current set with their multiplicities
    std::vector<int32_t> tk, tc, avail, used(n);
    std::vector<int32_t> final_t(n), final_d(n);
    for (int32_t b = 0; b < B; ++b) {
      const int32_t* ct = templates + size_t(b) * n;
      const int32_t* cd = demos + size_t(b) * n;
      tk.clear();
      tc.clear();
      for (int32_t i = 0; i < n; ++i) {
        size_t j = 0;
        while (j < tk.size() && tk[j] != ct[i]) ++j;
        if (j == tk.size()) {
          tk.push_back(ct[i]);
          tc.push_back(0);
        }
        ++tc[j];
      }
      // matching: candidates are the sets starting with a template of the current set
      int32_t best = -1, best_k = 0;
      for (size_t u = 0; u < tk.size(); ++u) {
        auto it = T.by_first.find(tk[u]);
        if (it == T.by_first.end()) continue;
        for (int32_t s : it->second) {
          avail = tc;
          const int32_t* ht = &T.tmpl[size_t(s) * n];
          int32_t k = 0;
          for (; k < n; ++k) {
            size_t j = 0;
            while (j < tk.size() && tk[j] != ht[k]) ++j;
            if (j == tk.size() || avail[j] == 0) break;
            --avail[j];
          }
          if (k > best_k || (k == best_k && k > 0 && T.stamp[s] > T.stamp[best])) {
            best = s;
            best_k = k;
          }
        }
      }
      int32_t* ot = out_templates + size_t(b) * n;
      int32_t* od = out_demos + size_t(b) * n;
      if (best_k == n) {  // rule (1): the target set as it is, refreshed
        memcpy(final_t.data(), &T.tmpl[size_t(best) * n], sizeof(int32_t) * n);
        memcpy(final_d.data(), &T.demo[size_t(best) * n], sizeof(int32_t) * n);
        T.touch(best);
      } else if (best_k == 0) {  // rule (2): unchanged, appended
        memcpy(final_t.data(), ct, sizeof(int32_t) * n);
        memcpy(final_d.data(), cd, sizeof(int32_t) * n);
        T.append(final_t.data(), final_d.data());
      } else {  // rule (3): modified and reordered, appended
        std::fill(used.begin(), used.end(), 0);
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
        T.append(final_t.data(), final_d.data());
      }
      memcpy(ot, final_t.data(), sizeof(int32_t) * n);
      memcpy(od, final_d.data(), sizeof(int32_t) * n);
      pmc[b] = best_k;
    }
  } catch (...) {
    return set_error(ILPC_EINVAL, "ilpc_pair_refine: out of host memory");
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
