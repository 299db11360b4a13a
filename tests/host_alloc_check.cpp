// Host allocation-failure check of the library's host entry points, built
// with g++ by tests/test_host_alloc.py.  The global operator new is replaced
// by one that can be told to fail from the k-th allocation on, so every
// allocation a call makes can be made to fail in turn:
//   * ilpc_pair_create fails with ILPC_ENOSPC and a NULL handle;
//   * ilpc_pair_refine allocates nothing at all (every allocation would fail
//     and the call still completes with the same results as without);
//   * ilpc_prefix_match (bump and LRU caches) either completes or fails with
//     ILPC_ENOSPC leaving the cache as it was: the same batch run afterwards
//     gives the tables, keys, usage and LRU order of a cache that never saw
//     the failure.
#include <cstdio>
#include <cstdlib>
#include <new>
#include <random>
#include <vector>

#include "ilpc.h"

static long g_count = 0;       // allocations attempted so far
static long g_fail_from = -1;  // attempts numbered >= this one fail (-1: none)

void* operator new(std::size_t n) {
  const long i = g_count++;
  if (g_fail_from >= 0 && i >= g_fail_from) throw std::bad_alloc();
  void* p = std::malloc(n ? n : 1);
  if (!p) throw std::bad_alloc();
  return p;
}
void* operator new[](std::size_t n) { return operator new(n); }
void* operator new(std::size_t n, const std::nothrow_t&) noexcept {
  try {
    return operator new(n);
  } catch (...) {
    return nullptr;
  }
}
void* operator new[](std::size_t n, const std::nothrow_t&) noexcept {
  try {
    return operator new(n);
  } catch (...) {
    return nullptr;
  }
}
void operator delete(void* p) noexcept { std::free(p); }
void operator delete[](void* p) noexcept { std::free(p); }
void operator delete(void* p, std::size_t) noexcept { std::free(p); }
void operator delete[](void* p, std::size_t) noexcept { std::free(p); }

#define CHECK(c)                                                       \
  do {                                                                 \
    if (!(c)) {                                                        \
      std::printf("FAILED %s:%d: %s (%s)\n", __FILE__, __LINE__, #c,   \
                  ilpc_last_error());                                  \
      return 1;                                                        \
    }                                                                  \
  } while (0)

namespace {

struct Batch {
  std::vector<int32_t> toks, cu, res;
};

// Prompts made of a few shared pieces, so batches hit each other's blocks.
std::vector<Batch> make_batches(std::mt19937& rng, int n_batches, int mb) {
  auto U = [&](int lo, int hi) { return std::uniform_int_distribution<int>(lo, hi)(rng); };
  std::vector<std::vector<int32_t>> pieces(5);
  for (auto& p : pieces) {
    p.resize(U(10, 50));
    for (auto& t : p) t = U(0, 40);
  }
  std::vector<Batch> out(n_batches);
  for (auto& b : out) {
    const int B = U(1, 4);
    b.cu.assign(1, 0);
    for (int r = 0; r < B; ++r) {
      const int k = U(1, 3);
      for (int i = 0; i < k; ++i) {
        auto& p = pieces[U(0, 4)];
        b.toks.insert(b.toks.end(), p.begin(), p.end());
      }
      b.toks.push_back(U(0, 40));
      if (int(b.toks.size()) - b.cu.back() > mb * 16 - 32) b.toks.resize(b.cu.back() + mb * 16 - 32);
      b.cu.push_back(int32_t(b.toks.size()));
      b.res.push_back(U(0, 16));
    }
  }
  return out;
}

struct State {
  std::vector<int32_t> cached, tables, lru;
  std::vector<uint64_t> keys;
  int64_t stats[4] = {}, usage[4] = {};
  bool operator==(const State& o) const {
    for (int i = 0; i < 4; ++i)
      if (stats[i] != o.stats[i] || usage[i] != o.usage[i]) return false;
    return cached == o.cached && tables == o.tables && keys == o.keys && lru == o.lru;
  }
};

// Match batch b on c and record the outputs and the cache's observable state.
// fail_at >= 0: the call's allocations from that one on fail.
int run_match(ilpc_cache* c, bool lru, const Batch& b, int mb, State* st, long fail_at = -1) {
  const int B = int(b.cu.size()) - 1;
  st->cached.assign(B, 0);
  st->tables.assign(size_t(B) * mb, 0);
  st->keys.assign(size_t(B) * mb, 0);
  if (fail_at >= 0) g_fail_from = g_count + fail_at;
  const int rc = ilpc_prefix_match(c, b.toks.data(), b.cu.data(), B, b.res.data(), mb, 0, st->cached.data(),
                                   st->tables.data(), st->keys.data());
  g_fail_from = -1;
  if (rc != ILPC_OK) return rc;
  ilpc_cache_stats(c, st->stats);
  if (lru) {
    ilpc_cache_usage(c, st->usage);
    st->lru.assign(4096, 0);
    int32_t n = 0;
    ilpc_cache_lru_order(c, st->lru.data(), int32_t(st->lru.size()), &n);
    st->lru.resize(n);
  }
  return ILPC_OK;
}

ilpc_cache* make_cache(bool lru) {
  ilpc_cache* c = nullptr;
  const int rc = lru ? ilpc_cache_create_lru(96, 16, 9, &c) : ilpc_cache_create(4000, 16, 12, &c);
  return rc == ILPC_OK ? c : nullptr;
}

}  // namespace

int main() {
  // ilpc_pair_create: every allocation it makes fails in turn.
  int create_points = 0;
  for (long k = 0;; ++k) {
    ilpc_pair_table* t = reinterpret_cast<ilpc_pair_table*>(&k);
    g_fail_from = g_count + k;
    const int rc = ilpc_pair_create(64, 5, &t);
    g_fail_from = -1;
    if (rc == ILPC_OK) {
      ilpc_pair_destroy(t);
      break;
    }
    CHECK(rc == ILPC_ENOSPC);
    CHECK(t == nullptr);
    ++create_points;
  }
  CHECK(create_points > 0);

  // ilpc_pair_refine: no allocation at all, at any table fill or eviction.
  {
    std::mt19937 rng(7);
    auto U = [&](int lo, int hi) { return std::uniform_int_distribution<int>(lo, hi)(rng); };
    const int n = 5;
    ilpc_pair_table *a = nullptr, *b = nullptr;
    CHECK(ilpc_pair_create(16, n, &a) == ILPC_OK);
    CHECK(ilpc_pair_create(16, n, &b) == ILPC_OK);
    for (int step = 0; step < 400; ++step) {
      const int B = U(1, 8);
      std::vector<int32_t> t(size_t(B) * n), d(size_t(B) * n);
      for (int i = 0; i < B * n; ++i) {
        t[i] = U(0, 3) == 0 ? U(-3, 12) : U(0, 4);  // hot templates, repeats, negatives
        d[i] = U(0, 200);
      }
      std::vector<int32_t> ta(t.size()), da(t.size()), pa(B), tb(t.size()), db(t.size()), pb(B);
      const long before = g_count;  // (nothing below allocates until the call returns)
      g_fail_from = g_count;  // any allocation from here on throws
      const int rc = ilpc_pair_refine(a, t.data(), d.data(), B, ta.data(), da.data(), pa.data());
      g_fail_from = -1;
      CHECK(rc == ILPC_OK);
      CHECK(g_count == before);
      CHECK(ilpc_pair_refine(b, t.data(), d.data(), B, tb.data(), db.data(), pb.data()) == ILPC_OK);
      CHECK(ta == tb && da == db && pa == pb);
    }
    std::vector<int32_t> ea(16 * n), fa(16 * n), eb(16 * n), fb(16 * n);
    int32_t na = 0, nb = 0;
    CHECK(ilpc_pair_entries(a, ea.data(), fa.data(), 16, &na) == ILPC_OK);
    CHECK(ilpc_pair_entries(b, eb.data(), fb.data(), 16, &nb) == ILPC_OK);
    CHECK(na == nb && ea == eb && fa == fb);
    ilpc_pair_destroy(a);
    ilpc_pair_destroy(b);
  }

  // ilpc_prefix_match: fail each allocation of batch i in turn, after the
  // batches before it; the cache must be as if the failed call never happened.
  long match_points = 0;
  for (int lru = 0; lru < 2; ++lru) {
    std::mt19937 rng(11 + lru);
    const int mb = 12;
    const std::vector<Batch> batches = make_batches(rng, 24, mb);
    std::vector<State> expect(batches.size());
    {
      ilpc_cache* c = make_cache(lru);
      CHECK(c);
      for (size_t i = 0; i < batches.size(); ++i) {
        CHECK(run_match(c, lru, batches[i], mb, &expect[i]) == ILPC_OK);
        if (lru && i % 3 == 2) CHECK(ilpc_cache_release(c, expect[i].tables.data(),
                                                        int32_t(expect[i].cached.size()), mb) == ILPC_OK);
      }
      ilpc_cache_destroy(c);
    }
    for (size_t i = 0; i < batches.size(); ++i) {
      for (long k = 0;; ++k) {
        ilpc_cache* c = make_cache(lru);
        CHECK(c);
        State st;
        for (size_t j = 0; j < i; ++j) {
          CHECK(run_match(c, lru, batches[j], mb, &st) == ILPC_OK);
          if (lru && j % 3 == 2)
            CHECK(ilpc_cache_release(c, st.tables.data(), int32_t(st.cached.size()), mb) == ILPC_OK);
        }
        const int rc = run_match(c, lru, batches[i], mb, &st, k);
        if (rc == ILPC_OK) {
          CHECK(st == expect[i]);
          ilpc_cache_destroy(c);
          break;
        }
        CHECK(rc == ILPC_ENOSPC);
        ++match_points;
        // the failed call changed nothing: this batch and the next match as expected
        CHECK(run_match(c, lru, batches[i], mb, &st) == ILPC_OK);
        CHECK(st == expect[i]);
        if (i + 1 < batches.size()) {
          if (lru && i % 3 == 2)
            CHECK(ilpc_cache_release(c, st.tables.data(), int32_t(st.cached.size()), mb) == ILPC_OK);
          CHECK(run_match(c, lru, batches[i + 1], mb, &st) == ILPC_OK);
          CHECK(st == expect[i + 1]);
        }
        ilpc_cache_destroy(c);
      }
    }
  }
  CHECK(match_points > 0);
  std::printf("host alloc ok: create %d, match %ld failure points\n", create_points, match_points);
  return 0;
}
