// Host-side stress of the prefix cache (bump and LRU) and the ICL table, built
// with AddressSanitizer and UndefinedBehaviorSanitizer by
// tests/test_host_sanitize.py: random batches with reuse, reserves and flags,
// releases, touches, LRU listings, usage checks, checkpoints and rollbacks,
// resets, refinements with repeated and negative template ids, and calls that
// must be refused.
#include <cstdio>
#include <cstdlib>
#include <random>
#include <vector>
#include "ilpc.h"

int main() {
  std::mt19937 rng(1234);
  auto U = [&](int lo, int hi) { return std::uniform_int_distribution<int>(lo, hi)(rng); };
  for (int lru = 0; lru < 2; ++lru) {
    ilpc_cache* c = nullptr;
    const int nb = lru ? 64 : 200000;
    if (lru) {
      if (ilpc_cache_create_lru(nb, 16, 8, &c)) { printf("create lru failed %s\n", ilpc_last_error()); return 1; }
    } else if (ilpc_cache_create(nb, 16, 18, &c)) {
      return 1;
    }
    std::vector<std::vector<int>> pieces(6);
    for (auto& p : pieces) { p.resize(U(5, 60)); for (auto& t : p) t = U(0, 50); }
    std::vector<std::vector<int32_t>> live;
    const int mb = 16;
    for (int step = 0; step < 3000; ++step) {
      const int B = U(0, 4);
      std::vector<int32_t> toks, cu(1, 0), res(B);
      for (int r = 0; r < B; ++r) {
        const int k = U(1, 3);
        for (int i = 0; i < k; ++i) { auto& p = pieces[U(0, 5)]; toks.insert(toks.end(), p.begin(), p.end()); }
        toks.push_back(U(0, 50));
        if ((int)(toks.size() - cu.back()) + 0 > mb * 16 - 16) toks.resize(cu.back() + mb * 16 - 16);
        cu.push_back((int32_t)toks.size());
        res[r] = U(0, 8);
      }
      std::vector<int32_t> cached(B), tables(size_t(B) * mb);
      std::vector<uint64_t> keys(size_t(B) * mb);
      const uint32_t flags = U(0, 9) == 0 ? U(0, 3) : 0;
      const int rc = ilpc_prefix_match(c, toks.data(), cu.data(), B, U(0, 1) ? res.data() : nullptr, mb, flags,
                                       cached.data(), tables.data(), U(0, 1) ? keys.data() : nullptr);
      if (rc == ILPC_OK && lru)
        for (int r = 0; r < B; ++r) live.emplace_back(tables.begin() + size_t(r) * mb, tables.begin() + size_t(r + 1) * mb);
      if (lru && (rc == ILPC_ENOSPC || U(0, 2) == 0) && !live.empty()) {
        const int k = U(1, (int)live.size());
        std::vector<int32_t> rows;
        for (int i = 0; i < k; ++i) { rows.insert(rows.end(), live.back().begin(), live.back().end()); live.pop_back(); }
        if (ilpc_cache_release(c, rows.data(), k, mb)) { printf("release failed %s\n", ilpc_last_error()); return 1; }
      }
      if (lru && U(0, 5) == 0) {
        int32_t ids[5]; for (auto& x : ids) x = U(-1, nb - 1);
        ilpc_cache_touch(c, ids, 5);
        int32_t bad = nb; if (ilpc_cache_touch(c, &bad, 1) == ILPC_OK) return 2;
        std::vector<int32_t> order(nb); int32_t n = 0;
        ilpc_cache_lru_order(c, order.data(), U(0, nb), &n);
        int64_t u[4]; ilpc_cache_usage(c, u);
        if (u[0] + u[1] + u[2] != nb) { printf("usage mismatch\n"); return 3; }
        int32_t badrow[2] = {nb, -1}; if (ilpc_cache_release(c, badrow, 1, 2) == ILPC_OK) return 6;
      }
      if (!lru && U(0, 50) == 0) { int64_t m[2]; ilpc_cache_checkpoint(c, m); ilpc_prefix_match(c, toks.data(), cu.data(), B, nullptr, mb, 0, cached.data(), tables.data(), nullptr); ilpc_cache_rollback(c, m); }
      if (U(0, 400) == 0) { ilpc_cache_reset(c); live.clear(); }
    }
    ilpc_cache_destroy(c);
  }
  // ICL table
  for (int cap : {1, 3, 17, 200}) {
    for (int n : {1, 3, 5, 8}) {
      ilpc_pair_table* t = nullptr;
      if (ilpc_pair_create(cap, n, &t)) return 4;
      for (int step = 0; step < 400; ++step) {
        const int B = U(0, 5);
        std::vector<int32_t> tp(size_t(B) * n), dm(size_t(B) * n), ot(tp.size()), od(tp.size()), pmc(B);
        for (size_t i = 0; i < tp.size(); ++i) { tp[i] = U(-3, 9); dm[i] = tp[i] * 7 + U(0, 2); }
        if (ilpc_pair_refine(t, tp.data(), dm.data(), B, ot.data(), od.data(), pmc.data())) return 5;
        std::vector<int32_t> et(size_t(cap) * n), ed(et.size()); int32_t ne = 0;
        ilpc_pair_entries(t, et.data(), ed.data(), U(0, cap), &ne);
        if (U(0, 100) == 0) ilpc_pair_reset(t);
      }
      ilpc_pair_destroy(t);
    }
  }
  printf("host fuzz ok\n");
  return 0;
}
