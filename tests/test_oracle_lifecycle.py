"""Pins of the block-lifecycle oracle (oracle/lifecycle_ref.py).

* with nothing ever released it is the bump-allocator cache of
  oracle/prefix_ref.py (itself pinned to the paper's example and brute force);
* a small scenario worked by hand: released prompts are evicted tail first, the
  free queue is used before any eviction, a hit revives a cached block, touch
  reorders the LRU list, a batch whose hits pin the only cached blocks is
  refused;
* a brute-force model keyed by exact token prefixes (no hashing) with
  time stamps for recency (no ordered list), over random streams of batches,
  releases and touches on a pool small enough to evict.
"""
import numpy as np
import pytest

from oracle.lifecycle_ref import LruPrefixCacheRef
from oracle.prefix_ref import BLOCK, OracleError, PrefixCacheRef
from paper_2507_08523_amd.workload import cache_op_stream


def _ar(a, b):
    return np.arange(a, b, dtype=np.int32)


def test_without_release_it_is_the_bump_cache():
    rng = np.random.default_rng(11)
    pieces = [rng.integers(0, 32000, int(rng.integers(5, 40))).astype(np.int32) for _ in range(6)]
    lru = LruPrefixCacheRef(num_blocks=4096)
    bump = PrefixCacheRef(num_blocks=4096, max_entries=1 << 16)
    for _ in range(8):
        prompts = [np.concatenate([pieces[i] for i in rng.permutation(6)[:int(rng.integers(1, 5))]])
                   for _ in range(int(rng.integers(1, 6)))]
        reserve = [int(x) for x in rng.integers(0, 20, len(prompts))]
        a = lru.match(prompts, reserve=reserve, max_blocks=24)
        b = bump.match(prompts, reserve=reserve, max_blocks=24)
        for x, y in zip(a, b):
            assert np.array_equal(x, y)
    assert lru.usage()[3] == 0


def test_hand_worked_lifecycle():
    c = LruPrefixCacheRef(num_blocks=6)
    A, B = _ar(0, 33), _ar(100, 133)          # 2 full blocks + 1 token each
    cl, t, _ = c.match([A])
    assert cl[0] == 0 and list(t[0]) == [0, 1, 2]
    c.release(t)                              # block 2 (partial) freed; 1 then 0 cached
    assert c.lru_order() == [1, 0] and list(c.free) == [3, 4, 5, 2]
    assert c.usage() == (0, 2, 4, 0)
    _, tb, _ = c.match([B])                   # free queue first
    assert list(tb[0]) == [3, 4, 5]
    _, tc, _ = c.match([_ar(200, 217)])       # 1 full block + 1 token
    assert list(tc[0]) == [2, 1]              # last free id, then evicts A's tail block 1
    assert c.usage() == (5, 1, 0, 1) and c.lru_order() == [0]
    c.release(tb)                             # B: 5 freed, then 4, 3 cached
    assert c.lru_order() == [0, 4, 3] and list(c.free) == [5]
    cl, ta, _ = c.match([A])                  # A's head block 0 survived: hit, revived
    assert cl[0] == BLOCK and list(ta[0]) == [0, 5, 4]
    assert c.usage() == (5, 1, 0, 2) and c.lru_order() == [3]
    c.release(tc)                             # C: partial block 1 freed, block 2 cached
    assert c.lru_order() == [3, 2] and list(c.free) == [1]
    c.touch([3])
    assert c.lru_order() == [2, 3]
    c.touch([-1, 0, 5])                       # in use: nothing changes
    assert c.lru_order() == [2, 3]
    _, td, _ = c.match([_ar(300, 340)])       # 3 blocks: free 1, evict 2, evict 3
    assert list(td[0]) == [1, 2, 3] and c.usage() == (6, 0, 0, 4)


def test_hits_are_pinned_before_capacity_is_counted():
    c = LruPrefixCacheRef(num_blocks=4)
    A = _ar(0, 33)
    _, t, _ = c.match([A])
    c.release(t)                              # cached [1, 0], free [3, 2]
    before = (c.lru_order(), list(c.free), list(c.ref), dict(c.table))
    with pytest.raises(OracleError) as e:     # A reuses 0, 1: only 2 blocks left for 1 + 3
        c.match([A, _ar(500, 533)])
    assert e.value.code == "ENOSPC"
    assert (c.lru_order(), list(c.free), list(c.ref), dict(c.table)) == before
    cl, t2, _ = c.match([A, _ar(500, 510)])   # 1 + 1 new blocks: the free queue suffices
    assert list(cl) == [32, 0] and list(t2[0]) == [0, 1, 3] and list(t2[1]) == [2, -1, -1]


def test_release_errors_leave_state_unchanged():
    c = LruPrefixCacheRef(num_blocks=8)
    _, t, _ = c.match([_ar(0, 40)])
    before = (list(c.ref), c.lru_order(), list(c.free))
    for bad in ([[0, 0, 0, 0]], [[9]], [[0, 1, 2, 2]]):
        with pytest.raises(OracleError):
            c.release(np.array(bad))
        assert (list(c.ref), c.lru_order(), list(c.free)) == before
    with pytest.raises(OracleError):
        c.touch([0, 8])


class _ExactPrefixModel:
    """Brute force: blocks named by their exact token prefix; recency by stamps."""

    def __init__(self, n):
        self.held, self.content = {}, {}
        self.ref, self.free = [0] * n, list(range(n))
        self.stamp, self.clock, self.evictions = {}, 0, 0

    def match(self, prompts, max_blocks):
        plans = []
        for p in prompts:
            m = 0
            while m < (len(p) - 1) // BLOCK and p[:BLOCK * (m + 1)].tobytes() in self.held:
                m += 1
            plans.append((p, m, -(-len(p) // BLOCK), [self.held[p[:BLOCK * (b + 1)].tobytes()]
                                                      for b in range(m)]))
        need = sum(n - m for (_, m, n, _) in plans)
        revive = {b for (_, _, _, h) in plans for b in h if self.ref[b] == 0}
        if need > len(self.free) + len(self.stamp) - len(revive):
            return None
        for (_, _, _, h) in plans:
            for b in h:
                self.stamp.pop(b, None)
                self.ref[b] += 1
        cached = np.array([BLOCK * m for (_, m, _, _) in plans], np.int32)
        tables = np.full((len(prompts), max_blocks), -1, np.int32)
        for r, (p, m, n, h) in enumerate(plans):
            ids = list(h)
            for _ in range(n - m):
                if self.free:
                    b = self.free.pop(0)
                else:
                    b = min(self.stamp, key=self.stamp.get)
                    del self.stamp[b]
                    del self.held[self.content.pop(b)]
                    self.evictions += 1
                self.ref[b] = 1
                ids.append(b)
            tables[r, :n] = ids
        for r, (p, m, n, _) in enumerate(plans):
            for b in range(m, len(p) // BLOCK):
                pre = p[:BLOCK * (b + 1)].tobytes()
                if pre not in self.held:
                    self.held[pre] = int(tables[r, b])
                    self.content[int(tables[r, b])] = pre
        return cached, tables

    def release(self, rows):
        for row in rows:
            for b in reversed([int(x) for x in row if x >= 0]):
                self.ref[b] -= 1
                if self.ref[b] == 0:
                    if b in self.content:
                        self.clock += 1
                        self.stamp[b] = self.clock
                    else:
                        self.free.append(b)

    def touch(self, ids):
        for b in ids:
            if b in self.stamp:
                self.clock += 1
                self.stamp[b] = self.clock

    def usage(self):
        return (sum(1 for c in self.ref if c > 0), len(self.stamp), len(self.free), self.evictions)

    def lru_order(self):
        return sorted(self.stamp, key=self.stamp.get)


@pytest.mark.parametrize("seed", range(6))
def test_random_streams_against_exact_prefix_model(seed):
    n_blocks, max_blocks = 40, 12
    ref, brute = LruPrefixCacheRef(n_blocks), _ExactPrefixModel(n_blocks)
    rng = np.random.default_rng(100 + seed)
    live = []                      # tables of requests not yet released
    n_hits = n_refused = 0
    for op, arg in cache_op_stream(seed):
        if op == "match":
            got = brute.match(arg, max_blocks)
            if got is None:
                with pytest.raises(OracleError):
                    ref.match(arg, max_blocks=max_blocks)
                n_refused += 1
                continue
            cl, t, _ = ref.match(arg, max_blocks=max_blocks)
            assert np.array_equal(cl, got[0]) and np.array_equal(t, got[1])
            n_hits += int((cl > 0).sum())
            live.extend(t)
        elif op == "release":
            k = int(round(arg * len(live)))
            picks = sorted(rng.permutation(len(live))[:k].tolist())
            rows = np.array([live[i] for i in picks]).reshape(len(picks), max_blocks)
            ref.release(rows)
            brute.release(rows)
            live = [x for i, x in enumerate(live) if i not in set(picks)]
        else:
            ids = [b for b in arg if b < n_blocks]
            ref.touch(ids)
            brute.touch(ids)
        assert ref.usage() == brute.usage()
        assert ref.lru_order() == brute.lru_order()
        assert sum(ref.usage()[:3]) == n_blocks
    assert n_hits > 5 and ref.usage()[3] > 5  # reuse and eviction both happened
