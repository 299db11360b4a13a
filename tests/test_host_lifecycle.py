"""The native block lifecycle (ilpc_cache_create_lru and friends) on the CPU,
bit-exact against the oracle: cached lengths, block tables, block keys, the
usage counters and the LRU order after every operation.
"""
import os

import numpy as np
import pytest

from oracle.lifecycle_ref import LruPrefixCacheRef
from oracle.prefix_ref import OracleError
from paper_2507_08523_amd import ilpc
from paper_2507_08523_amd.workload import cache_op_stream


@pytest.fixture(scope="module", autouse=True)
def lib():
    if not os.path.exists(ilpc.LIB_PATH):
        pytest.fail("libilpc.so is not built: run `python -m paper_2507_08523_amd.build`")
    return ilpc.load()


class Both:
    """Drives the native cache and the oracle with the same operations."""

    def __init__(self, n_blocks, log2cap=None):
        log2cap = log2cap or max(4, int(np.ceil(np.log2(n_blocks * 8 / 7 + 1))))
        self.n = n_blocks
        self.nat = ilpc.PrefixCache(n_blocks, log2cap, lru=True)
        self.ref = LruPrefixCacheRef(n_blocks)

    def check_state(self):
        assert self.nat.usage() == self.ref.usage()
        assert self.nat.lru_order() == self.ref.lru_order()
        u = self.nat.usage()
        assert u[0] + u[1] + u[2] == self.n

    def match(self, prompts, max_blocks, flags=0, **kw):
        kw_ref = dict(kw, no_lookup=bool(flags & 1), no_register=bool(flags & 2))
        kw["flags"] = flags
        try:
            want = self.ref.match(prompts, max_blocks=max_blocks, **kw_ref)
        except OracleError as e:
            with pytest.raises(ilpc.ILPCError) as got:
                self.nat.match(prompts, max_blocks=max_blocks, want_keys=True, **kw)
            assert got.value.code == getattr(ilpc, e.code)
            self.check_state()
            return None
        got = self.nat.match(prompts, max_blocks=max_blocks, want_keys=True, **kw)
        for a, b in zip(got, want):
            assert np.array_equal(a, b)
        self.check_state()
        return got

    def release(self, tables):
        self.nat.release(tables)
        self.ref.release(tables)
        self.check_state()

    def touch(self, ids):
        self.nat.touch(ids)
        self.ref.touch(ids)
        self.check_state()


def _ar(a, b):
    return np.arange(a, b, dtype=np.int32)


def test_hand_worked_lifecycle_bit_exact():
    c = Both(6)
    A, B = _ar(0, 33), _ar(100, 133)
    _, t, _ = c.match([A], 3)
    c.release(t)
    _, tb, _ = c.match([B], 3)
    _, tc, _ = c.match([_ar(200, 217)], 3)
    c.release(tb)
    cl, ta, _ = c.match([A], 3)
    assert cl[0] == 16 and list(ta[0]) == [0, 5, 4]
    c.release(tc)
    c.touch([3])
    c.touch([-1, 0, 5])
    _, td, _ = c.match([_ar(300, 340)], 3)
    assert list(td[0]) == [1, 2, 3] and c.nat.usage() == (6, 0, 0, 4)


@pytest.mark.parametrize("seed", range(8))
@pytest.mark.parametrize("n_blocks", [24, 40, 64])
def test_random_streams_bit_exact(seed, n_blocks):
    c = Both(n_blocks)
    rng = np.random.default_rng(200 + seed)
    live, max_blocks = [], 12
    for op, arg in cache_op_stream(seed, n_steps=80):
        if op == "match":
            reserve = [int(x) for x in rng.integers(0, 12, len(arg))]
            got = c.match(arg, max_blocks, reserve=reserve)
            if got is not None:
                live.extend(got[1])
        elif op == "release":
            k = int(round(arg * len(live)))
            picks = set(rng.permutation(len(live))[:k].tolist())
            rows = np.array([live[i] for i in sorted(picks)], np.int32).reshape(len(picks), max_blocks)
            c.release(rows)
            live = [x for i, x in enumerate(live) if i not in picks]
        else:
            c.touch([b for b in arg if b < n_blocks])
    c.release(np.array(live, np.int32).reshape(len(live), max_blocks))
    assert c.nat.usage()[0] == 0


def test_many_evictions_keep_the_key_table_consistent():
    """A long stream on a small pool with a tight key table: evictions delete
    keys from the middle of probe runs, and every later lookup must agree."""
    c = Both(48, log2cap=6)          # 64 slots, 56 keys max >= 48 blocks
    rng = np.random.default_rng(7)
    pieces = [rng.integers(0, 32000, 16 * int(rng.integers(1, 4))).astype(np.int32) for _ in range(12)]
    for step in range(300):
        prompts = [np.concatenate([pieces[i] for i in rng.permutation(12)[:int(rng.integers(1, 4))]]
                                  + [rng.integers(0, 32000, 3).astype(np.int32)])
                   for _ in range(int(rng.integers(1, 3)))]
        got = c.match(prompts, 12)
        if got is not None:
            c.release(got[1])
    assert c.nat.usage()[3] > 100


def test_flags_and_without_release_equals_bump_cache():
    rng = np.random.default_rng(5)
    prompts = [rng.integers(0, 50, int(rng.integers(20, 90))).astype(np.int32) for _ in range(6)]
    prompts += [p.copy() for p in prompts[:3]]
    bump = ilpc.PrefixCache(4096, 14)
    c = Both(4096, 14)
    for i in range(0, len(prompts), 3):
        a = bump.match(prompts[i:i + 3], max_blocks=8)
        b = c.match(prompts[i:i + 3], 8)
        assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])
    c.match(prompts[:2], 8, flags=1)
    c.match(prompts[:2], 8, flags=2)


def test_errors_and_unsupported_calls():
    with pytest.raises(ilpc.ILPCError) as e:
        ilpc.PrefixCache(1000, 10, lru=True)     # 896 keys < 1000 blocks
    assert e.value.code == ilpc.EINVAL
    c = Both(8)
    _, t, _ = c.match([_ar(0, 40)], 4)
    for bad in ([[0, 0, 0, 0]], [[9, -1, -1, -1]], [[0, 1, 2, 2]], [[-7, -1, -1, -1]]):
        with pytest.raises(ilpc.ILPCError):
            c.nat.release(np.array(bad))
        c.check_state()
    with pytest.raises(ilpc.ILPCError):
        c.nat.touch([0, 8])
    c.check_state()
    with pytest.raises(ilpc.ILPCError) as e:
        c.nat.checkpoint()
    assert e.value.code == ilpc.EUNSUP
    bump = ilpc.PrefixCache(8, 4)
    for call in (lambda: bump.release(np.zeros((1, 2))), lambda: bump.touch([0])):
        with pytest.raises(ilpc.ILPCError) as e:
            call()
        assert e.value.code == ilpc.EUNSUP
    assert bump.lru_order() == []
    c.nat.reset()
    c.ref = LruPrefixCacheRef(8)
    c.check_state()
    c.match([_ar(0, 40)], 4)
