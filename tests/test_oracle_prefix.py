"""Pins of the prefix-cache oracle against facts outside itself.

* fmix64 against SMHasher's published verification value of MurmurHash3_x64_128
  (the finaliser is that hash's last step; the body is written out here);
* the paper's three-request example (section 2.1.2, figure on prefix caching):
  req2 reuses b1, b2; req3 reuses b1..b3 but not req2's b7, b8;
* brute force: the cached length equals the block-aligned longest common
  prefix with any previously committed prompt, capped so one token is
  recomputed; cached block ids equal those first allocated for that prefix;
* the stored key vectors written by tests/golden/make_golden.py.
"""
import os

import numpy as np
import pytest

from oracle.prefix_ref import (BLOCK, OracleError, PrefixCacheRef, block_digest, block_digests,
                               chain_keys, fmix64)
from paper_2507_08523_amd import workload

M64 = (1 << 64) - 1


def _rotl(x, r):
    return ((x << r) | (x >> (64 - r))) & M64


def _murmur3_x64_128(data: bytes, seed: int) -> bytes:
    """MurmurHash3_x64_128 (Appleby) written out, finalised by the oracle's fmix64."""
    c1, c2 = 0x87C37B91114253D5, 0x4CF5AD432745937F
    h1 = h2 = seed & M64
    n = len(data)
    nb = n // 16
    for i in range(nb):
        k1 = int.from_bytes(data[16 * i:16 * i + 8], "little")
        k2 = int.from_bytes(data[16 * i + 8:16 * i + 16], "little")
        k1 = _rotl((k1 * c1) & M64, 31) * c2 & M64
        h1 ^= k1
        h1 = (_rotl(h1, 27) + h2) & M64
        h1 = (h1 * 5 + 0x52DCE729) & M64
        k2 = _rotl((k2 * c2) & M64, 33) * c1 & M64
        h2 ^= k2
        h2 = (_rotl(h2, 31) + h1) & M64
        h2 = (h2 * 5 + 0x38495AB5) & M64
    tail = data[16 * nb:]
    if len(tail) > 8:
        k2 = int.from_bytes(tail[8:], "little")
        h2 ^= _rotl((k2 * c2) & M64, 33) * c1 & M64
    if len(tail) > 0:
        k1 = int.from_bytes(tail[:8], "little")
        h1 ^= _rotl((k1 * c1) & M64, 31) * c2 & M64
    h1 ^= n
    h2 ^= n
    h1 = (h1 + h2) & M64
    h2 = (h2 + h1) & M64
    h1, h2 = fmix64(h1), fmix64(h2)
    h1 = (h1 + h2) & M64
    h2 = (h2 + h1) & M64
    return h1.to_bytes(8, "little") + h2.to_bytes(8, "little")


def test_fmix64_matches_smhasher_verification_value():
    # SMHasher VerificationTest: hash {0}, {0,1}, ... with seed 256-len, hash the
    # concatenation with seed 0; the first 4 bytes little-endian are published.
    key = bytearray(256)
    acc = b""
    for i in range(256):
        key[i] = i
        acc += _murmur3_x64_128(bytes(key[:i]), 256 - i)
    final = _murmur3_x64_128(acc, 0)
    assert int.from_bytes(final[:4], "little") == 0x6384BA69


def test_fmix64_is_bijective_on_sample():
    rng = np.random.default_rng(1)
    xs = {int(x) for x in rng.integers(0, 2**63, 20000, dtype=np.int64)}
    assert len({fmix64(x) for x in xs}) == len(xs)
    assert fmix64(0) == 0


def test_vectorised_digest_equals_scalar_digest():
    rng = np.random.default_rng(2)
    toks = rng.integers(-2**31, 2**31, 16 * 37, dtype=np.int64).astype(np.int32)
    vec = block_digests(toks).tolist()
    for b in range(37):
        assert vec[b] == block_digest(toks[16 * b:16 * (b + 1)])


def test_digest_depends_on_token_order_and_value():
    base = np.arange(16, dtype=np.int32)
    d0 = block_digest(base)
    swapped = base.copy()
    swapped[[0, 1]] = swapped[[1, 0]]
    assert block_digest(swapped) != d0
    bumped = base.copy()
    bumped[15] += 1
    assert block_digest(bumped) != d0


def test_chain_key_depends_on_predecessors():
    a = np.arange(32, dtype=np.int32)
    b = a.copy()
    b[0] = 999  # same second block, different first block
    assert chain_keys(a)[1] != chain_keys(b)[1]
    assert chain_keys(a)[0] == chain_keys(a[:16])[0]
    assert len(chain_keys(a[:31])) == 1


def test_golden_key_vectors():
    path = os.path.join(os.path.dirname(__file__), "golden", "chain_keys.txt")
    n_lines = 0
    with open(path) as f:
        for line in f:
            if line.startswith("#"):
                continue
            head, dig, keys = line.rstrip("\n").split(" | ")
            parts = head.split()
            n = int(parts[1])
            toks = np.array([int(t) for t in parts[2:2 + n]], dtype=np.int32)
            assert [f"{int(x):016x}" for x in block_digests(toks).tolist()] == dig.split()
            assert [f"{x:016x}" for x in chain_keys(toks)] == keys.split()
            n_lines += 1
    assert n_lines >= 8


def test_paper_three_request_example():
    # req1 = b1 b2 b3 b4 b5, req2 = b1 b2 b6 b7 b8, req3 = b1 b2 b3 b7 b8
    rng = np.random.default_rng(3)
    blk = {i: rng.integers(0, 32000, BLOCK).astype(np.int32) for i in range(1, 9)}
    q = [rng.integers(0, 32000, 1).astype(np.int32) for _ in range(3)]
    req1 = np.concatenate([blk[1], blk[2], blk[3], blk[4], blk[5], q[0]])
    req2 = np.concatenate([blk[1], blk[2], blk[6], blk[7], blk[8], q[1]])
    req3 = np.concatenate([blk[1], blk[2], blk[3], blk[7], blk[8], q[2]])
    cache = PrefixCacheRef(num_blocks=64, max_entries=1024)
    c1, t1, _ = cache.match([req1], max_blocks=6)
    c2, t2, _ = cache.match([req2], max_blocks=6)
    c3, t3, _ = cache.match([req3], max_blocks=6)
    assert (c1[0], c2[0], c3[0]) == (0, 2 * BLOCK, 3 * BLOCK)
    assert list(t2[0, :2]) == list(t1[0, :2])
    assert list(t3[0, :3]) == list(t1[0, :3])
    # req3 cannot reuse req2's b7, b8 (different predecessor): fresh ids
    assert not set(t3[0, 3:5]) & set(t2[0, 3:5])
    assert t3[0, 3] == t2[0, 5] + 1  # bump allocator continues after req2


def _lcp(a, b):
    n = min(len(a), len(b))
    eq = np.asarray(a[:n]) == np.asarray(b[:n])
    return n if eq.all() else int(np.argmin(eq))


def test_brute_force_lcp_and_block_ids_over_batches():
    rng = np.random.default_rng(4)
    pieces = [rng.integers(0, 32000, int(rng.integers(5, 40))).astype(np.int32) for _ in range(6)]
    cache = PrefixCacheRef(num_blocks=100000, max_entries=1 << 16)
    committed = []          # prompts of earlier batches, in commit order
    first_id = {}           # exact full-block prefix -> id of its first allocation
    next_id = 0
    n_hits = 0
    for batch in range(6):
        prompts = []
        for _ in range(int(rng.integers(1, 7))):
            k = int(rng.integers(1, 5))
            order = rng.permutation(len(pieces))[:k]
            p = np.concatenate([pieces[i] for i in order] + [rng.integers(0, 32000, int(rng.integers(0, 20))).astype(np.int32)])
            if len(p) == 0:
                p = np.array([5], np.int32)
            prompts.append(p)
        if batch == 3:
            prompts.append(prompts[0].copy())  # duplicate inside one batch
        reserve = [int(x) for x in rng.integers(0, 20, len(prompts))]
        cached, tables, keys = cache.match(prompts, reserve=reserve, max_blocks=64)
        for r, p in enumerate(prompts):
            L = len(p)
            best = 0
            for s in committed:
                best = max(best, min(_lcp(p, s), BLOCK * (len(s) // BLOCK)) // BLOCK)
            m = min(best, (L - 1) // BLOCK)
            assert cached[r] == BLOCK * m, (batch, r)
            n_hits += m > 0
            for b in range(m):
                assert tables[r, b] == first_id[p[:BLOCK * (b + 1)].tobytes()]
            n_total = -(-(L + reserve[r]) // BLOCK)
            assert list(tables[r, m:n_total]) == list(range(next_id, next_id + n_total - m))
            assert (tables[r, n_total:] == -1).all()
            next_id += n_total - m
        for r, p in enumerate(prompts):  # register after the batch, first writer wins
            for b in range(len(p) // BLOCK):
                first_id.setdefault(p[:BLOCK * (b + 1)].tobytes(), int(tables[r, b]))
        committed.extend(prompts)
    assert n_hits >= 5  # the case exercises reuse, not only misses


def test_frozen_snapshot_inside_a_batch():
    p = np.arange(40, dtype=np.int32)
    cache = PrefixCacheRef(num_blocks=100, max_entries=100)
    c, t, _ = cache.match([p, p.copy()], max_blocks=3)
    assert list(c) == [0, 0]
    assert t[0, 0] != t[1, 0]
    c2, t2, _ = cache.match([p.copy()], max_blocks=3)
    assert c2[0] == 32 and list(t2[0, :2]) == list(t[0, :2])  # lower index registered


def test_fully_cached_prompt_recomputes_last_block():
    p = np.arange(48, dtype=np.int32)  # L % 16 == 0
    cache = PrefixCacheRef(num_blocks=100, max_entries=100)
    _, t0, _ = cache.match([p], max_blocks=3)
    c, t, _ = cache.match([p.copy()], max_blocks=3)
    assert c[0] == 32  # capped at (L-1)//16 = 2 blocks, S = 16
    assert t[0, 2] != t0[0, 2]
    assert cache.table[chain_keys(p)[2]] == t0[0, 2]  # not re-registered


def test_flags_no_lookup_and_no_register():
    p = np.arange(40, dtype=np.int32)
    cache = PrefixCacheRef(num_blocks=100, max_entries=100)
    cache.match([p], max_blocks=3, no_register=True)
    assert cache.table == {}
    cache.match([p], max_blocks=3)
    c, _, _ = cache.match([p], max_blocks=3, no_lookup=True)
    assert c[0] == 0


@pytest.mark.parametrize("what,code", [("pool", "ENOSPC"), ("table", "ETABLE"),
                                       ("empty", "EINVAL"), ("max_blocks", "EINVAL"),
                                       ("reserve", "EINVAL")])
def test_errors_leave_state_unchanged(what, code):
    cache = PrefixCacheRef(num_blocks=8, max_entries=4)
    cache.match([np.arange(20, dtype=np.int32)], max_blocks=4)  # 2 blocks, 1 entry
    before = (dict(cache.table), cache.next_block)
    p = np.arange(100, 180, dtype=np.int32)                    # 5 full blocks
    with pytest.raises(OracleError) as e:
        if what == "pool":
            cache.match([p[:40], p[:70] + 1], max_blocks=8)     # 3 + 5 blocks > 6 left
        elif what == "table":
            cache.match([p[:70]], max_blocks=8)                 # 1 held + 4 new > 4
        elif what == "empty":
            cache.match([p[:20], np.zeros(0, np.int32)], max_blocks=8)
        elif what == "max_blocks":
            cache.match([p], max_blocks=4)
        else:
            cache.match([p[:20]], reserve=[-1], max_blocks=8)
    assert e.value.code == code
    assert (dict(cache.table), cache.next_block) == before


@pytest.mark.parametrize("name,expect", [("sweep0", 0), ("sweep25", 256), ("sweep50", 496),
                                         ("sweep75", 736), ("sweep100", 976)])
def test_sweep_workloads_reach_their_cached_fraction(name, expect):
    wl = workload.build(name)
    cache = PrefixCacheRef(num_blocks=1 << 20, max_entries=1 << 20)
    if wl.warm:
        cache.match(wl.warm)
    cached, _, _ = cache.match(wl.prompts)
    assert (cached == expect).all()


@pytest.mark.parametrize("name", ["tiny", "llama8b"])
def test_warm_protocol_gives_longest_shared_block_prefix(name):
    wl = workload.build(name)
    cache = PrefixCacheRef(num_blocks=1 << 20, max_entries=1 << 20)
    cache.match(wl.warm)
    cached, _, _ = cache.match(wl.prompts)
    for r, p in enumerate(wl.prompts):
        best = max(_lcp(p, s) for j, s in enumerate(wl.prompts) if j != r)
        assert cached[r] == BLOCK * min(best // BLOCK, (len(p) - 1) // BLOCK)
    if name == "tiny":
        assert (cached == 64).all()
