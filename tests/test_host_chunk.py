"""Host scheduling policy in the library (CPU only): the token-budget steps of
a chunked prefill (ilpc_chunk_schedule) and the cascade split point
(ilpc_shared_prefix_len), against brute-force models written here."""
import numpy as np
import pytest

from paper_2507_08523_amd import ilpc
from paper_2507_08523_amd.pipeline import chunk_schedule, shared_prefix_len


def _fcfs_by_token(q_lens, budget):
    """Brute force: hand out the packed new-token rows one at a time, a step
    closing after every `budget` tokens; group consecutive tokens of one
    request within one step into a piece."""
    steps = []
    t = 0
    for r, n in enumerate(q_lens):
        for i in range(n):
            s = t // budget
            while len(steps) <= s:
                steps.append([])
            if steps[s] and steps[s][-1][0] == r:
                rr, o, m = steps[s][-1]
                steps[s][-1] = (rr, o, m + 1)
            else:
                steps[s].append((r, i, 1))
            t += 1
    return steps


@pytest.mark.parametrize("seed", range(5))
@pytest.mark.parametrize("budget", [1, 7, 64, 512, 100000])
def test_schedule_covers_every_token_once_in_order(seed, budget):
    rng = np.random.default_rng(seed)
    q_lens = rng.integers(0, 300, int(rng.integers(1, 20)))
    steps = chunk_schedule(q_lens, budget)
    assert steps == _fcfs_by_token(q_lens.tolist(), budget)
    flat = [(r, o + i) for step in steps for (r, o, n) in step for i in range(n)]
    assert flat == [(r, i) for r, n in enumerate(q_lens.tolist()) for i in range(n)]
    sizes = [sum(n for (_, _, n) in step) for step in steps]
    assert all(s == budget for s in sizes[:-1]) and 0 < sizes[-1] <= budget if steps else True
    assert len(steps) == -(-int(q_lens.sum()) // budget)
    for step in steps:                     # a request appears at most once per step
        rs = [r for (r, _, _) in step]
        assert rs == sorted(set(rs)) and all(n > 0 for (_, _, n) in step)


def test_schedule_edge_cases():
    assert chunk_schedule([], 8) == []
    assert chunk_schedule([0, 0], 8) == []
    assert chunk_schedule([3, 0, 5], 4) == [[(0, 0, 3), (2, 0, 1)], [(2, 1, 4)]]
    assert chunk_schedule([4, 4], 4) == [[(0, 0, 4)], [(1, 0, 4)]]
    with pytest.raises(ilpc.ILPCError):
        chunk_schedule([3], 0)
    with pytest.raises(ilpc.ILPCError):
        chunk_schedule([3, -1], 4)


def test_schedule_sizes_itself_and_refuses_short_arrays():
    import ctypes

    lib = ilpc.load()
    q = np.array([10, 0, 25, 3], np.int32)
    n_p, n_s = ctypes.c_int32(), ctypes.c_int32()
    arr = [np.zeros(2, np.int32) for _ in range(4)]
    rc = lib.ilpc_chunk_schedule(q.ctypes.data, 4, 8, 2, *(a.ctypes.data for a in arr),
                                 ctypes.byref(n_p), ctypes.byref(n_s))
    assert rc == ilpc.EINVAL and n_p.value == 7 and n_s.value == 5
    assert all((a == 0).all() for a in arr)   # nothing written


def _shared_brute(cached, tables):
    n = min(cached) // 16
    run = 0
    while run < n and tables[0][run] >= 0 and all(t[run] == tables[0][run] for t in tables):
        run += 1
    return 16 * run


@pytest.mark.parametrize("seed", range(20))
def test_shared_prefix_len_against_brute_force(seed):
    rng = np.random.default_rng(seed)
    B, mb = int(rng.integers(1, 9)), int(rng.integers(1, 12))
    common = rng.integers(0, 50, mb)
    cut = rng.integers(0, mb + 1, B)          # rows share the first cut[r] ids
    tables = np.array([[common[i] if i < cut[r] else 100 + r * mb + i for i in range(mb)] for r in range(B)],
                      np.int32)
    if rng.random() < 0.3:                    # rows end early: -1 padding from some block on
        tables[:, int(rng.integers(0, mb + 1)):] = -1
    cached = (16 * rng.integers(0, mb + 1, B)).astype(np.int32)
    assert shared_prefix_len(cached, tables) == _shared_brute(cached.tolist(), tables.tolist())


def test_shared_prefix_len_cases():
    t = np.array([[5, 6, 7, 8], [5, 6, 9, 10], [5, 6, 7, -1]], np.int32)
    assert shared_prefix_len([64, 64, 64], t) == 32     # ids diverge at block 2
    assert shared_prefix_len([64, 16, 64], t) == 16     # capped by the shortest cached prefix
    assert shared_prefix_len([64], t[:1]) == 64
    assert shared_prefix_len([], np.zeros((0, 4), np.int32)) == 0
    neg = np.array([[-1, 3], [-1, 3]], np.int32)
    assert shared_prefix_len([32, 32], neg) == 0
    with pytest.raises(ilpc.ILPCError):
        shared_prefix_len([-16, 32], neg)


def test_prefer_shared_split_rule():
    # the split is chosen for prefill-shaped batches whose shared keys span at
    # least three 64-key tiles and whose requests have at most 128 keys of
    # their own past them
    from paper_2507_08523_amd.ilpc import prefer_shared_split

    def pick(L, shared, q=48, Hq=32, Hkv=8):
        return prefer_shared_split(L, q, Hq, Hkv, shared)

    assert pick([1024] * 128, 976)                        # sweep100: 48 own keys
    assert not pick([1024 + 32] * 128, 976, q=1)          # its decode steps: decode-shaped
    assert not pick([1024] * 128, 976, q=8)               # 8 rows x G 4 = 32 columns: decode-shaped
    assert pick([1024] * 128, 976, q=9)                   # 36 columns: prefill-shaped
    assert not pick([1024] * 128, 736)                    # sweep75: 288 own keys
    assert not pick([604] * 64, 256)                      # llama8b
    assert pick([192 + 128, 192], 192)                    # both limits met exactly
    assert not pick([192 + 129, 192], 192)                # one request past 128
    assert not pick([176 + 64] * 4, 176)                  # under three tiles shared
    assert not pick([], 0)
    for bad in (([100], 200, 48, 32, 8), ([100], -1, 48, 32, 8), ([100], 0, 48, 6, 4)):
        with pytest.raises(ilpc.ILPCError):
            pick(bad[0], bad[1], q=bad[2], Hq=bad[3], Hkv=bad[4])
