"""Host side of chunked prefill: the token-budget scheduler."""
import numpy as np
import pytest

from paper_2507_08523_amd import ilpc
from paper_2507_08523_amd.pipeline import chunk_schedule


@pytest.mark.parametrize("seed", range(5))
@pytest.mark.parametrize("budget", [1, 7, 64, 512, 100000])
def test_schedule_covers_every_token_once_in_order(seed, budget):
    rng = np.random.default_rng(seed)
    q_lens = rng.integers(0, 300, int(rng.integers(1, 20)))
    steps = chunk_schedule(q_lens, budget)
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
    with pytest.raises(ilpc.ILPCError):
        chunk_schedule([3], 0)
