"""The native ICL table of prefix-aware demonstration refinement, on the CPU,
bit-exact against the oracle: final sets, PMC per request and the table's
contents (in LRU order) after every request.
"""
import os

import numpy as np
import pytest

from oracle.pair_ref import PairTableRef
from paper_2507_08523_amd import ilpc

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "pair_worked_example.txt")


@pytest.fixture(scope="module", autouse=True)
def lib():
    if not os.path.exists(ilpc.LIB_PATH):
        pytest.fail("libilpc.so is not built: run `python -m paper_2507_08523_amd.build`")
    return ilpc.load()


def _split(ds):
    return np.array([[t for t, _ in ds]], np.int32), np.array([[d for _, d in ds]], np.int32)


def _pairs(t, d):
    return [(int(a), int(b)) for a, b in zip(t, d)]


def _check_stream(capacity, n, stream, batch=1):
    """Run `stream` (list of sets) through both tables, `batch` requests per call."""
    ref = PairTableRef(capacity, n)
    tab = ilpc.PairTable(capacity, n)
    for s in range(0, len(stream), batch):
        chunk = stream[s:s + batch]
        t = np.array([[x for x, _ in ds] for ds in chunk], np.int32)
        d = np.array([[y for _, y in ds] for ds in chunk], np.int32)
        ot, od, k = tab.refine(t, d)
        for i, ds in enumerate(chunk):
            f_ref, k_ref = ref.process(ds)
            assert int(k[i]) == k_ref, (s + i, ds)
            assert _pairs(ot[i], od[i]) == f_ref, (s + i, ds)
        et, ed = tab.entries()
        assert [_pairs(a, b) for a, b in zip(et, ed)] == ref.entries(), s
    tab.close()


def test_paper_worked_example():
    g = {}
    with open(GOLDEN) as f:
        for line in f:
            if not line.startswith("#") and ":" in line:
                k, v = line.split(":", 1)
                g[k.strip()] = v.strip()
    tid, did = {}, {}

    def ids(text):
        out = []
        for x in text.split(";"):
            t, d = x.strip().split("|", 1)
            out.append((tid.setdefault(t, len(tid)), did.setdefault(d, len(did))))
        return out

    ds1, ds2, cur, final = ids(g["DS_1"]), ids(g["DS_2"]), ids(g["current"]), ids(g["final"])
    tab = ilpc.PairTable(8, 3)
    for ds in (ds1, ds2):
        ot, od, k = tab.refine(*_split(ds))
        assert int(k[0]) == 0 and _pairs(ot[0], od[0]) == ds
    ot, od, k = tab.refine(*_split(cur))
    assert int(k[0]) == int(g["pmc DS_2"]) == 2
    assert _pairs(ot[0], od[0]) == final
    et, ed = tab.entries()
    assert [_pairs(a, b) for a, b in zip(et, ed)] == [ds1, ds2, final]


def test_rules_ties_and_eviction():
    a = [(0, 1), (1, 2), (2, 3)]
    x = [(7, 9), (8, 8), (9, 7)]
    stream = [
        a, x,
        [(2, 30), (0, 10), (1, 20)],   # rule 1 against a
        [(5, 1), (6, 2), (4, 3)],      # rule 2
        [(1, 40), (0, 41), (5, 42)],   # rule 3 against a (PMC 2)
        [(0, 50), (1, 51), (6, 52)],   # tie at PMC 2: the most recent set wins
        [(3, 60), (3, 61), (3, 62)],   # repeated template
        [(3, 63), (3, 64), (0, 65)],   # PMC 2 with one-to-one counting
        [(3, 63), (3, 64), (0, 65)],   # the same set again
        x,                             # evicted by now at capacity 4
    ]
    _check_stream(4, 3, stream)
    _check_stream(1, 3, stream)
    _check_stream(16, 3, stream, batch=4)


def _skewed_stream(rng, n_req, n, n_templates, n_logs, zipf):
    """Template-labelled demonstration sets with a hotspot: templates drawn by a
    Zipf-like law (a few templates dominate, as in production log streams), a
    handful of concrete logs per template, and the order of the set shuffled."""
    w = 1.0 / np.arange(1, n_templates + 1) ** zipf
    w /= w.sum()
    out = []
    for _ in range(n_req):
        ts = rng.choice(n_templates, size=n, replace=True, p=w)
        out.append([(int(t), int(t) * n_logs + int(rng.integers(n_logs))) for t in ts])
    return out


@pytest.mark.parametrize("seed,capacity,n,n_templates,zipf,batch", [
    (0, 8, 3, 6, 1.2, 1),
    (1, 32, 5, 20, 1.1, 7),
    (2, 64, 8, 50, 0.9, 32),
    (3, 3, 4, 5, 1.5, 5),
])
def test_random_streams_match_oracle(seed, capacity, n, n_templates, zipf, batch):
    rng = np.random.default_rng(seed)
    stream = _skewed_stream(rng, 300, n, n_templates, 3, zipf)
    _check_stream(capacity, n, stream, batch=batch)


def test_reset_and_empty_batch():
    tab = ilpc.PairTable(4, 2)
    tab.refine(np.array([[0, 1]]), np.array([[5, 6]]))
    assert tab.entries()[0].shape == (1, 2)
    ot, od, k = tab.refine(np.zeros((0, 2)), np.zeros((0, 2)))
    assert ot.shape == (0, 2) and k.shape == (0,)
    tab.reset()
    assert tab.entries()[0].shape == (0, 2)
    ot, od, k = tab.refine(np.array([[1, 0]]), np.array([[6, 5]]))
    assert int(k[0]) == 0


def test_argument_errors():
    with pytest.raises(ilpc.ILPCError):
        ilpc.PairTable(0, 3)
    with pytest.raises(ilpc.ILPCError):
        ilpc.PairTable(4, 0)
    with pytest.raises(ilpc.ILPCError):
        ilpc.PairTable(4, 5000)
    tab = ilpc.PairTable(4, 3)
    with pytest.raises(ilpc.ILPCError):
        tab.refine(np.zeros((2, 2)), np.zeros((2, 2)))
    lib = ilpc.load()
    assert lib.ilpc_pair_refine(None, None, None, 1, None, None, None) != 0
    assert lib.ilpc_pair_reset(None) != 0


# -- the ICL request stream and what refinement does to its cache hits ---------

from paper_2507_08523_amd import pipeline, workload  # noqa: E402


def test_icl_stream_hotspot_frequencies():
    """The five hottest templates land in about 36.2/27.2/24.7/21.2/17.1% of requests."""
    st = workload.icl_stream("icl_llama8b")
    R, k = st.templates.shape
    assert R == 2000 and k == 5
    assert all(len(set(row)) == k for row in st.templates.tolist())
    assert (st.demos // st.spec.logs_per_template == st.templates).all()
    freq = np.sort(np.bincount(st.templates.ravel(), minlength=st.spec.n_templates) / R)[::-1][:5]
    np.testing.assert_allclose(freq, [0.362, 0.272, 0.247, 0.212, 0.171], atol=0.03)


def _small_icl(history=400, n_prompts=16):
    return workload.scaled_spec("icl_llama8b", n_prompts, history=history)


def test_history_warm_batch_gives_the_stream_cache_state():
    """The measured batch's cached lengths after the derived warm batch equal
    those after serving the whole history through the prefix cache."""
    sp = _small_icl()
    st = workload.icl_stream(sp)
    _, fd, _ = pipeline.pair_refine_stream(st, 64, sp.n_prompts)
    prompts = st.prompts(demos=fd)
    hist, meas = prompts[:sp.history], prompts[sp.history:]
    nb = sum(-(-len(p) // 16) for p in prompts) + 1
    a = ilpc.PrefixCache(nb, 16)
    for s in range(0, len(hist), sp.n_prompts):
        a.match(hist[s:s + sp.n_prompts])
    c_stream, _, _ = a.match(meas)
    wl = workload.build(sp, demos=fd)
    assert all(np.array_equal(x, y) for x, y in zip(wl.prompts, meas))
    b = ilpc.PrefixCache(nb, 16)
    b.match(wl.warm)
    c_warm, _, _ = b.match(wl.prompts)
    assert np.array_equal(c_stream, c_warm)
    assert c_warm.min() >= 256  # the instruction is always held


def test_refinement_raises_the_stream_hit_rate():
    sp = _small_icl(history=800)
    st = workload.icl_stream(sp)
    naive = pipeline.stream_hit_rate(st.prompts(), sp.n_prompts)
    ft, fd, pmc = pipeline.pair_refine_stream(st, pipeline.ICL_TABLE_CAPACITY, sp.n_prompts)
    # refinement only reorders and swaps logs of the same template
    assert (np.sort(ft, axis=1) == np.sort(st.templates, axis=1)).all()
    assert (fd // sp.logs_per_template == ft).all()
    pair = pipeline.stream_hit_rate(st.prompts(demos=fd), sp.n_prompts)
    assert pair["prompt_tokens"] == naive["prompt_tokens"]
    assert pair["hit_rate"] > 1.1 * naive["hit_rate"], (naive, pair)
    assert pmc.max() == sp.n_demos and pmc.min() == 0
