"""GPU parity across shapes the named workloads do not reach: every head-group
size from MHA (G = 1) to the largest accepted (G = 64) at both head dims, a
context of about 12 K keys (190 key tiles), and a block table 70 000 entries
wide.  Every output row is checked against the fp64 oracle (max |err| <= 2e-2,
mean |err| <= 2e-3), on ragged cached and query lengths.
"""
import sys

import numpy as np
import pytest
import torch

from oracle.attn_ref import prefill_attention_ref
from oracle.prefix_ref import PrefixCacheRef
from paper_2507_08523_amd import ilpc, workload
from paper_2507_08523_amd.pipeline import PagedPrefixCache, max_blocks_of, pool_blocks_needed

pytestmark = pytest.mark.gpu

MAX_ABS, MEAN_ABS = 2e-2, 2e-3


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a ROCm GPU (run with -m 'not gpu' on the CPU)")
    ilpc.load()
    yield
    torch.cuda.synchronize()


def log(*a):
    import conftest

    print(*a, flush=True)
    sys.stdout.flush()
    conftest.PARITY_LINES.append(" ".join(str(x) for x in a))


def _run_and_check(spec, max_blocks=None, tag=""):
    wl = workload.build(spec)
    wl.materialize("cuda")
    sp = wl.spec
    nb = pool_blocks_needed(wl)
    mb = max_blocks or max_blocks_of(wl)
    pc = PagedPrefixCache(sp.n_kv_heads, sp.head_dim, nb, mb, max(len(wl.prompts), len(wl.warm), 1), 16)
    ref = PrefixCacheRef(nb, (1 << 16) - (1 << 13))
    if wl.warm:
        c, t = pc.match(wl.warm)
        ref.match(wl.warm, max_blocks=mb)
        rows = wl.packed_warm(c)
        pc.append(pc.upload_prefill(c, t, [len(p) for p in wl.warm]), rows["k_new"], rows["v_new"])
    c, t = pc.match(wl.prompts)
    c_ref, t_ref, _ = ref.match(wl.prompts, max_blocks=mb)
    assert np.array_equal(c, c_ref) and np.array_equal(t, t_ref)
    rows = wl.packed_suffix(c)
    b = pc.upload_prefill(c, t, wl.seq_lens)
    pc.append(b, rows["k_new"], rows["v_new"])
    out = torch.full_like(rows["q"], float("nan"))
    pc.attend(b, rows["q"], out, sp.scale)
    torch.cuda.synchronize()
    worst, tot, cnt = 0.0, 0.0, 0
    for r in range(len(wl.prompts)):
        L, P = int(wl.seq_lens[r]), int(c[r])
        k, v = wl.dense_kv(r, L)
        expect = prefill_attention_ref(wl.q_rows(r, P, L).float().cpu().numpy(), k.float().cpu().numpy(),
                                       v.float().cpu().numpy(), sp.scale)
        got = out[int(rows["cu"][r]):int(rows["cu"][r + 1])].float().cpu().numpy()
        assert np.isfinite(got).all(), r
        err = np.abs(got - expect)
        worst = max(worst, float(err.max()))
        tot += float(err.sum())
        cnt += err.size
    log(f"[parity] {sp.name}{tag}: Hq {sp.n_q_heads} / Hkv {sp.n_kv_heads} / D {sp.head_dim}, "
        f"{len(wl.prompts)} requests, cached {c.tolist()}, max_blocks {mb}: max_abs={worst:.3e} "
        f"mean_abs={tot / cnt:.3e}")
    assert worst <= MAX_ABS and tot / cnt <= MEAN_ABS
    return c


@pytest.mark.parametrize("G,Hkv", [(1, 8), (2, 4), (3, 2), (5, 3), (16, 2), (64, 1)])
@pytest.mark.parametrize("D", [64, 128])
def test_head_groups(G, Hkv, D):
    spec = workload.WorkloadSpec(name=f"groups_G{G}", n_q_heads=G * Hkv, n_kv_heads=Hkv, head_dim=D,
                                 n_prompts=6, instr_len=80, n_demos=3, demo_len=40, pool_size=5,
                                 query_len=(1, 70), seed=600 + 10 * G + D)
    c = _run_and_check(spec)
    assert c.max() > 0   # the batch shares cached prefixes


def test_long_context_twelve_thousand_keys():
    # each prompt's own 11 968-token prefix is cached; 1..100 new tokens follow
    spec = workload.WorkloadSpec(name="long12k", n_q_heads=8, n_kv_heads=1, head_dim=128, n_prompts=3,
                                 instr_len=0, n_demos=187, demo_len=64, pool_size=200, query_len=(1, 100),
                                 warm="own_prefix", own_prefix_len=11968, seed=700)
    c = _run_and_check(spec)
    assert (c == 11968).all()


def test_block_table_seventy_thousand_wide():
    # rows of 70 000 block ids (-1 past each prompt's blocks): the kernel reads
    # ids by clamped index and position, whatever the row width
    spec = workload.scaled_spec("llama8b", 4)
    _run_and_check(spec, max_blocks=70000, tag=" (wide table)")
