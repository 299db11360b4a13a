"""GPU: the fused RoPE + K/V append, and chunked prefill under a token budget,
against the oracles (rotation in float64, attention in float64).

Rotated rows are bf16: each element within one bf16 unit of the float64
rotation, plus the angle's fp32 rounding (positions < 4096).  Attention
outputs use the usual tolerance (max-abs 2e-2, mean-abs 2e-3).
"""
import sys

import numpy as np
import pytest
import torch

from oracle.attn_ref import prefill_attention_ref
from oracle.rope_ref import rope
from paper_2507_08523_amd import ilpc, workload
from paper_2507_08523_amd.pipeline import (PagedPrefixCache, chunk_schedule, max_blocks_of,
                                           pool_blocks_needed, rope_inv_freq)

pytestmark = pytest.mark.gpu

MAX_ABS, MEAN_ABS = 2e-2, 2e-3
BLOCK = 16


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


def _setup(name, n_prompts, base=None):
    wl = workload.build(workload.scaled_spec(name, n_prompts))
    wl.materialize("cuda")
    sp = wl.spec
    pc = PagedPrefixCache(sp.n_kv_heads, sp.head_dim, pool_blocks_needed(wl), max_blocks_of(wl),
                          max(len(wl.prompts), len(wl.warm), 1), 16)
    inv_freq = None
    if base is not None:
        inv_freq = torch.from_numpy(rope_inv_freq(sp.head_dim, base)).cuda()
    if wl.warm:
        c, t = pc.match(wl.warm)
        rows = wl.packed_warm(c)
        b = pc.upload_prefill(c, t, [len(p) for p in wl.warm])
        if inv_freq is None:
            pc.append(b, rows["k_new"], rows["v_new"])
        else:
            pc.append_rope(b, rows["k_new"], rows["v_new"], inv_freq)
    c, t = pc.match(wl.prompts)
    return wl, pc, c, t, inv_freq


def _rope_bound(ref, x_rows):
    # one bf16 unit of the result + fp32 angle rounding at positions < 4096
    return 2.0 ** -7 * np.abs(ref) + 3e-4 * np.abs(x_rows).max(axis=-1, keepdims=True) + 1e-6


@pytest.mark.parametrize("name,base", [("llama8b", 500000.0), ("qwen7b", 1000000.0), ("tiny", 10000.0)])
def test_rope_append_against_oracle(name, base):
    wl, pc, c, t, inv_freq = _setup(name, 6, base)
    sp = wl.spec
    rows = wl.packed_suffix(c)
    q, k_new, v_new = rows["q"], rows["k_new"], rows["v_new"]
    q_out = torch.empty_like(q)
    b = pc.upload_prefill(c, t, wl.seq_lens)
    pc.append_rope(b, k_new, v_new, inv_freq, q, q_out)
    q_in = q.clone()
    pc.append_rope(b, k_new, v_new, inv_freq, q_in, q_in)      # in place: same bits
    torch.cuda.synchronize()
    assert torch.equal(q_in, q_out)
    f = inv_freq.cpu().numpy()
    cu = rows["cu"]
    worst = 0.0
    kp, vp = pc.k_pool.cpu(), pc.v_pool.cpu()
    for r in range(len(wl.prompts)):
        P, L = int(c[r]), int(wl.seq_lens[r])
        pos = np.arange(P, L)
        sl = slice(int(cu[r]), int(cu[r + 1]))
        x = q[sl].float().cpu().numpy()
        ref = rope(x, pos, f)
        err = np.abs(q_out[sl].float().cpu().numpy() - ref)
        assert (err <= _rope_bound(ref, x)).all(), f"request {r}: Q rotation off by {err.max():.3e}"
        worst = max(worst, float(err.max()))
        xk = k_new[sl].float().cpu().numpy()
        refk = rope(xk, pos, f)
        phys = t[r, pos // BLOCK]
        gotk = kp[phys, :, pos % BLOCK, :].float().numpy()           # [n, Hkv, D]
        errk = np.abs(gotk - refk)
        assert (errk <= _rope_bound(refk, xk)).all(), f"request {r}: K rotation off by {errk.max():.3e}"
        gotv = vp[phys, :, :, pos % BLOCK]                             # [n, Hkv, D]
        assert torch.equal(gotv, v_new[sl].cpu()), f"request {r}: V changed"
    log(f"[rope] {sp.name}: Q/K max_abs={worst:.3e}")


def test_rope_append_without_queries_and_bad_arguments():
    wl, pc, c, t, inv_freq = _setup("tiny", 4, 10000.0)
    rows = wl.packed_suffix(c)
    b = pc.upload_prefill(c, t, wl.seq_lens)
    pc.append_rope(b, rows["k_new"], rows["v_new"], inv_freq)          # K/V only
    torch.cuda.synchronize()
    with pytest.raises(ilpc.ILPCError):
        pc.append_rope(b, rows["k_new"], rows["v_new"], inv_freq, rows["q"], None)
    with pytest.raises(ilpc.ILPCError):
        pc.append_rope(b, rows["k_new"], rows["v_new"], inv_freq[:3], rows["q"], rows["q"])


def _oracle_rows(wl, r, P, L, f=None):
    k, v = wl.dense_kv(r, L)
    q = wl.q_rows(r, P, L)
    q, k, v = q.float().cpu().numpy(), k.float().cpu().numpy(), v.float().cpu().numpy()
    if f is not None:
        q = rope(q, np.arange(P, L), f)
        k = rope(k, np.arange(L), f)
    return prefill_attention_ref(q, k, v, wl.spec.scale)


@pytest.mark.parametrize("budget", [1 << 20, 512, 100, 37])
@pytest.mark.parametrize("use_rope", [False, True])
def test_chunked_prefill_against_oracle(budget, use_rope):
    wl, pc, c, t, inv_freq = _setup("llama8b", 12, 500000.0 if use_rope else None)
    rows = wl.packed_suffix(c)
    out = torch.empty_like(rows["q"])
    q_rot = torch.empty_like(rows["q"]) if use_rope else None
    n_steps = pc.prefill_chunked(c, t, wl.seq_lens, rows["q"], rows["k_new"], rows["v_new"], out,
                                 wl.spec.scale, budget, inv_freq=inv_freq, q_rot=q_rot)
    torch.cuda.synchronize()
    S = wl.seq_lens - c
    assert n_steps == len(chunk_schedule(S, budget)) == -(-int(S.sum()) // budget)
    # each query row meets the same keys in the same tile order however the
    # suffix is cut, so chunking does not change a single bit
    one = torch.empty_like(out)
    pc2 = _setup("llama8b", 12, 500000.0 if use_rope else None)[1]
    pc2.prefill_chunked(c, t, wl.seq_lens, rows["q"], rows["k_new"], rows["v_new"], one, wl.spec.scale,
                        1 << 30, inv_freq=inv_freq, q_rot=torch.empty_like(rows["q"]) if use_rope else None)
    torch.cuda.synchronize()
    assert torch.equal(one, out)
    f = inv_freq.cpu().numpy() if use_rope else None
    cu = rows["cu"]
    worst, tot, cnt = 0.0, 0.0, 0
    for r in range(len(wl.prompts)):
        ref = _oracle_rows(wl, r, int(c[r]), int(wl.seq_lens[r]), f)
        got = out[int(cu[r]):int(cu[r + 1])].float().cpu().numpy()
        err = np.abs(got - ref)
        worst = max(worst, float(err.max()))
        tot += float(err.sum())
        cnt += err.size
    mean = tot / cnt
    log(f"[chunked] budget {budget} rope {use_rope}: {n_steps} steps max_abs={worst:.3e} mean_abs={mean:.3e}")
    assert worst <= MAX_ABS and mean <= MEAN_ABS
