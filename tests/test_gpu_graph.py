"""GPU: decode steps captured as a HIP graph (pipeline.DecodeGraph) replay to
exactly the eager results, replay after replay with eager work in between,
on both decode paths (the one-wave-per-pair kernel and the persistent kernel
with its work-queue workspace), and agree with the fp64 oracle.  The same
holds for the scheduler steps of a chunked prefill (pipeline.ChunkGraph),
with and without RoPE in the append.
"""
import sys

import numpy as np
import pytest
import torch

from oracle.attn_ref import decode_step_ref
from paper_2507_08523_amd import ilpc, workload
from paper_2507_08523_amd.pipeline import DecodeGraph, PagedPrefixCache, max_blocks_of, pool_blocks_needed

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


# 16 prompts x 8 kv heads = 128 pairs (fewer than the compute units: the
# persistent kernel); 64 prompts: 512 pairs (the decode kernel)
@pytest.mark.parametrize("n_prompts", [16, 64])
def test_decode_graph_replays_equal_eager(n_prompts):
    wl = workload.build(workload.scaled_spec("sweep100_decode", n_prompts, decode_steps=6))
    wl.materialize("cuda")
    sp = wl.spec
    dec = sp.decode_steps
    pc = PagedPrefixCache(sp.n_kv_heads, sp.head_dim, pool_blocks_needed(wl), max_blocks_of(wl),
                          max(len(wl.prompts), len(wl.warm)), 16)
    if wl.warm:
        c, t = pc.match(wl.warm)
        rows = wl.packed_warm(c)
        pc.append(pc.upload_prefill(c, t, [len(p) for p in wl.warm]), rows["k_new"], rows["v_new"])
    B = len(wl.prompts)
    c, t = pc.match(wl.prompts, reserve=[dec] * B)
    rows = wl.packed_suffix(c)
    L = wl.seq_lens.astype(np.int32)
    pc.append(pc.upload_prefill(c, t, L), rows["k_new"], rows["v_new"])
    dec_in = [wl.decode_inputs(s) for s in range(dec)]
    cu = np.arange(B + 1, dtype=np.int32)
    eager = []
    for s in range(dec):
        b = pc.upload(t, cu, L + s + 1, L + s)
        pc.append(b, dec_in[s]["k_new"], dec_in[s]["v_new"])
        o = torch.empty_like(dec_in[s]["q"])
        pc.attend(b, dec_in[s]["q"], o, sp.scale)
        eager.append(o)
    torch.cuda.synchronize()

    outs = [torch.empty_like(x["q"]) for x in dec_in]
    g = DecodeGraph(pc, t, L, dec_in, outs, sp.scale)
    torch.cuda.synchronize()
    for rep in range(3):
        for o in outs:
            o.zero_()
        g.replay()
        torch.cuda.synchronize()
        for s in range(dec):
            assert torch.equal(outs[s], eager[s]), f"replay {rep}, step {s} differs from the eager run"
        # eager work on the default stream between replays
        b = pc.upload(t, cu, L + 1, L)
        scratch = torch.empty_like(dec_in[0]["q"])
        pc.attend(b, dec_in[0]["q"], scratch, sp.scale)
        torch.cuda.synchronize()
        assert torch.equal(scratch, eager[0])
    worst = 0.0
    for r in (0, B // 2, B - 1):
        for s in (0, dec - 1):
            k, v = wl.dense_kv(r, int(L[r]) + s + 1)
            ref = decode_step_ref(dec_in[s]["q"][r].float().cpu().numpy(), k.float().cpu().numpy(),
                                  v.float().cpu().numpy(), sp.scale)
            err = np.abs(outs[s][r].float().cpu().numpy() - ref)
            worst = max(worst, float(err.max()))
            assert err.max() <= MAX_ABS and err.mean() <= MEAN_ABS
    log(f"[graph] {sp.name}: {dec} captured decode steps, 3 replays equal to eager, oracle max_abs={worst:.3e}")


@pytest.mark.parametrize("budget,rope", [(1024, False), (300, True)])
def test_chunk_graph_replays_equal_eager(budget, rope):
    """The steps of a chunked prefill captured as one graph (pipeline.ChunkGraph):
    every replay equals the eager chunked run bit for bit, with eager work on
    the default stream between replays, and agrees with the fp64 oracle."""
    from oracle.attn_ref import prefill_attention_ref
    from oracle.rope_ref import rope
    from paper_2507_08523_amd.pipeline import ChunkGraph, rope_inv_freq

    wl = workload.build(workload.scaled_spec("llama8b", 24))
    wl.materialize("cuda")
    sp = wl.spec
    pc = PagedPrefixCache(sp.n_kv_heads, sp.head_dim, pool_blocks_needed(wl), max_blocks_of(wl),
                          max(len(wl.prompts), len(wl.warm)), 16)
    inv = torch.from_numpy(rope_inv_freq(sp.head_dim, 5e5)).cuda() if rope else None
    c, t = pc.match(wl.warm)
    rows = wl.packed_warm(c)
    b = pc.upload_prefill(c, t, [len(p) for p in wl.warm])
    if rope:
        pc.append_rope(b, rows["k_new"], rows["v_new"], inv)
    else:
        pc.append(b, rows["k_new"], rows["v_new"])
    c, t = pc.match(wl.prompts)
    rows = wl.packed_suffix(c)
    L = wl.seq_lens.astype(np.int32)
    q, k_new, v_new = rows["q"], rows["k_new"], rows["v_new"]
    q_rot = torch.empty_like(q) if rope else None
    eager = torch.full_like(q, float("nan"))
    n = pc.prefill_chunked(c, t, L, q, k_new, v_new, eager, sp.scale, budget, None, inv, q_rot)
    torch.cuda.synchronize()
    assert n == -(-int((L - c).sum()) // budget)
    eager_rot = q_rot.clone() if rope else None

    out = torch.empty_like(q)
    g = ChunkGraph(pc, c, t, L, q, k_new, v_new, out, sp.scale, budget, inv, q_rot)
    torch.cuda.synchronize()
    assert g.n_steps == n
    for rep in range(3):
        out.fill_(float("nan"))
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(out, eager), f"replay {rep} differs from the eager chunked run"
        if rope:
            assert torch.equal(q_rot, eager_rot)
        # eager work on the default stream between replays
        other = torch.empty_like(q)
        pc.prefill_chunked(c, t, L, q, k_new, v_new, other, sp.scale, budget, None, inv, q_rot)
        torch.cuda.synchronize()
        assert torch.equal(other, eager)
    worst = 0.0
    for r in (0, len(L) // 2, len(L) - 1):
        P, Lr = int(c[r]), int(L[r])
        k, v = wl.dense_kv(r, Lr)
        qr = wl.q_rows(r, P, Lr).float().cpu().numpy()
        k = k.float().cpu().numpy()
        v = v.float().cpu().numpy()
        if rope:
            f = inv.cpu().numpy()
            qr = rope(qr, np.arange(P, Lr), f)
            k = rope(k, np.arange(Lr), f)
        ref = prefill_attention_ref(qr, k, v, sp.scale)
        got = out[int(rows["cu"][r]):int(rows["cu"][r + 1])].float().cpu().numpy()
        err = np.abs(got - ref)
        assert err.max() <= MAX_ABS and err.mean() <= MEAN_ABS, r
        worst = max(worst, float(err.max()))
    log(f"[graph] chunked prefill llama8b[24] budget {budget}{' rope' if rope else ''}: {n} steps, "
        f"3 replays bit-identical, max_abs={worst:.3e}")
