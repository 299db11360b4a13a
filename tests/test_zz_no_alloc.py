"""ilpc_paged_prefill_attn_noalloc (the allocation-free attention call, whose
workspace is the library's static device scratch) against
ilpc_paged_prefill_attn on the same inputs: two calls in a row, the second on
a smaller batch, for the persistent prefill kernel and for split decode.

Both calls run the same kernels on the same inputs, so their outputs must be
equal bit for bit; the allocation-free output is also held to the attention
tolerance of the fp64 oracle on sampled requests.
"""
import sys

import numpy as np
import pytest
import torch

from oracle.attn_ref import decode_step_ref, prefill_attention_ref
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


def _prefill(spec):
    """Warm + measured batch of `spec` appended into fresh pools."""
    wl = workload.build(spec)
    wl.materialize("cuda")
    sp = wl.spec
    pc = PagedPrefixCache(sp.n_kv_heads, sp.head_dim, pool_blocks_needed(wl), max_blocks_of(wl),
                          max(len(wl.prompts), len(wl.warm), 1), 20)
    if wl.warm:
        c, t = pc.match(wl.warm)
        rows = wl.packed_warm(c)
        pc.append(pc.upload_prefill(c, t, [len(p) for p in wl.warm]), rows["k_new"], rows["v_new"])
    dec = sp.decode_steps
    c, t = pc.match(wl.prompts, reserve=[dec] * len(wl.prompts) if dec else None)
    rows = wl.packed_suffix(c)
    b = pc.upload_prefill(c, t, wl.seq_lens)
    pc.append(b, rows["k_new"], rows["v_new"])
    torch.cuda.synchronize()
    return wl, pc, c, t, rows, b


def _both(pc, b, q, scale, ws_bytes):
    ws = torch.zeros(ws_bytes, dtype=torch.uint8, device="cuda")
    ref = torch.full_like(q, float("nan"))
    ilpc.paged_prefill_attn(q, pc.k_pool, pc.v_pool, b.block_tables, b.cu_q, b.seq_lens, b.max_q_len, scale,
                            ref, ws)
    got = torch.full_like(q, float("nan"))
    ilpc.paged_prefill_attn_noalloc(q, pc.k_pool, pc.v_pool, b.block_tables, b.cu_q, b.seq_lens, b.max_q_len,
                                    scale, got)
    torch.cuda.synchronize()
    assert int(ws[:64].count_nonzero()) == 0
    return ref, got


def _check_prefill(wl, c, rows, got, requests):
    worst = 0.0
    for r in requests:
        L, P = int(wl.seq_lens[r]), int(c[r])
        k, v = wl.dense_kv(r, L)
        ref = prefill_attention_ref(wl.q_rows(r, P, L).float().cpu().numpy(), k.float().cpu().numpy(),
                                    v.float().cpu().numpy(), wl.spec.scale)
        out = got[int(rows["cu"][r]):int(rows["cu"][r + 1])].float().cpu().numpy()
        err = np.abs(out - ref)
        assert err.max() <= MAX_ABS and err.mean() <= MEAN_ABS, r
        worst = max(worst, float(err.max()))
    return worst


def test_noalloc_prefill_equals_workspace_call_twice_second_smaller():
    for spec in (workload.scaled_spec("llama8b", 24), workload.SPECS["tiny"]):
        wl, pc, c, t, rows, b = _prefill(spec)
        ref, got = _both(pc, b, rows["q"], wl.spec.scale, 64)
        assert torch.equal(got, ref), spec.name
        worst = _check_prefill(wl, c, rows, got, range(0, len(wl.prompts), 3))
        print(f"[noalloc] {spec.name}: {int(rows['q'].shape[0])} query rows, bit-identical to the "
              f"workspace call, max_abs={worst:.3e}", flush=True)
        sys.stdout.flush()


def test_noalloc_split_decode_equals_workspace_call_twice_second_smaller():
    # decode steps of small batches: few (request, kv head) pairs, so the keys
    # of each pair are split over several waves with partials in the scratch
    for n_prompts in (16, 4):
        wl, pc, c, t, rows, _ = _prefill(workload.scaled_spec("large", n_prompts, decode_steps=2))
        sp = wl.spec
        B = len(wl.prompts)
        L = wl.seq_lens.astype(np.int32)
        d = wl.decode_inputs(0)
        bd = pc.upload(t, np.arange(B + 1, dtype=np.int32), L + 1, L)
        pc.append(bd, d["k_new"], d["v_new"])
        assert ilpc.decode_split(B, sp.n_kv_heads, pc.max_blocks) > 1
        need = ilpc.attn_workspace_bytes(B, 1, sp.n_q_heads, sp.n_kv_heads, sp.head_dim)
        assert need <= ilpc.NOALLOC_SCRATCH_BYTES
        ref, got = _both(pc, bd, d["q"], sp.scale, ilpc.NOALLOC_SCRATCH_BYTES)
        assert torch.equal(got, ref), n_prompts
        worst = 0.0
        for r in range(B):
            k, v = wl.dense_kv(r, int(L[r]) + 1)
            expect = decode_step_ref(d["q"][r].float().cpu().numpy(), k.float().cpu().numpy(),
                                     v.float().cpu().numpy(), sp.scale)
            err = np.abs(got[r].float().cpu().numpy() - expect)
            assert err.max() <= MAX_ABS and err.mean() <= MEAN_ABS, r
            worst = max(worst, float(err.max()))
        print(f"[noalloc] large[{n_prompts}] decode step: split path bit-identical to the workspace call, "
              f"max_abs={worst:.3e}", flush=True)


def test_noalloc_rejects_bad_arguments():
    wl, pc, c, t, rows, b = _prefill(workload.SPECS["tiny"])
    lib = ilpc.load()
    q = rows["q"]
    rc = lib.ilpc_paged_prefill_attn_noalloc(q.data_ptr(), pc.k_pool.data_ptr(), pc.v_pool.data_ptr(),
                                             pc.num_blocks, b.block_tables.data_ptr(), pc.max_blocks,
                                             b.cu_q.data_ptr(), b.seq_lens.data_ptr(), b.B, b.max_q_len,
                                             4, 1, 96, 16, 0.125, q.data_ptr(), None)
    assert rc == ilpc.EUNSUP
    assert lib.ilpc_last_error().decode()
