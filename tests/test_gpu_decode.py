"""GPU: the decode-shaped attention kernel (ilpc_paged_decode_attn) against the
fp64 oracle, on every prompt of scaled workloads, with the last q_len tokens
of each prompt as queries (q_len * Hq / Hkv up to 32), ragged lengths and
physically permuted blocks, unsplit and with each pair's keys cut into
several ranges (empty ranges and ranges where a query sees no key included);
and the automatic choice of that kernel inside ilpc_paged_prefill_attn.
"""
import sys

import numpy as np
import pytest
import torch

from oracle.attn_ref import prefill_attention_ref
from paper_2507_08523_amd import ilpc, workload
from paper_2507_08523_amd.pipeline import PagedPrefixCache

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


class Full:
    """Every prompt's K/V appended (no prefix reuse), blocks permuted."""

    def __init__(self, spec, perm_seed=1):
        self.wl = wl = workload.build(spec)
        wl.materialize("cuda")
        sp = wl.spec
        L = wl.seq_lens
        nb = int(sum(-(-int(x) // BLOCK) for x in L)) + 1
        mb = int(max(-(-int(x) // BLOCK) for x in L))
        self.pc = PagedPrefixCache(sp.n_kv_heads, sp.head_dim, nb, mb, len(wl.prompts), 16)
        c, t = self.pc.match(wl.prompts, flags=1)  # no lookup: every block new
        assert (c == 0).all()
        perm = np.random.default_rng(perm_seed).permutation(nb).astype(np.int32)
        self.tables = np.where(t >= 0, perm[np.maximum(t, 0)], -1).astype(np.int32)
        rows = wl.packed_rows([(r, 0, int(L[r])) for r in range(len(L))], with_q=False)
        b = self.pc.upload_prefill(np.zeros(len(L), np.int32), self.tables, L)
        self.pc.append(b, rows["k_new"], rows["v_new"])
        torch.cuda.synchronize()

    def queries(self, q_len):
        """Q rows of each prompt's last q_len positions, packed, and their metadata."""
        wl = self.wl
        L = wl.seq_lens
        qn = np.minimum(q_len, L).astype(np.int32)
        q = torch.cat([wl.q_rows(r, int(L[r] - qn[r]), int(L[r])) for r in range(len(L))]).contiguous()
        cu = np.zeros(len(L) + 1, np.int32)
        cu[1:] = np.cumsum(qn)
        return q, cu, qn

    def check(self, out, cu, qn, tag):
        wl = self.wl
        L = wl.seq_lens
        worst, tot, cnt = 0.0, 0.0, 0
        for r in range(len(L)):
            k, v = wl.dense_kv(r, int(L[r]))
            qr = wl.q_rows(r, int(L[r] - qn[r]), int(L[r]))
            ref = prefill_attention_ref(qr.float().cpu().numpy(), k.float().cpu().numpy(),
                                        v.float().cpu().numpy(), wl.spec.scale)
            got = out[int(cu[r]):int(cu[r + 1])].float().cpu().numpy()
            assert np.isfinite(got).all(), f"request {r}: non-finite output"
            err = np.abs(got - ref)
            worst = max(worst, float(err.max()))
            tot += float(err.sum())
            cnt += err.size
        mean = tot / cnt
        log(f"[decode] {wl.spec.name} {tag}: max_abs={worst:.3e} mean_abs={mean:.3e}")
        assert worst <= MAX_ABS and mean <= MEAN_ABS


@pytest.mark.parametrize("name,n_prompts,q_len", [
    ("tiny", 4, 1), ("tiny", 4, 8),            # D 64, G 4
    ("llama8b", 12, 1), ("llama8b", 12, 8),    # D 128, G 4
    ("qwen7b", 12, 1), ("qwen7b", 12, 4),      # G 7, ragged lengths
    ("large", 6, 1), ("large", 6, 4),          # G 8, 2112-token contexts
])
def test_decode_kernel_against_oracle(name, n_prompts, q_len):
    f = Full(workload.scaled_spec(name, n_prompts))
    sp = f.wl.spec
    q, cu, qn = f.queries(q_len)
    out = torch.empty_like(q)
    b = f.pc.upload(f.tables, cu, f.wl.seq_lens, f.wl.seq_lens - qn)
    ilpc.paged_decode_attn(q, f.pc.k_pool, f.pc.v_pool, b.block_tables, b.cu_q, b.seq_lens, int(qn.max()),
                           sp.scale, out)
    torch.cuda.synchronize()
    f.check(out, cu, qn, f"q_len {q_len}")
    # the same batch through the prefill entry (fewer pairs than compute units:
    # the persistent kernel)
    out2 = torch.empty_like(q)
    f.pc.attend(b, q, out2, sp.scale)
    torch.cuda.synchronize()
    f.check(out2, cu, qn, f"q_len {q_len}, prefill entry")


def test_decode_kernel_short_contexts_and_rejection():
    # contexts shorter than one 32-key step, and not multiples of 16
    f = Full(workload.scaled_spec("tiny", 4, instr_len=3, query_len=(2, 30)))
    sp = f.wl.spec
    q, cu, qn = f.queries(2)
    out = torch.empty_like(q)
    b = f.pc.upload(f.tables, cu, f.wl.seq_lens, f.wl.seq_lens - qn)
    ilpc.paged_decode_attn(q, f.pc.k_pool, f.pc.v_pool, b.block_tables, b.cu_q, b.seq_lens, int(qn.max()),
                           sp.scale, out)
    torch.cuda.synchronize()
    f.check(out, cu, qn, "short contexts")
    q9, cu9, qn9 = f.queries(9)                   # 9 rows x G 4 = 36 columns > 32
    b9 = f.pc.upload(f.tables, cu9, f.wl.seq_lens, f.wl.seq_lens - qn9)
    with pytest.raises(ilpc.ILPCError) as e:
        ilpc.paged_decode_attn(q9, f.pc.k_pool, f.pc.v_pool, b9.block_tables, b9.cu_q, b9.seq_lens,
                               int(qn9.max()), sp.scale, torch.empty_like(q9))
    assert e.value.code == ilpc.EUNSUP


def test_prefill_entry_takes_the_decode_kernel_for_wide_batches():
    # 64 prompts x 8 kv heads = 512 pairs >= 256 compute units: the automatic
    # path is the decode kernel, split as the library chooses when the
    # workspace has room (fewer pairs than SIMDs), unsplit with 64 bytes
    f = Full(workload.scaled_spec("large", 64))
    sp = f.wl.spec
    q, cu, qn = f.queries(1)
    out_auto, out_dec, out_small, out_one = (torch.empty_like(q) for _ in range(4))
    b = f.pc.upload(f.tables, cu, f.wl.seq_lens, f.wl.seq_lens - qn)
    f.pc.attend(b, q, out_auto, sp.scale)
    ilpc.paged_decode_attn(q, f.pc.k_pool, f.pc.v_pool, b.block_tables, b.cu_q, b.seq_lens, 1, sp.scale,
                           out_dec, n_split=0)
    ilpc.paged_prefill_attn(q, f.pc.k_pool, f.pc.v_pool, b.block_tables, b.cu_q, b.seq_lens, 1, sp.scale,
                            out_small, torch.zeros(64, dtype=torch.uint8, device="cuda"))
    ilpc.paged_decode_attn(q, f.pc.k_pool, f.pc.v_pool, b.block_tables, b.cu_q, b.seq_lens, 1, sp.scale,
                           out_one, n_split=1)
    torch.cuda.synchronize()
    assert torch.equal(out_auto, out_dec)
    assert torch.equal(out_small, out_one)
    f.check(out_auto, cu, qn, "automatic")
    f.check(out_small, cu, qn, "automatic, 64-byte workspace")


def test_prefill_entry_splits_small_decode_batches():
    # 6 prompts x 8 kv heads = 48 pairs: with a full-size workspace the entry
    # runs the split decode kernel (the same bits as the library's split
    # choice); with only the 64 queue bytes, the persistent kernel
    f = Full(workload.scaled_spec("large", 6))
    sp = f.wl.spec
    q, cu, qn = f.queries(1)
    b = f.pc.upload(f.tables, cu, f.wl.seq_lens, f.wl.seq_lens - qn)
    B, mb = len(qn), b.block_tables.shape[1]
    n = ilpc.decode_split(B, sp.n_kv_heads, mb)
    assert n > 1
    need = ilpc.attn_workspace_bytes(B, 1, sp.n_q_heads, sp.n_kv_heads, sp.head_dim)
    assert need >= 64 + ilpc.decode_workspace_bytes(B, 1, sp.n_q_heads, sp.n_kv_heads, sp.head_dim, n)
    ws = torch.zeros(need, dtype=torch.uint8, device="cuda")
    small = torch.zeros(64, dtype=torch.uint8, device="cuda")
    out_entry, out_split, out_small = (torch.empty_like(q) for _ in range(3))
    ilpc.paged_prefill_attn(q, f.pc.k_pool, f.pc.v_pool, b.block_tables, b.cu_q, b.seq_lens, 1, sp.scale,
                            out_entry, ws)
    ilpc.paged_decode_attn(q, f.pc.k_pool, f.pc.v_pool, b.block_tables, b.cu_q, b.seq_lens, 1, sp.scale,
                           out_split, n_split=0)
    ilpc.paged_prefill_attn(q, f.pc.k_pool, f.pc.v_pool, b.block_tables, b.cu_q, b.seq_lens, 1, sp.scale,
                            out_small, small)
    torch.cuda.synchronize()
    assert torch.equal(out_entry, out_split)
    assert int(ws[:64].count_nonzero()) == 0 and int(small.count_nonzero()) == 0
    f.check(out_entry, cu, qn, f"prefill entry, {n} key ranges")
    f.check(out_small, cu, qn, "prefill entry, 64-byte workspace")
