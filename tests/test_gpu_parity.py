"""GPU parity: the HIP path (through the C ABI) against the fp64 oracle.

Tolerance on bf16 attention outputs: max |err| <= 2e-2 and mean |err| <= 2e-3
against the float64 oracle on the same bf16 inputs.  Prefix lengths and block
tables are compared bit-exactly, K/V appends by exact read-back.

Every workload runs at full size in the launch configuration the benchmark
times.  tiny, llama8b, the ICL stream batches and every hit-rate sweep point
are checked on every request; qwen7b, large and large_prefixwarm on a fixed seeded set of 16
requests (the extremes of cached length P and query length S, then seeded
picks) over all heads, and large's 32 decode steps on those 16 requests at
every step.  Each check logs its max and mean absolute error.
"""
import sys

import numpy as np
import pytest
import torch

from oracle.attn_ref import decode_step_ref, prefill_attention_ref
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


class Run:
    """Warm + measured pass of one workload through the library."""

    def __init__(self, spec, flags=0, perm_seed=None, table_log2_cap=20, demos=None):
        self.wl = wl = workload.build(spec, demos=demos)
        wl.materialize("cuda")
        sp = wl.spec
        nb = pool_blocks_needed(wl)
        self.pc = PagedPrefixCache(sp.n_kv_heads, sp.head_dim, nb, max_blocks_of(wl),
                                   max(len(wl.prompts), len(wl.warm), 1), table_log2_cap)
        self.perm = None
        if perm_seed is not None:  # physical ids permuted: output must not change
            self.perm = np.random.default_rng(perm_seed).permutation(nb).astype(np.int32)
        self.ref_cache = PrefixCacheRef(nb, (1 << table_log2_cap) - (1 << table_log2_cap) // 8)
        if wl.warm:
            c, t = self.pc.match(wl.warm)
            c_ref, t_ref, _ = self.ref_cache.match(wl.warm, max_blocks=self.pc.max_blocks)
            assert np.array_equal(c, c_ref) and np.array_equal(t, t_ref)
            rows = wl.packed_warm(c)
            b = self.pc.upload_prefill(c, self._phys(t), [len(p) for p in wl.warm])
            self.pc.append(b, rows["k_new"], rows["v_new"])
        dec = sp.decode_steps
        reserve = [dec] * len(wl.prompts) if dec else None
        c, t = self.pc.match(wl.prompts, reserve=reserve, flags=flags)
        c_ref, t_ref, _ = self.ref_cache.match(wl.prompts, reserve=reserve, max_blocks=self.pc.max_blocks,
                                               no_lookup=bool(flags & 1), no_register=bool(flags & 2))
        assert np.array_equal(c, c_ref), "cached lengths differ from the oracle"
        assert np.array_equal(t, t_ref), "block tables differ from the oracle"
        self.cached, self.tables = c, t
        self.rows = wl.packed_suffix(c)
        self.batch = self.pc.upload_prefill(c, self._phys(t), wl.seq_lens)
        self.pc.append(self.batch, self.rows["k_new"], self.rows["v_new"])
        self.out = torch.empty_like(self.rows["q"])
        self.attend()

    def _phys(self, t):
        if self.perm is None:
            return t
        return np.where(t >= 0, self.perm[np.maximum(t, 0)], -1).astype(np.int32)

    def attend(self):
        self.pc.attend(self.batch, self.rows["q"], self.out, self.wl.spec.scale)
        torch.cuda.synchronize()
        return self.out

    def request_rows(self, r):
        cu = self.rows["cu"]
        return self.out[int(cu[r]):int(cu[r + 1])]

    def check(self, requests, tag=""):
        wl = self.wl
        worst, tot, cnt = 0.0, 0.0, 0
        for r in requests:
            L, P = int(wl.seq_lens[r]), int(self.cached[r])
            k, v = wl.dense_kv(r, L)
            q = wl.q_rows(r, P, L)
            ref = prefill_attention_ref(q.float().cpu().numpy(), k.float().cpu().numpy(),
                                        v.float().cpu().numpy(), wl.spec.scale)
            got = self.request_rows(r).float().cpu().numpy()
            assert np.isfinite(got).all(), f"request {r}: non-finite output"
            err = np.abs(got - ref)
            worst = max(worst, float(err.max()))
            tot += float(err.sum())
            cnt += err.size
        mean = tot / max(cnt, 1)
        log(f"[parity] {wl.spec.name}{tag}: {len(requests)} requests max_abs={worst:.3e} mean_abs={mean:.3e}")
        assert worst <= MAX_ABS and mean <= MEAN_ABS
        return worst, mean


def _sample(run, n_rand, seed=0):
    c = run.cached
    S = run.wl.seq_lens - c
    picks = {int(np.argmin(c)), int(np.argmax(c)), int(np.argmin(S)), int(np.argmax(S))}
    rng = np.random.default_rng(seed)
    picks |= {int(x) for x in rng.choice(len(c), size=min(n_rand, len(c)), replace=False)}
    return sorted(picks)


def _pick(run, n, seed=0):
    """A fixed seeded set of n requests: the extremes of cached length P and
    of query length S first (argmin/argmax of each), then seeded picks."""
    c = run.cached
    S = run.wl.seq_lens - c
    picks = []
    for r in (np.argmax(S), np.argmin(c), np.argmax(c), np.argmin(S)):
        if int(r) not in picks:
            picks.append(int(r))
    for r in np.random.default_rng(seed).permutation(len(c)):
        if len(picks) == n:
            break
        if int(r) not in picks:
            picks.append(int(r))
    return picks


# Full-size runs are kept between the tests that check parts of them; only one
# is held at a time (the large batch needs about 60 GB of device memory).
_RUNS: dict = {}


def _full_run(name):
    if name not in _RUNS:
        _RUNS.clear()
        torch.cuda.empty_cache()
        _RUNS[name] = Run(name)
    return _RUNS[name]


@pytest.mark.parametrize("name", ["tiny", "llama8b"])
def test_prefill_full_check(name):
    run = Run(name)
    run.check(range(len(run.wl.prompts)))


@pytest.mark.parametrize("pair", [True, False])
def test_icl_stream_batch_full_check(pair):
    """The measured batch of the 2000-request ICL stream, demonstrations refined
    by the ICL table (or in the selector's order), checked in full."""
    from paper_2507_08523_amd.pipeline import ICL_TABLE_CAPACITY, pair_refine_stream

    sp = workload.SPECS["icl_llama8b"]
    demos = None
    if pair:
        _, demos, _ = pair_refine_stream(workload.icl_stream(sp), ICL_TABLE_CAPACITY, sp.n_prompts)
    run = Run(sp, demos=demos)
    assert run.cached.min() >= sp.instr_len
    run.check(range(len(run.wl.prompts)), tag=" pair" if pair else " naive")


def test_qwen7b_full_size_16_requests():
    run = _full_run("qwen7b")
    assert (run.wl.seq_lens - run.cached).min() >= 20
    picks = _pick(run, 16)
    assert len(picks) == 16
    run.check(picks, tag=" 16 requests")


SWEEP_PARTS = 4


@pytest.mark.parametrize("name,part", [(f"sweep{p}", i) for p in (0, 25, 50, 75, 100)
                                       for i in range(SWEEP_PARTS)])
def test_sweep_full_size_every_request(name, part):
    """Every one of the 128 requests of each hit-rate sweep point, in four
    parts of 32 (one full-size launch per point)."""
    run = _full_run(name)
    expect = {"sweep0": 0, "sweep25": 256, "sweep50": 496, "sweep75": 736, "sweep100": 976}[name]
    assert (run.cached == expect).all()
    B = len(run.wl.prompts)
    assert B == 128
    n = B // SWEEP_PARTS
    run.check(range(part * n, (part + 1) * n), tag=f" requests {part * n}..{(part + 1) * n - 1}")


LARGE_PICKS, LARGE_PARTS = 16, 8


@pytest.mark.parametrize("part", range(LARGE_PARTS))
def test_large_prefill_16_requests(part):
    """The large batch (512 prompts x 2112 tokens, 64 q / 8 kv heads) at full
    size: 16 seeded requests spanning min/max P and S, all heads, in parts."""
    run = _full_run("large")
    picks = _pick(run, LARGE_PICKS)
    assert len(picks) == LARGE_PICKS
    n = LARGE_PICKS // LARGE_PARTS
    run.check(picks[part * n:(part + 1) * n], tag=f" prefill picks {part * n}..{(part + 1) * n - 1}")


def test_large_decode_every_step_16_requests():
    """32 decode steps of the whole large batch (one query per prompt over the
    grown context); the same 16 requests checked at every step."""
    run = _full_run("large")
    wl, pc = run.wl, run.pc
    picks = _pick(run, LARGE_PICKS)
    B, steps = len(wl.prompts), wl.spec.decode_steps
    assert steps == 32
    L = wl.seq_lens.astype(np.int32)
    cu = np.arange(B + 1, dtype=np.int32)
    dense = {}
    for r in picks:
        k, v = wl.dense_kv(r, int(L[r]) + steps)
        dense[r] = (k.float().cpu().numpy(), v.float().cpu().numpy())
    worst, tot, cnt = 0.0, 0.0, 0
    for s in range(steps):
        d = wl.decode_inputs(s)
        b = pc.upload(run.tables, cu, L + s + 1, L + s)
        pc.append(b, d["k_new"], d["v_new"])
        out = torch.empty_like(d["q"])
        pc.attend(b, d["q"], out, wl.spec.scale)
        torch.cuda.synchronize()
        got_all = out.float().cpu().numpy()
        q_all = d["q"].float().cpu().numpy()
        for r in picks:
            n = int(L[r]) + s + 1
            k, v = dense[r]
            ref = decode_step_ref(q_all[r], k[:n], v[:n], wl.spec.scale)
            err = np.abs(got_all[r] - ref)
            assert np.isfinite(got_all[r]).all(), (s, r)
            worst = max(worst, float(err.max()))
            tot += float(err.sum())
            cnt += err.size
            assert err.max() <= MAX_ABS and err.mean() <= MEAN_ABS, (s, r)
    log(f"[parity] large decode: {steps} steps x {len(picks)} requests max_abs={worst:.3e} "
        f"mean_abs={tot / cnt:.3e}")
    _RUNS.clear()
    torch.cuda.empty_cache()


PREFIXWARM_PARTS = 2


@pytest.mark.parametrize("part", range(PREFIXWARM_PARTS))
def test_large_prefixwarm_16_requests(part):
    """The large shapes with each prompt's own 2048-token prefix cached (512 x
    64 suffix queries over 2112 keys): 16 seeded requests, all heads."""
    run = _full_run("large_prefixwarm")
    assert (run.cached == 2048).all()
    picks = _pick(run, LARGE_PICKS)
    n = LARGE_PICKS // PREFIXWARM_PARTS
    run.check(picks[part * n:(part + 1) * n], tag=f" picks {part * n}..{(part + 1) * n - 1}")
    if part == PREFIXWARM_PARTS - 1:
        _RUNS.clear()
        torch.cuda.empty_cache()


def test_kv_append_read_back_bit_exact():
    run = Run(workload.scaled_spec("llama8b", 24))
    bt = torch.from_numpy(run.tables).cuda().long()
    for r in range(len(run.wl.prompts)):
        P, L = int(run.cached[r]), int(run.wl.seq_lens[r])
        pos = torch.arange(P, L, device="cuda")
        blk = bt[r, pos // 16]
        slot = pos % 16
        k_rows = run.pc.k_pool[blk, :, slot, :]                 # [S, Hkv, D]
        v_rows = run.pc.v_pool[blk, :, :, slot]                 # [S, Hkv, D]
        cu = run.rows["cu"]
        assert torch.equal(k_rows, run.rows["k_new"][int(cu[r]):int(cu[r + 1])])
        assert torch.equal(v_rows, run.rows["v_new"][int(cu[r]):int(cu[r + 1])])


@pytest.mark.parametrize("D", [64, 128])
def test_kv_append_partial_blocks_leave_neighbours(D):
    # runs starting mid-block, single tokens, and a run spanning three blocks
    torch.manual_seed(0)
    Hkv, NB, MB = 2, 12, 4
    k_pool = torch.full((NB, Hkv, 16, D), 7.0, dtype=torch.bfloat16, device="cuda")
    v_pool = torch.full((NB, Hkv, D, 16), 7.0, dtype=torch.bfloat16, device="cuda")
    starts, lens = [5, 0, 15, 31], [1, 16, 18, 2]
    tables = torch.tensor([[0, 1, 2, 3], [4, 5, -1, -1], [6, 7, 8, -1], [9, 10, 11, -1]],
                          dtype=torch.int32, device="cuda")
    cu = torch.tensor(np.concatenate([[0], np.cumsum(lens)]), dtype=torch.int32, device="cuda")
    k_new = torch.randn(sum(lens), Hkv, D, device="cuda").to(torch.bfloat16)
    v_new = torch.randn(sum(lens), Hkv, D, device="cuda").to(torch.bfloat16)
    ilpc.kv_append(k_new, v_new, k_pool, v_pool, tables,
                   cu, torch.tensor(starts, dtype=torch.int32, device="cuda"), max(lens))
    torch.cuda.synchronize()
    expect_k = torch.full_like(k_pool, 7.0)
    expect_v = torch.full_like(v_pool, 7.0)
    tb = tables.cpu().numpy()
    row = 0
    for r, (s, n) in enumerate(zip(starts, lens)):
        for p in range(s, s + n):
            b = int(tb[r, p // 16])
            expect_k[b, :, p % 16, :] = k_new[row]
            expect_v[b, :, :, p % 16] = v_new[row]
            row += 1
    assert torch.equal(k_pool, expect_k) and torch.equal(v_pool, expect_v)


def test_prefix_cached_rows_bit_identical_to_full_prefill():
    spec = workload.scaled_spec("llama8b", 16)
    cached = Run(spec)
    full = Run(spec, flags=ilpc.NO_LOOKUP)
    assert (full.cached == 0).all() and (cached.cached > 0).all()
    for r in range(len(cached.wl.prompts)):
        P = int(cached.cached[r])
        a = cached.request_rows(r)
        b = full.request_rows(r)[P:]
        assert torch.equal(a, b), r


def test_physical_block_permutation_and_rerun_bit_identical():
    spec = workload.scaled_spec("qwen7b", 12)
    a = Run(spec)
    b = Run(spec, perm_seed=3)
    assert torch.equal(a.out, b.out)
    first = a.out.clone()
    assert torch.equal(a.attend(), first)


def test_upload_views_survive_the_next_upload():
    """The metadata staging alternates between two buffers, so a batch's views
    stay valid across the next upload (here: other prompts' metadata)."""
    run = Run("tiny")
    first = run.out.clone()
    # the same tables as a full prefill: other query offsets and start positions
    b2 = run.pc.upload_prefill(np.zeros_like(run.cached), run.tables, run.wl.seq_lens)
    torch.cuda.synchronize()
    assert not torch.equal(b2.cu_q, run.batch.cu_q)
    assert torch.equal(run.attend(), first)


def test_fully_cached_prompt_and_ragged_group():
    # L % 16 == 0 and already registered: S = 16 recomputed; G = 7 columns
    spec = workload.WorkloadSpec(name="capcase", n_q_heads=28, n_kv_heads=4, head_dim=128, n_prompts=3,
                                 instr_len=96, n_demos=0, demo_len=0, pool_size=0, query_len=(0, 0),
                                 warm="own_prefix", own_prefix_len=96, seed=9)
    run = Run(spec)
    assert (run.cached == 80).all()
    run.check(range(3))


def test_empty_and_zero_length_requests():
    run = Run("tiny")
    wl = run.wl
    # B == 0 is a no-op
    e = torch.zeros(0, wl.spec.n_q_heads, wl.spec.head_dim, dtype=torch.bfloat16, device="cuda")
    z32 = torch.zeros(1, dtype=torch.int32, device="cuda")
    ilpc.paged_prefill_attn(e, run.pc.k_pool, run.pc.v_pool,
                            torch.zeros(0, run.pc.max_blocks, dtype=torch.int32, device="cuda"), z32,
                            torch.zeros(0, dtype=torch.int32, device="cuda"), 0, wl.spec.scale, e.clone())
    # requests 1 and 3 have no queries: the others are unchanged, nothing else is written
    cu = run.rows["cu"].copy()
    keep = [0, 2]
    rows = torch.cat([run.request_rows(r) for r in keep])
    qs = torch.cat([run.rows["q"][int(cu[r]):int(cu[r + 1])] for r in keep])
    new_cu = np.array([0, 32, 32, 64, 64], np.int32)
    out = torch.full_like(qs, float("nan"))
    ilpc.paged_prefill_attn(qs, run.pc.k_pool, run.pc.v_pool, run.batch.block_tables,
                            torch.from_numpy(new_cu).cuda(), run.batch.seq_lens, 32, wl.spec.scale, out)
    torch.cuda.synchronize()
    assert torch.equal(out, rows)


def test_abi_rejects_bad_arguments_on_device():
    # every case is refused by host-side validation before any launch
    run = Run("tiny")
    b, pc, q = run.batch, run.pc, run.rows["q"]
    lib = ilpc.load()

    ws = torch.zeros(64, dtype=torch.uint8, device="cuda")

    def call(q_ptr, Hq, Hkv, D, ws_ptr=None, ws_bytes=0):
        return lib.ilpc_paged_prefill_attn(q_ptr, pc.k_pool.data_ptr(), pc.v_pool.data_ptr(),
                                           pc.num_blocks, b.block_tables.data_ptr(), pc.max_blocks,
                                           b.cu_q.data_ptr(), b.seq_lens.data_ptr(), b.B, b.max_q_len,
                                           Hq, Hkv, D, 16, 0.125, run.out.data_ptr(), ws_ptr, ws_bytes, None)

    assert call(q.data_ptr(), 4, 1, 96) == ilpc.EUNSUP       # head_dim
    assert call(q.data_ptr() + 2, 4, 1, 64) == ilpc.EINVAL   # misaligned Q
    assert call(q.data_ptr(), 6, 4, 64) == ilpc.EUNSUP       # Hq % Hkv != 0
    assert call(None, 4, 1, 64) == ilpc.EINVAL               # NULL
    assert call(q.data_ptr(), 4, 1, 64) == ilpc.EINVAL       # no workspace
    assert call(q.data_ptr(), 4, 1, 64, ws.data_ptr(), 32) == ilpc.EINVAL       # short workspace
    assert call(q.data_ptr(), 4, 1, 64, ws.data_ptr() + 4, 60) == ilpc.EINVAL   # misaligned workspace
    assert lib.ilpc_last_error().decode()


def test_work_queue_workspace_reused_and_left_zeroed():
    # The persistent attention kernel hands out work items from counters in the
    # workspace and the last workgroup clears them: back-to-back calls on one
    # workspace, and calls on a second stream with their own workspace, give
    # identical outputs and leave every workspace zero-filled.
    run = Run("qwen7b")
    b, pc, q, scale = run.batch, run.pc, run.rows["q"], run.wl.spec.scale
    ws = torch.zeros(ilpc.attn_workspace_bytes(b.B, b.max_q_len, 28, 4, 128), dtype=torch.uint8, device="cuda")
    outs = []
    for _ in range(3):
        out = torch.empty_like(q)
        ilpc.paged_prefill_attn(q, pc.k_pool, pc.v_pool, b.block_tables, b.cu_q, b.seq_lens, b.max_q_len,
                                scale, out, ws)
        outs.append(out)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        out = torch.empty_like(q)
        ilpc.paged_prefill_attn(q, pc.k_pool, pc.v_pool, b.block_tables, b.cu_q, b.seq_lens, b.max_q_len,
                                scale, out, None, side)
        outs.append(out)
    torch.cuda.synchronize()
    for o in outs[1:]:
        assert torch.equal(o, outs[0])
    assert int(ws.count_nonzero()) == 0
    assert int(ilpc.attn_workspace(None, side).count_nonzero()) == 0


@pytest.mark.parametrize("n_prompts", [1, 3, 7, 9, 13, 260, 300])
def test_item_assignment_and_queue_reset(n_prompts):
    """tiny gives one work item per request.  Up to the number of compute
    units, every workgroup takes one item by position (fewer items than
    queues, uneven queues); 260 and 300 items go through the queues, where
    the workgroups left after the first round take the remaining items from
    other XCDs' queues or stop on the drained-queue count.  Every request
    matches the oracle, twice in a row on one workspace, and the workspace is
    left zero-filled."""
    run = Run(workload.scaled_spec("tiny", n_prompts))
    b, pc, q, scale = run.batch, run.pc, run.rows["q"], run.wl.spec.scale
    ws = torch.zeros(64, dtype=torch.uint8, device="cuda")
    for rep in range(2):
        run.out.fill_(0)
        ilpc.paged_prefill_attn(q, pc.k_pool, pc.v_pool, b.block_tables, b.cu_q, b.seq_lens, b.max_q_len,
                                scale, run.out, ws)
        torch.cuda.synchronize()
        run.check(range(n_prompts), tag=f" call {rep}")
        assert int(ws.count_nonzero()) == 0


# -- shared-prefix split (cascade) -------------------------------------------

def _cascade(run, shared_len=None):
    from paper_2507_08523_amd.pipeline import shared_prefix_len

    sl = shared_prefix_len(run.cached, run._phys(run.tables)) if shared_len is None else shared_len
    ws = run.pc.cascade_workspace(run.batch, run.wl.spec.n_q_heads)
    out = torch.full_like(run.rows["q"], float("nan"))
    run.pc.attend_cascade(run.batch, run.rows["q"], out, run.wl.spec.scale, sl, ws)
    torch.cuda.synchronize()
    return sl, out, ws


@pytest.mark.parametrize("name", ["tiny", "llama8b", "sweep100", "qwen7b"])
def test_cascade_against_oracle(name):
    # All query rows of the batch attend to the shared prefix in one pass, then
    # each request to its own keys, merged by rescaling: same result as the
    # single pass within the tolerance, and the queue counters left zeroed.
    run = Run(name)
    sl, out, ws = _cascade(run)
    log(f"[cascade] {name}: shared_len={sl}")
    assert sl > 0
    run.out = out
    run.check(range(len(run.wl.prompts)) if name in ("tiny", "llama8b") else _sample(run, 8), tag=" cascade")
    assert int(ws[:128].count_nonzero()) == 0


@pytest.mark.parametrize("shared_len", [16, 48, 112])
def test_cascade_split_inside_a_tile(shared_len):
    # Split points that cut a 64-key tile: the shared half masks keys past the
    # split, the suffix half the keys before it.
    run = Run("llama8b")
    sl, out, _ = _cascade(run, shared_len)
    run.out = out
    run.check(range(0, len(run.wl.prompts), 4), tag=f" cascade@{sl}")


def test_cascade_zero_shared_len_is_the_single_pass():
    run = Run("llama8b")
    _, out, _ = _cascade(run, 0)
    assert torch.equal(out, run.attend())


def test_cascade_abi_rejections():
    run = Run("tiny")
    b, pc, q = run.batch, run.pc, run.rows["q"]
    lib = ilpc.load()
    ws = pc.cascade_workspace(b, run.wl.spec.n_q_heads)

    def call(shared_len, ws_bytes):
        return lib.ilpc_paged_prefill_attn_cascade(
            q.data_ptr(), pc.k_pool.data_ptr(), pc.v_pool.data_ptr(), pc.num_blocks, b.block_tables.data_ptr(),
            pc.max_blocks, b.cu_q.data_ptr(), b.seq_lens.data_ptr(), b.B, b.max_q_len, 4, 1, 64, 16, shared_len,
            0.125, run.out.data_ptr(), ws.data_ptr(), ws_bytes, None)

    assert call(8, ws.numel()) == ilpc.EINVAL                          # not a multiple of 16
    assert call(-16, ws.numel()) == ilpc.EINVAL
    assert call(16 * (pc.max_blocks + 1), ws.numel()) == ilpc.EINVAL   # past the table
    assert call(64, ws.numel() - 1) == ilpc.EINVAL                      # short workspace
    assert call(64, ws.numel()) == ilpc.OK
    torch.cuda.synchronize()


def test_cascade_decode_steps_against_oracle():
    # Decode over a prefix all prompts share: every step splits at the shared
    # prefix (one query row per prompt, all rows in one shared pass).
    from paper_2507_08523_amd.pipeline import shared_prefix_len

    run = Run(workload.scaled_spec("sweep100_decode", 32, decode_steps=6))
    wl, pc = run.wl, run.pc
    B = len(wl.prompts)
    L = wl.seq_lens.astype(np.int32)
    cu = np.arange(B + 1, dtype=np.int32)
    sl = shared_prefix_len(run.cached, run.tables)
    assert sl == 976
    ws = torch.zeros(ilpc.attn_cascade_workspace_bytes(B, 1, wl.spec.n_q_heads, wl.spec.n_kv_heads,
                                                       wl.spec.head_dim), dtype=torch.uint8, device="cuda")
    worst = 0.0
    for s in range(wl.spec.decode_steps):
        d = wl.decode_inputs(s)
        b = pc.upload(run.tables, cu, L + s + 1, L + s)
        pc.append(b, d["k_new"], d["v_new"])
        out = torch.full_like(d["q"], float("nan"))
        pc.attend_cascade(b, d["q"], out, wl.spec.scale, sl, ws)
        torch.cuda.synchronize()
        for r in (0, 7, B - 1):
            k, v = wl.dense_kv(r, int(L[r]) + s + 1)
            ref = decode_step_ref(d["q"][r].float().cpu().numpy(), k.float().cpu().numpy(),
                                  v.float().cpu().numpy(), wl.spec.scale)
            err = np.abs(out[r].float().cpu().numpy() - ref)
            worst = max(worst, float(err.max()))
            assert err.max() <= MAX_ABS and err.mean() <= MEAN_ABS, (s, r)
    log(f"[parity] sweep100 decode (cascade): {wl.spec.decode_steps} steps, max_abs={worst:.3e}")


@pytest.mark.parametrize("q_pattern", ["ragged", "small", "with_empty"])
def test_cascade_fused_many_requests_per_item(q_pattern):
    # Prefill-shaped cascades with at least three shared 64-key tiles run as
    # one launch whose items are 256 columns of the whole batch: here each
    # request keeps only its last k queries (k ragged, small so that one item
    # spans up to 64 requests, or zero for some requests), so items mix many
    # requests and request tiles are masked to their own columns.
    from paper_2507_08523_amd.pipeline import shared_prefix_len

    run = Run(workload.scaled_spec("sweep100", 40))
    wl, pc, sp = run.wl, run.pc, run.wl.spec
    B = len(wl.prompts)
    L = wl.seq_lens.astype(np.int64)
    S = L - run.cached
    rng = np.random.default_rng({"ragged": 1, "small": 2, "with_empty": 3}[q_pattern])
    if q_pattern == "ragged":
        k = rng.integers(1, S + 1)
    elif q_pattern == "small":
        k = rng.integers(1, 17, B)
        k[0] = 16  # max_q_len * G = 64: still prefill-shaped, so the one-launch split
    else:
        k = np.where(rng.random(B) < 0.3, 0, rng.integers(1, S + 1))
    k = np.minimum(k, S).astype(np.int64)
    cu = np.zeros(B + 1, np.int64)
    cu[1:] = np.cumsum(k)
    rows = wl.packed_rows([(r, int(L[r] - k[r]), int(L[r])) for r in range(B)])
    q = rows["q"]
    b = pc.upload(run.tables, cu.astype(np.int32), L.astype(np.int32), (L - k).astype(np.int32))
    sl = shared_prefix_len(run.cached, run.tables)
    assert sl == 976
    ws = pc.cascade_workspace(b, sp.n_q_heads)
    out = torch.full_like(q, float("nan"))
    pc.attend_cascade(b, q, out, sp.scale, sl, ws)
    torch.cuda.synchronize()
    worst, tot, cnt = 0.0, 0.0, 0
    for r in range(B):
        if k[r] == 0:
            continue
        kk, vv = wl.dense_kv(r, int(L[r]))
        ref = prefill_attention_ref(wl.q_rows(r, int(L[r] - k[r]), int(L[r])).float().cpu().numpy(),
                                    kk.float().cpu().numpy(), vv.float().cpu().numpy(), sp.scale)
        got = out[int(cu[r]):int(cu[r + 1])].float().cpu().numpy()
        assert np.isfinite(got).all(), r
        err = np.abs(got - ref)
        worst = max(worst, float(err.max()))
        tot += float(err.sum())
        cnt += err.size
    log(f"[parity] sweep100[40] cascade, {q_pattern} queries ({int(k.sum())} rows, {int((k == 0).sum())} "
        f"empty requests): max_abs={worst:.3e} mean_abs={tot / cnt:.3e}")
    assert worst <= MAX_ABS and tot / cnt <= MEAN_ABS
