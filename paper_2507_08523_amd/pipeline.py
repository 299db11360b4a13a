"""One attention layer's prefix-cached prefill, step by step.

    match   host C++ prefix matching (cached length + block table per prompt)
    upload  one pinned host->device copy of the batch metadata
    append  HIP kv_append of the cache-missing tokens' K/V
    attend  HIP paged attention of the suffix queries

The host state (prefix cache) and device state (K/V pools) live together in
``PagedPrefixCache``.  PyTorch provides the device memory and the stream; all
computation runs in libilpc.so.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

from . import ilpc

BLOCK = ilpc.BLOCK


@dataclass
class DeviceBatch:
    """Device-side metadata of one batch (views into one int32 buffer)."""

    block_tables: object   # int32 [B, max_blocks]
    cu_q: object           # int32 [B+1]
    seq_lens: object       # int32 [B]
    start_pos: object      # int32 [B]
    max_q_len: int
    total_q: int
    B: int


class PagedPrefixCache:
    """Prefix cache (host) + paged K/V pools (device) for one attention layer."""

    def __init__(self, n_kv_heads: int, head_dim: int, num_blocks: int, max_blocks: int,
                 max_batch: int, table_log2_cap: int = 20, device="cuda", lru: bool = False):
        import torch

        self.n_kv_heads, self.head_dim = n_kv_heads, head_dim
        self.num_blocks, self.max_blocks, self.max_batch = num_blocks, max_blocks, max_batch
        self.device = torch.device(device)
        self.cache = ilpc.PrefixCache(num_blocks, table_log2_cap, lru=lru)
        self.k_pool, self.v_pool = ilpc.alloc_pools(num_blocks, n_kv_heads, head_dim, self.device)
        n = max_batch * max_blocks + 3 * max_batch + 1
        self._host = [torch.empty(n, dtype=torch.int32, pin_memory=True) for _ in range(2)]
        self._host_np = [h.numpy() for h in self._host]
        self._host_ev = [torch.cuda.Event(), torch.cuda.Event()]
        self._host_used = [False, False]
        self._flip = 0
        # Host and device staging are both double-buffered: the DeviceBatch of
        # an upload stays valid until the second upload after it.
        self._dev = [torch.empty(n, dtype=torch.int32, device=self.device) for _ in range(2)]
        self._views = {}  # (buffer, batch size) -> device views of that metadata buffer
        self._dev_tables = [None, None]  # host copy of the block table each device buffer holds
        self._steps_host = self._steps_dev = self._steps_ev = None

    # -- host ---------------------------------------------------------------
    def match(self, prompts=None, reserve=None, flags=0, packed=None):
        return self.cache.match(prompts, reserve=reserve, max_blocks=self.max_blocks, flags=flags,
                                packed=packed)[:2]

    def release(self, tables):
        """Requests finished (LRU caches): their blocks become cached or free.

        The caller orders this after the device work that reads those blocks;
        a block taken again by a later batch is only rewritten by work queued
        after it on the same stream.
        """
        self.cache.release(tables)

    # -- host -> device -----------------------------------------------------
    def upload(self, tables: np.ndarray, cu_q: np.ndarray, seq_lens: np.ndarray,
               start_pos: np.ndarray, stream=None) -> DeviceBatch:
        """Stage metadata in pinned memory and copy it with one async H2D copy.

        The returned views stay valid until the second upload after this one
        (the staging buffers alternate).  The copy is queued on ``stream``;
        work that reads the views must be ordered after it (same stream, or an
        event the caller waits on) and before that later upload's copy.
        """
        import torch

        B = int(tables.shape[0])
        if B > self.max_batch or tables.shape[1] != self.max_blocks:
            raise ilpc.ILPCError(ilpc.EINVAL, "upload: batch larger than the staging buffers")
        current = torch.cuda.current_stream(self.device)
        stream = stream or current
        i = self._flip
        self._flip ^= 1
        if self._host_used[i]:
            self._host_ev[i].synchronize()  # the copy that last read this buffer is done
        h, hn = self._host[i], self._host_np[i]
        nbt = B * self.max_blocks
        # A block table equal to the one this device buffer already holds (the
        # copy that wrote it is complete: its event was waited for above) is
        # not sent again; only the lengths are.  Decode steps keep their table.
        held = self._dev_tables[i]
        lo = nbt if held is not None and held.shape == tables.shape and np.array_equal(held, tables) else 0
        if lo == 0:
            hn[:nbt] = tables.reshape(-1)
            self._dev_tables[i] = np.array(tables, dtype=np.int32, copy=True)
        hn[nbt:nbt + B + 1] = cu_q
        hn[nbt + B + 1:nbt + 2 * B + 1] = seq_lens
        hn[nbt + 2 * B + 1:nbt + 3 * B + 1] = start_pos
        n = nbt + 3 * B + 1
        dev = self._dev[i]
        if stream == current:
            dev[lo:n].copy_(h[lo:n], non_blocking=True)
        else:
            with torch.cuda.stream(stream):
                dev[lo:n].copy_(h[lo:n], non_blocking=True)
        self._host_ev[i].record(stream)
        self._host_used[i] = True
        views = self._views.get((i, B))
        if views is None:
            views = (dev[:nbt].view(B, self.max_blocks), dev[nbt:nbt + B + 1], dev[nbt + B + 1:nbt + 2 * B + 1],
                     dev[nbt + 2 * B + 1:nbt + 3 * B + 1])
            self._views[(i, B)] = views
        q_lens = np.diff(np.asarray(cu_q, dtype=np.int64))
        return DeviceBatch(block_tables=views[0], cu_q=views[1], seq_lens=views[2], start_pos=views[3],
                           max_q_len=int(q_lens.max()) if B else 0, total_q=int(cu_q[-1]) if B else 0,
                           B=B)

    def upload_steps(self, steps, stream=None) -> list:
        """Metadata of several batches, ``steps`` = [(tables, cu_q, seq_lens, start_pos)],
        staged together and sent with one async H2D copy; returns a DeviceBatch each.

        The staging buffers grow on demand (a first call may allocate) and are
        reused: a later call first waits for the copy that last read them, and
        the batches it returned are valid only until that later call.
        """
        import torch

        stream = stream or torch.cuda.current_stream(self.device)
        sizes = [int(t.shape[0]) * self.max_blocks + 3 * int(t.shape[0]) + 1 for (t, _, _, _) in steps]
        n = int(sum(sizes))
        if self._steps_host is None or self._steps_host.numel() < n:
            if self._steps_ev is not None:
                self._steps_ev.synchronize()
            cap = max(n, 2 * (self._steps_host.numel() if self._steps_host is not None else 0))
            self._steps_host = torch.empty(cap, dtype=torch.int32, pin_memory=True)
            self._steps_dev = torch.empty(cap, dtype=torch.int32, device=self.device)
        elif self._steps_ev is not None:
            self._steps_ev.synchronize()
        h = self._steps_host.numpy()
        out, o = [], 0
        for (tables, cu_q, seq_lens, start_pos), size in zip(steps, sizes):
            B = int(tables.shape[0])
            if tables.shape[1] != self.max_blocks:
                raise ilpc.ILPCError(ilpc.EINVAL, "upload_steps: block table width differs from max_blocks")
            nbt = B * self.max_blocks
            h[o:o + nbt] = tables.reshape(-1)
            h[o + nbt:o + nbt + B + 1] = cu_q
            h[o + nbt + B + 1:o + nbt + 2 * B + 1] = seq_lens
            h[o + nbt + 2 * B + 1:o + size] = start_pos
            d = self._steps_dev
            q_lens = np.diff(np.asarray(cu_q, dtype=np.int64))
            out.append(DeviceBatch(block_tables=d[o:o + nbt].view(B, self.max_blocks),
                                   cu_q=d[o + nbt:o + nbt + B + 1],
                                   seq_lens=d[o + nbt + B + 1:o + nbt + 2 * B + 1],
                                   start_pos=d[o + nbt + 2 * B + 1:o + size],
                                   max_q_len=int(q_lens.max()) if B else 0,
                                   total_q=int(cu_q[-1]) if B else 0, B=B))
            o += size
        with torch.cuda.stream(stream):
            self._steps_dev[:n].copy_(self._steps_host[:n], non_blocking=True)
            self._steps_ev = torch.cuda.Event()
            self._steps_ev.record(stream)
        return out

    def upload_prefill(self, cached_len, tables, seq_lens, stream=None) -> DeviceBatch:
        """Metadata of a prefill: queries are positions cached_len[r]..seq_lens[r]-1."""
        seq_lens = np.asarray(seq_lens, dtype=np.int32)
        cached_len = np.asarray(cached_len, dtype=np.int32)
        cu = np.zeros(len(seq_lens) + 1, np.int32)
        cu[1:] = np.cumsum(seq_lens - cached_len)
        return self.upload(tables, cu, seq_lens, cached_len, stream)

    # -- device ---------------------------------------------------------------
    def append(self, batch: DeviceBatch, k_new, v_new, stream=None):
        ilpc.kv_append(k_new, v_new, self.k_pool, self.v_pool, batch.block_tables, batch.cu_q,
                       batch.start_pos, batch.max_q_len, stream)

    def append_rope(self, batch: DeviceBatch, k_new, v_new, inv_freq, q=None, q_out=None, stream=None):
        """kv_append with K (and Q into q_out) rotated at their absolute positions."""
        ilpc.rope_kv_append(q, q_out, k_new, v_new, self.k_pool, self.v_pool, batch.block_tables,
                            batch.cu_q, batch.start_pos, batch.max_q_len, inv_freq, stream)

    def prefill_chunked(self, cached_len, tables, seq_lens, q, k_new, v_new, out, scale: float,
                        budget: int, stream=None, inv_freq=None, q_rot=None):
        """Prefill of a matched batch in scheduler steps of at most ``budget`` tokens.

        q, k_new, v_new, out: the batch's suffix rows, packed request by
        request (as for a single pass).  Step s covers packed rows
        [s * budget, (s + 1) * budget): the rest of one request, whole
        requests, the head of another (first come, first served; the
        library's ilpc_chunk_schedule).  Each step appends its rows' K/V and
        attends its queries over every key up to its last row.  The metadata
        of all steps goes to the device in one copy, so a step costs the host
        two launches (ChunkGraph replays them all as one).  With ``inv_freq``
        the append also rotates K and Q (into ``q_rot``, which attention then
        reads).  Returns the number of steps.
        """
        meta = chunk_metadata(cached_len, tables, seq_lens, budget)
        run_chunk_steps(self, self.upload_steps(meta, stream), q, k_new, v_new, out, scale, stream, inv_freq,
                        q_rot)
        return len(meta)

    def attend(self, batch: DeviceBatch, q, out, scale: float, stream=None):
        ilpc.paged_prefill_attn(q, self.k_pool, self.v_pool, batch.block_tables, batch.cu_q,
                                batch.seq_lens, batch.max_q_len, scale, out, None, stream)

    def attend_cascade(self, batch: DeviceBatch, q, out, scale: float, shared_len: int, workspace,
                       stream=None):
        """Attention split at `shared_len` keys every request shares (see shared_prefix_len)."""
        ilpc.paged_prefill_attn_cascade(q, self.k_pool, self.v_pool, batch.block_tables, batch.cu_q,
                                        batch.seq_lens, batch.max_q_len, shared_len, scale, out,
                                        workspace, stream)

    def cascade_workspace(self, batch: DeviceBatch, n_q_heads: int):
        """A workspace for attend_cascade on this batch shape (first 128 bytes zeroed)."""
        import torch

        n = ilpc.attn_cascade_workspace_bytes(batch.B, batch.max_q_len, n_q_heads, self.n_kv_heads,
                                              self.head_dim)
        ws = torch.empty(n, dtype=torch.uint8, device=self.device)
        ws[:128].zero_()
        return ws


class DecodeGraph:
    """A run of decode steps captured once as a HIP graph and replayed as one launch.

    Step s appends the new K/V row of every request at position L_r + s and
    attends that request's one query row over keys 0 .. L_r + s.  The block
    tables must already hold blocks for every decode position (a reserve at
    match time).  All steps' metadata is staged, with one copy, into a device
    buffer the graph owns; the per-step inputs (q, k_new, v_new: [B, H, D])
    and outputs are the caller's tensors, read and written at every replay.
    Replays repeat the same appends into the same slots, so they are
    idempotent.  The capture stream keeps the default priority.
    """

    def __init__(self, pc: PagedPrefixCache, tables, seq_lens, inputs, outs, scale: float):
        import torch

        tables = np.ascontiguousarray(tables, dtype=np.int32)
        B, mb = tables.shape
        if mb != pc.max_blocks:
            raise ilpc.ILPCError(ilpc.EINVAL, "DecodeGraph: block table width differs from max_blocks")
        L = np.asarray(seq_lens, dtype=np.int32)
        n = len(inputs)
        per = B * mb + 3 * B + 1
        host = np.empty(n * per, np.int32)
        cu = np.arange(B + 1, dtype=np.int32)
        for s in range(n):
            o = s * per
            host[o:o + B * mb] = tables.reshape(-1)
            host[o + B * mb:o + B * mb + B + 1] = cu
            host[o + B * mb + B + 1:o + B * mb + 2 * B + 1] = L + s + 1
            host[o + B * mb + 2 * B + 1:o + per] = L + s
        self.meta = torch.from_numpy(host).to(pc.device)
        d = self.meta
        self.batches = []
        for s in range(n):
            o = s * per
            self.batches.append(DeviceBatch(block_tables=d[o:o + B * mb].view(B, mb),
                                            cu_q=d[o + B * mb:o + B * mb + B + 1],
                                            seq_lens=d[o + B * mb + B + 1:o + B * mb + 2 * B + 1],
                                            start_pos=d[o + B * mb + 2 * B + 1:o + per],
                                            max_q_len=1, total_q=B, B=B))
        self.stream = torch.cuda.Stream(pc.device)
        # the capture stream starts after the caller's queued work (appends, inputs)
        self.stream.wait_stream(torch.cuda.current_stream(pc.device))
        # the attention workspace is created before the capture
        ilpc.attn_workspace(pc.device, self.stream,
                            ilpc.attn_workspace_bytes(B, 1, inputs[0]["q"].shape[1], pc.n_kv_heads, pc.head_dim))
        self._run(pc, inputs, outs, scale)           # eager once on the capture stream
        self.stream.synchronize()
        self.graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(self.graph, stream=self.stream):
            self._run(pc, inputs, outs, scale)

    def _run(self, pc, inputs, outs, scale):
        for b, x, o in zip(self.batches, inputs, outs):
            pc.append(b, x["k_new"], x["v_new"], self.stream)
            pc.attend(b, x["q"], o, scale, self.stream)

    def replay(self):
        """Launch every captured step on the current stream."""
        self.graph.replay()


def chunk_metadata(cached_len, tables, seq_lens, budget: int) -> list:
    """Per scheduler step of a chunked prefill: (block tables, cu_q, seq_lens,
    start positions) of the pieces it runs, in the layout PagedPrefixCache.upload
    takes.  A piece's queries attend to every key up to its last row."""
    cached_len = np.asarray(cached_len, dtype=np.int64)
    q_lens = np.asarray(seq_lens, dtype=np.int64) - cached_len
    meta = []
    for step in chunk_schedule(q_lens, budget):
        rs = [r for (r, _, _) in step]
        n = np.array([m for (_, _, m) in step], np.int64)
        off = np.array([o for (_, o, _) in step], np.int64)
        start = cached_len[rs] + off
        cu = np.zeros(len(step) + 1, np.int32)
        cu[1:] = np.cumsum(n)
        meta.append((np.ascontiguousarray(tables[rs]), cu, (start + n).astype(np.int32), start.astype(np.int32)))
    return meta


def run_chunk_steps(pc, batches, q, k_new, v_new, out, scale, stream=None, inv_freq=None, q_rot=None):
    """Append + attention of every scheduler step, step after step on `stream`."""
    row = 0
    for b in batches:
        rows = slice(row, row + b.total_q)
        if inv_freq is None:
            pc.append(b, k_new[rows], v_new[rows], stream)
            pc.attend(b, q[rows], out[rows], scale, stream)
        else:
            pc.append_rope(b, k_new[rows], v_new[rows], inv_freq, q[rows], q_rot[rows], stream)
            pc.attend(b, q_rot[rows], out[rows], scale, stream)
        row += b.total_q


def _device_batches(meta, max_blocks, device):
    """All batches' metadata in one device buffer (one copy); DeviceBatch views."""
    import torch

    sizes = [int(t.shape[0]) * max_blocks + 3 * int(t.shape[0]) + 1 for (t, _, _, _) in meta]
    host = np.empty(int(sum(sizes)), np.int32)
    o = 0
    for (tables, cu_q, seq_lens, start_pos), size in zip(meta, sizes):
        B = int(tables.shape[0])
        nbt = B * max_blocks
        host[o:o + nbt] = np.asarray(tables).reshape(-1)
        host[o + nbt:o + nbt + B + 1] = cu_q
        host[o + nbt + B + 1:o + nbt + 2 * B + 1] = seq_lens
        host[o + nbt + 2 * B + 1:o + size] = start_pos
        o += size
    d = torch.from_numpy(host).to(device)
    out, o = [], 0
    for (tables, cu_q, _, _), size in zip(meta, sizes):
        B = int(tables.shape[0])
        nbt = B * max_blocks
        q_lens = np.diff(np.asarray(cu_q, dtype=np.int64))
        out.append(DeviceBatch(block_tables=d[o:o + nbt].view(B, max_blocks), cu_q=d[o + nbt:o + nbt + B + 1],
                               seq_lens=d[o + nbt + B + 1:o + nbt + 2 * B + 1],
                               start_pos=d[o + nbt + 2 * B + 1:o + size],
                               max_q_len=int(q_lens.max()) if B else 0, total_q=int(cu_q[-1]) if B else 0,
                               B=B))
        o += size
    return d, out


class ChunkGraph:
    """The scheduler steps of a chunked prefill captured once as a HIP graph.

    Every step (append of its rows' K/V, optionally rotated, then attention of
    its queries) is recorded in order on one default-priority capture stream
    and replayed as one launch, so the steps run back to back without the
    host's two launches per step.  The steps' metadata lives in a device
    buffer the graph owns; q, k_new, v_new, out (and q_rot) are the caller's
    tensors, read and written at every replay.  Replays repeat the same
    appends into the same slots, so they are idempotent.  Nothing in the
    capture clears memory with a memset: the attention workspace is created
    (zero-filled) before the capture and every attention call leaves its
    counters zero.
    """

    def __init__(self, pc: PagedPrefixCache, cached_len, tables, seq_lens, q, k_new, v_new, out, scale: float,
                 budget: int, inv_freq=None, q_rot=None):
        import torch

        meta = chunk_metadata(cached_len, tables, seq_lens, budget)
        self.n_steps = len(meta)
        self.meta, self.batches = _device_batches(meta, pc.max_blocks, pc.device)
        self.stream = torch.cuda.Stream(pc.device)
        self.stream.wait_stream(torch.cuda.current_stream(pc.device))
        Hq = q.shape[1]
        need = max([ilpc.attn_workspace_bytes(b.B, b.max_q_len, Hq, pc.n_kv_heads, pc.head_dim)
                    for b in self.batches] + [64])
        ilpc.attn_workspace(pc.device, self.stream, need)
        args = (pc, self.batches, q, k_new, v_new, out, scale, self.stream, inv_freq, q_rot)
        run_chunk_steps(*args)                  # eager once on the capture stream
        self.stream.synchronize()
        self.graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(self.graph, stream=self.stream):
            run_chunk_steps(*args)

    def replay(self):
        """Launch every captured step on the current stream."""
        self.graph.replay()


def chunk_schedule(q_lens, budget: int):
    """Scheduler steps of at most ``budget`` new tokens (max-num-batched-tokens):
    first come, first served over the batch's requests, as the library's
    ilpc_chunk_schedule computes them.  Returns, per step, a list of
    (request, offset into its new tokens, count)."""
    return ilpc.chunk_schedule(q_lens, budget)


def rope_inv_freq(head_dim: int, base: float):
    """fp32 angle table of plain RoPE: base^(-2i/D), i < D/2 (a model constant,
    passed to the append kernel as data)."""
    return (base ** (-np.arange(0, head_dim, 2, dtype=np.float64) / head_dim)).astype(np.float32)


def prefer_shared_split(seq_lens, max_q_len: int, n_q_heads: int, n_kv_heads: int, shared_len: int) -> bool:
    """Whether attend_cascade at shared_len should beat attend for this batch
    (the library's ilpc_prefer_shared_split: prefill-shaped, at least three
    64-key tiles shared, at most 128 own keys per request)."""
    return ilpc.prefer_shared_split(seq_lens, max_q_len, n_q_heads, n_kv_heads, shared_len)


def shared_prefix_len(cached_len, block_tables) -> int:
    """Keys at the front that every request of a batch shares (the library's
    ilpc_shared_prefix_len): the longest run of leading block ids equal across
    all rows of the host block table, capped by the shortest cached prefix."""
    return ilpc.shared_prefix_len(cached_len, block_tables)


# Sets the ICL table holds.  The paper sizes the table offline from the
# prompts' token profile and the GPU memory free for KV; 512 sets of a
# 5-demonstration Llama-3-8B prompt hold about 36 GB of KV over all 32 layers,
# a fraction of one MI355X's 288 GB.
ICL_TABLE_CAPACITY = 512


def pair_refine_stream(stream, capacity: int, batch: int):
    """Prefix-aware refinement of an ICL stream's demonstration sets.

    Requests are refined in arrival order, ``batch`` per call to the ICL table
    (each request sees the table as updated by every earlier one).  Returns the
    final (templates, demos) int32 [R, n_demos] and the PMC of each request.
    """
    n = stream.templates.shape[1]
    tab = ilpc.PairTable(capacity, n)
    out_t, out_d = np.empty_like(stream.templates), np.empty_like(stream.demos)
    pmc = np.empty(len(stream.templates), np.int32)
    for s in range(0, len(stream.templates), batch):
        e = s + batch
        out_t[s:e], out_d[s:e], pmc[s:e] = tab.refine(stream.templates[s:e], stream.demos[s:e])
    tab.close()
    return out_t, out_d, pmc


def stream_hit_rate(prompts, batch: int, pool_blocks: int | None = None) -> dict:
    """Prefix-cache hit rate of a request stream served ``batch`` prompts at a time.

    Without ``pool_blocks`` the pool holds the whole stream and nothing is
    evicted.  With it, the pool has that many blocks: each batch's requests
    finish before the next batch arrives, and cached blocks are evicted least
    recently used first.  The rate is cached prompt tokens over prompt tokens.
    """
    lru = pool_blocks is not None
    n_blocks = pool_blocks if lru else sum(-(-len(p) // BLOCK) for p in prompts) + 1
    log2cap = max(4, int(np.ceil(np.log2(n_blocks * 8 / 7 + 1))) + 1)
    cache = ilpc.PrefixCache(n_blocks, log2cap, lru=lru)
    cached = 0
    for s in range(0, len(prompts), batch):
        c, t, _ = cache.match(prompts[s:s + batch])
        cached += int(c.sum())
        if lru:
            cache.release(t)
    total = int(sum(len(p) for p in prompts))
    out = {"cached_tokens": cached, "prompt_tokens": total, "hit_rate": cached / total}
    if lru:
        out["evictions"] = cache.usage()[3]
    cache.close()
    return out


def pool_blocks_needed(wl) -> int:
    """Blocks a workload's warm + measured batches can allocate (no reuse assumed)."""
    dec = wl.spec.decode_steps
    n = sum(-(-len(p) // BLOCK) for p in wl.warm)
    n += sum(-(-(len(p) + dec) // BLOCK) for p in wl.prompts)
    return n + 1


def max_blocks_of(wl) -> int:
    dec = wl.spec.decode_steps
    return max(-(-(len(p) + dec) // BLOCK) for p in wl.prompts)
