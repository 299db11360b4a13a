"""ctypes binding of libilpc.so (C ABI in include/ilpc.h).

Argument marshalling only: every step of the path runs in the library (host
C++ prefix matching, HIP kernels for K/V append and attention).  Loading fails
loudly if the library has not been built; there is no fallback.

Device tensors are torch tensors (PyTorch supplies device memory and streams);
they are checked for dtype, device, contiguity and shape before their
pointers are handed over.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libilpc.so")

OK, EINVAL, ENOSPC, ETABLE, EUNSUP, EHIP = 0, -1, -2, -3, -4, -5
NO_LOOKUP, NO_REGISTER = 1, 2
BLOCK = 16
_NAMES = {EINVAL: "EINVAL", ENOSPC: "ENOSPC", ETABLE: "ETABLE", EUNSUP: "EUNSUP", EHIP: "EHIP"}

# (name, restype, argtypes) of every exported symbol
_i32, _u32, _i64, _f32, _vp = ctypes.c_int32, ctypes.c_uint32, ctypes.c_int64, ctypes.c_float, ctypes.c_void_p
_SIGS = [
    ("ilpc_last_error", ctypes.c_char_p, []),
    ("ilpc_cache_create", _i32, [_i32, _i32, _i32, ctypes.POINTER(_vp)]),
    ("ilpc_cache_destroy", None, [_vp]),
    ("ilpc_cache_reset", _i32, [_vp]),
    ("ilpc_cache_stats", _i32, [_vp, _vp]),
    ("ilpc_cache_checkpoint", _i32, [_vp, _vp]),
    ("ilpc_cache_rollback", _i32, [_vp, _vp]),
    ("ilpc_prefix_match", _i32, [_vp, _vp, _vp, _i32, _vp, _i32, _u32, _vp, _vp, _vp]),
    ("ilpc_kv_append", _i32, [_vp, _vp, _vp, _vp, _i32, _vp, _i32, _vp, _vp, _i32, _i32, _i32,
                              _i32, _i32, _vp]),
    ("ilpc_rope_kv_append", _i32, [_vp, _vp, _i32, _vp, _vp, _vp, _vp, _i32, _vp, _i32, _vp, _vp, _i32,
                                   _i32, _i32, _i32, _i32, _vp, _vp]),
    ("ilpc_attn_workspace_bytes", _i32, [_i32, _i32, _i32, _i32, _i32, ctypes.POINTER(ctypes.c_size_t)]),
    ("ilpc_paged_prefill_attn", _i32, [_vp, _vp, _vp, _i32, _vp, _i32, _vp, _vp, _i32, _i32, _i32,
                                       _i32, _i32, _i32, _f32, _vp, _vp, ctypes.c_size_t, _vp]),
    ("ilpc_paged_prefill_attn_noalloc", _i32, [_vp, _vp, _vp, _i32, _vp, _i32, _vp, _vp, _i32, _i32, _i32,
                                               _i32, _i32, _i32, _f32, _vp, _vp]),
    ("ilpc_paged_decode_attn", _i32, [_vp, _vp, _vp, _i32, _vp, _i32, _vp, _vp, _i32, _i32, _i32,
                                      _i32, _i32, _i32, _f32, _vp, _i32, _vp, ctypes.c_size_t, _vp]),
    ("ilpc_decode_split", _i32, [_i32, _i32, _i32, ctypes.POINTER(_i32)]),
    ("ilpc_decode_workspace_bytes", _i32, [_i32, _i32, _i32, _i32, _i32, _i32,
                                           ctypes.POINTER(ctypes.c_size_t)]),
    ("ilpc_attn_cascade_workspace_bytes", _i32, [_i32, _i32, _i32, _i32, _i32,
                                                 ctypes.POINTER(ctypes.c_size_t)]),
    ("ilpc_paged_prefill_attn_cascade", _i32, [_vp, _vp, _vp, _i32, _vp, _i32, _vp, _vp, _i32, _i32,
                                               _i32, _i32, _i32, _i32, _i32, _f32, _vp, _vp,
                                               ctypes.c_size_t, _vp]),
    ("ilpc_chunk_schedule", _i32, [_vp, _i32, _i32, _i32, _vp, _vp, _vp, _vp, ctypes.POINTER(_i32),
                                   ctypes.POINTER(_i32)]),
    ("ilpc_shared_prefix_len", _i32, [_vp, _vp, _i32, _i32, ctypes.POINTER(_i32)]),
    ("ilpc_prefer_shared_split", _i32, [_vp, _i32, _i32, _i32, _i32, _i32, ctypes.POINTER(_i32)]),
    ("ilpc_cache_create_lru", _i32, [_i32, _i32, _i32, ctypes.POINTER(_vp)]),
    ("ilpc_cache_release", _i32, [_vp, _vp, _i32, _i32]),
    ("ilpc_cache_touch", _i32, [_vp, _vp, _i32]),
    ("ilpc_cache_usage", _i32, [_vp, _vp]),
    ("ilpc_cache_lru_order", _i32, [_vp, _vp, _i32, ctypes.POINTER(_i32)]),
    ("ilpc_pair_create", _i32, [_i32, _i32, ctypes.POINTER(_vp)]),
    ("ilpc_pair_destroy", None, [_vp]),
    ("ilpc_pair_reset", _i32, [_vp]),
    ("ilpc_pair_refine", _i32, [_vp, _vp, _vp, _i32, _vp, _vp, _vp]),
    ("ilpc_pair_entries", _i32, [_vp, _vp, _vp, _i32, ctypes.POINTER(_i32)]),
]
SYMBOLS = [s[0] for s in _SIGS]

_lib = None


class ILPCError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"{_NAMES.get(code, code)}: {msg}")
        self.code = code


def load():
    """The loaded library; raises if libilpc.so is missing (build it first)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ILPCError(EINVAL, f"{LIB_PATH} is missing: run `python -m paper_2507_08523_amd.build`")
        lib = ctypes.CDLL(LIB_PATH)
        for name, res, args in _SIGS:
            fn = getattr(lib, name)
            fn.restype = res
            fn.argtypes = args
        _lib = lib
    return _lib


def _check(rc: int):
    if rc != OK:
        raise ILPCError(rc, load().ilpc_last_error().decode())


def _np_ptr(a: np.ndarray):
    return ctypes.c_void_p(a.ctypes.data) if a is not None else None


class PrefixCache:
    """Host prefix cache over a pool of ``num_blocks`` 16-token blocks.

    ``lru=True`` gives blocks a lifecycle (reference counts, a free queue and
    least-recently-used eviction of cached blocks; see ``release``).
    """

    def __init__(self, num_blocks: int, table_log2_cap: int = 20, lru: bool = False):
        lib = load()
        h = ctypes.c_void_p()
        create = lib.ilpc_cache_create_lru if lru else lib.ilpc_cache_create
        _check(create(num_blocks, BLOCK, table_log2_cap, ctypes.byref(h)))
        self._h, self.num_blocks, self.lru = h, num_blocks, lru

    def close(self):
        h, self._h = getattr(self, "_h", None), None
        if h and _lib is not None:  # (at interpreter exit the library may be gone already)
            _lib.ilpc_cache_destroy(h)

    __del__ = close

    def reset(self):
        _check(load().ilpc_cache_reset(self._h))

    def stats(self) -> dict:
        s = np.zeros(4, np.int64)
        _check(load().ilpc_cache_stats(self._h, _np_ptr(s)))
        return {"keys": int(s[0]), "next_block": int(s[1]), "capacity": int(s[2]), "num_blocks": int(s[3])}

    def release(self, block_tables):
        """Requests finished: release the blocks of each row (up to its first -1)."""
        t = np.ascontiguousarray(block_tables, dtype=np.int32)
        if t.ndim != 2:
            raise ILPCError(EINVAL, "release: block_tables must be [B, max_blocks]")
        if t.shape[0]:
            _check(load().ilpc_cache_release(self._h, _np_ptr(t), t.shape[0], t.shape[1]))

    def touch(self, block_ids):
        ids = np.ascontiguousarray(block_ids, dtype=np.int32).reshape(-1)
        _check(load().ilpc_cache_touch(self._h, _np_ptr(ids), ids.size))

    def usage(self) -> tuple:
        """(blocks in use, cached blocks, free blocks, evictions so far)."""
        u = np.zeros(4, np.int64)
        _check(load().ilpc_cache_usage(self._h, _np_ptr(u)))
        return tuple(int(x) for x in u)

    def lru_order(self) -> list:
        """Cached blocks, least recently used first."""
        out = np.zeros(max(self.num_blocks, 1), np.int32)
        n = ctypes.c_int32()
        _check(load().ilpc_cache_lru_order(self._h, _np_ptr(out), out.size, ctypes.byref(n)))
        return out[:n.value].tolist()

    def checkpoint(self) -> np.ndarray:
        m = np.zeros(2, np.int64)
        _check(load().ilpc_cache_checkpoint(self._h, _np_ptr(m)))
        return m

    def rollback(self, mark: np.ndarray):
        m = np.ascontiguousarray(mark, dtype=np.int64)
        _check(load().ilpc_cache_rollback(self._h, _np_ptr(m)))

    def match(self, prompts, reserve=None, max_blocks=None, flags=0, want_keys=False, packed=None):
        """Prefix-match a batch (list of int32 token arrays, or ``packed`` = (tokens, cu)).

        Returns (cached_len int32[B], block_tables int32[B, max_blocks], keys or None).
        """
        if packed is not None:
            tokens, cu = packed
        else:
            cu = np.zeros(len(prompts) + 1, np.int32)
            cu[1:] = np.cumsum([len(p) for p in prompts])
            tokens = np.concatenate(prompts).astype(np.int32) if prompts else np.zeros(0, np.int32)
        tokens = np.ascontiguousarray(tokens, dtype=np.int32)
        cu = np.ascontiguousarray(cu, dtype=np.int32)
        B = len(cu) - 1
        res = None if reserve is None else np.ascontiguousarray(reserve, dtype=np.int32)
        if max_blocks is None:
            L = np.diff(cu).astype(np.int64) + (0 if res is None else res)
            max_blocks = int(max(1, (L.max() + BLOCK - 1) // BLOCK)) if B else 1
        cached = np.zeros(B, np.int32)
        tables = np.zeros((B, max_blocks), np.int32)
        keys = np.zeros((B, max_blocks), np.uint64) if want_keys else None
        tok = tokens if tokens.size else np.zeros(1, np.int32)
        _check(load().ilpc_prefix_match(self._h, _np_ptr(tok), _np_ptr(cu), B, _np_ptr(res), max_blocks,
                                        flags, _np_ptr(cached), _np_ptr(tables), _np_ptr(keys)))
        return cached, tables, keys


class PairTable:
    """ICL table of prefix-aware demonstration refinement (host, library-owned).

    A demonstration is a (template id, demonstration id) pair of int32; a
    demonstration set is ``n_demos`` of them.
    """

    def __init__(self, capacity: int, n_demos: int):
        lib = load()
        h = ctypes.c_void_p()
        _check(lib.ilpc_pair_create(capacity, n_demos, ctypes.byref(h)))
        self._h, self.capacity, self.n_demos = h, capacity, n_demos

    def close(self):
        h, self._h = getattr(self, "_h", None), None
        if h and _lib is not None:
            _lib.ilpc_pair_destroy(h)

    __del__ = close

    def reset(self):
        _check(load().ilpc_pair_reset(self._h))

    def refine(self, templates, demos):
        """Refine B requests' sets in order.

        templates, demos: int32 [B, n_demos].  Returns (final templates, final
        demos) int32 [B, n_demos] and the PMC of each request int32 [B].
        """
        t = np.ascontiguousarray(templates, dtype=np.int32)
        d = np.ascontiguousarray(demos, dtype=np.int32)
        if t.ndim != 2 or t.shape != d.shape or t.shape[1] != self.n_demos:
            raise ILPCError(EINVAL, f"refine: templates and demos must both be [B, {self.n_demos}]")
        B = t.shape[0]
        ot, od = np.zeros_like(t), np.zeros_like(d)
        pmc = np.zeros(B, np.int32)
        if B:
            _check(load().ilpc_pair_refine(self._h, _np_ptr(t), _np_ptr(d), B, _np_ptr(ot), _np_ptr(od),
                                           _np_ptr(pmc)))
        return ot, od, pmc

    def entries(self):
        """Held sets, least recently used first: (templates, demos) int32 [E, n_demos]."""
        n = ctypes.c_int32()
        cap = self.capacity
        t = np.zeros((cap, self.n_demos), np.int32)
        d = np.zeros_like(t)
        _check(load().ilpc_pair_entries(self._h, _np_ptr(t), _np_ptr(d), cap, ctypes.byref(n)))
        return t[:n.value].copy(), d[:n.value].copy()


# -- host scheduling policy ---------------------------------------------------

def chunk_schedule(q_lens, budget: int):
    """Scheduler steps of at most ``budget`` new tokens (ilpc_chunk_schedule).

    Returns, per step, a list of (request, offset into its new tokens, count).
    """
    q = np.ascontiguousarray(q_lens, dtype=np.int32)
    B = int(q.shape[0])
    lib = load()
    n_p, n_s = _i32(), _i32()
    rc = lib.ilpc_chunk_schedule(_np_ptr(q), B, int(budget), 0, None, None, None, None,
                                 ctypes.byref(n_p), ctypes.byref(n_s))
    if rc != OK and n_p.value == 0:
        _check(rc)
    n = n_p.value
    req, off, ln, st = (np.empty(max(n, 1), np.int32) for _ in range(4))
    _check(lib.ilpc_chunk_schedule(_np_ptr(q), B, int(budget), n, _np_ptr(req), _np_ptr(off), _np_ptr(ln),
                                   _np_ptr(st), ctypes.byref(n_p), ctypes.byref(n_s)))
    steps = [[] for _ in range(n_s.value)]
    for k in range(n):
        steps[int(st[k])].append((int(req[k]), int(off[k]), int(ln[k])))
    return steps


def shared_prefix_len(cached_len, block_tables) -> int:
    """Keys every request shares at the front (ilpc_shared_prefix_len)."""
    c = np.ascontiguousarray(cached_len, dtype=np.int32)
    t = np.ascontiguousarray(block_tables, dtype=np.int32)
    B = int(c.shape[0])
    if t.ndim != 2 or t.shape[0] != B:
        raise ILPCError(EINVAL, "shared_prefix_len: block_tables must be [B, max_blocks]")
    out = _i32()
    _check(load().ilpc_shared_prefix_len(_np_ptr(c), _np_ptr(t), B, int(t.shape[1]), ctypes.byref(out)))
    return int(out.value)


def prefer_shared_split(seq_lens, max_q_len: int, n_q_heads: int, n_kv_heads: int, shared_len: int) -> bool:
    """Whether the shared-prefix split beats the single pass (ilpc_prefer_shared_split)."""
    L = np.ascontiguousarray(seq_lens, dtype=np.int32)
    out = _i32()
    _check(load().ilpc_prefer_shared_split(_np_ptr(L), int(L.shape[0]), int(max_q_len), int(n_q_heads),
                                           int(n_kv_heads), int(shared_len), ctypes.byref(out)))
    return bool(out.value)


# -- device steps ------------------------------------------------------------

def _dev(t, dtype, name, ndim=None):
    import torch

    if not isinstance(t, torch.Tensor) or t.device.type != "cuda":
        raise ILPCError(EINVAL, f"{name} must be a CUDA/HIP torch tensor")
    if t.dtype != dtype:
        raise ILPCError(EINVAL, f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ILPCError(EINVAL, f"{name} must be contiguous")
    if ndim is not None and t.dim() != ndim:
        raise ILPCError(EINVAL, f"{name} must have {ndim} dims, got {t.dim()}")
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    import torch

    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def alloc_pools(num_blocks: int, n_kv_heads: int, head_dim: int, device="cuda"):
    """Empty K pool [NB, Hkv, 16, D] and V pool [NB, Hkv, D, 16] (bf16)."""
    import torch

    k = torch.empty((num_blocks, n_kv_heads, BLOCK, head_dim), dtype=torch.bfloat16, device=device)
    v = torch.empty((num_blocks, n_kv_heads, head_dim, BLOCK), dtype=torch.bfloat16, device=device)
    return k, v


def kv_append(k_new, v_new, k_pool, v_pool, block_tables, cu_new, start_pos, max_new: int, stream=None):
    """Write packed new K/V rows [total, Hkv, D] into the pools (async on the stream)."""
    import torch

    NB, Hkv, bs, D = k_pool.shape
    if v_pool.shape != (NB, Hkv, D, bs) or k_new.shape[1:] != (Hkv, D) or v_new.shape != k_new.shape:
        raise ILPCError(EINVAL, "kv_append: inconsistent K/V/pool shapes")
    B = cu_new.shape[0] - 1
    if block_tables.dim() != 2 or block_tables.shape[0] != B or start_pos.shape[0] != B:
        raise ILPCError(EINVAL, "kv_append: inconsistent batch shapes")
    args = (_dev(k_new, torch.bfloat16, "k_new", 3), _dev(v_new, torch.bfloat16, "v_new", 3),
            _dev(k_pool, torch.bfloat16, "k_pool", 4), _dev(v_pool, torch.bfloat16, "v_pool", 4), NB,
            _dev(block_tables, torch.int32, "block_tables", 2), block_tables.shape[1],
            _dev(cu_new, torch.int32, "cu_new", 1), _dev(start_pos, torch.int32, "start_pos", 1),
            B, int(max_new), Hkv, D, bs, _stream(stream))
    _check(load().ilpc_kv_append(*args))


def rope_kv_append(q, q_out, k_new, v_new, k_pool, v_pool, block_tables, cu_new, start_pos, max_new: int,
                   inv_freq, stream=None):
    """Rotate new K (and Q, if given) at their positions and write K/V into the pools.

    q, q_out: [total, Hq, D] bf16 or both None (q_out may be q); inv_freq: fp32 [D/2].
    """
    import torch

    NB, Hkv, bs, D = k_pool.shape
    if v_pool.shape != (NB, Hkv, D, bs) or k_new.shape[1:] != (Hkv, D) or v_new.shape != k_new.shape:
        raise ILPCError(EINVAL, "rope_kv_append: inconsistent K/V/pool shapes")
    if (q is None) != (q_out is None):
        raise ILPCError(EINVAL, "rope_kv_append: q and q_out must both be given or both be None")
    Hq = Hkv
    if q is not None:
        Hq = q.shape[1]
        if q.shape != (k_new.shape[0], Hq, D) or q_out.shape != q.shape:
            raise ILPCError(EINVAL, "rope_kv_append: q / q_out must be [total, Hq, D] like k_new")
    if inv_freq.shape != (D // 2,):
        raise ILPCError(EINVAL, "rope_kv_append: inv_freq must be [D/2]")
    B = cu_new.shape[0] - 1
    if block_tables.dim() != 2 or block_tables.shape[0] != B or start_pos.shape[0] != B:
        raise ILPCError(EINVAL, "rope_kv_append: inconsistent batch shapes")
    qp = _dev(q, torch.bfloat16, "q", 3) if q is not None else None
    qo = _dev(q_out, torch.bfloat16, "q_out", 3) if q_out is not None else None
    args = (qp, qo, Hq, _dev(k_new, torch.bfloat16, "k_new", 3), _dev(v_new, torch.bfloat16, "v_new", 3),
            _dev(k_pool, torch.bfloat16, "k_pool", 4), _dev(v_pool, torch.bfloat16, "v_pool", 4), NB,
            _dev(block_tables, torch.int32, "block_tables", 2), block_tables.shape[1],
            _dev(cu_new, torch.int32, "cu_new", 1), _dev(start_pos, torch.int32, "start_pos", 1),
            B, int(max_new), Hkv, D, bs, _dev(inv_freq, torch.float32, "inv_freq", 1), _stream(stream))
    _check(load().ilpc_rope_kv_append(*args))


def attn_workspace_bytes(B, max_q_len, Hq, Hkv, D) -> int:
    n = ctypes.c_size_t()
    _check(load().ilpc_attn_workspace_bytes(B, max_q_len, Hq, Hkv, D, ctypes.byref(n)))
    return int(n.value)


_workspaces = {}
_ws_bytes = {}


def attn_workspace(device=None, stream=None, nbytes: int = 64):
    """An attention workspace of at least `nbytes` kept for one (device, stream)
    pair, its first 64 bytes zero-filled.

    The attention call leaves those bytes zero-filled again (the rest is
    scratch), so one buffer serves every call issued on that stream; calls on
    different streams get different buffers because concurrent calls must not
    share one.  A request for more bytes than the kept buffer holds replaces
    it with a larger one (an allocation: make the first call of a shape before
    a graph capture).
    """
    import torch

    if stream is None:
        stream = torch.cuda.current_stream(device)
    key = (stream.device.index, stream.cuda_stream)
    ws = _workspaces.get(key)
    if ws is None or ws.numel() < nbytes:
        if ws is not None:
            ws.record_stream(stream)  # its memory is reused only after the stream's queued work
        with torch.cuda.stream(stream):  # zero-filled in order with the calls that will use it
            ws = torch.zeros(max(nbytes, attn_workspace_bytes(0, 0, 1, 1, 1)), dtype=torch.uint8,
                             device=stream.device)
        _workspaces[key] = ws
    return ws


def paged_prefill_attn(q, k_pool, v_pool, block_tables, cu_q, seq_lens, max_q_len: int, scale: float,
                       out, workspace=None, stream=None):
    """Causal GQA attention of packed queries [total, Hq, D] over the paged pools.

    `workspace` defaults to the buffer attn_workspace() keeps for the stream
    the call is issued on, grown to attn_workspace_bytes() for this shape
    (decode-shaped batches with few (request, kv head) pairs use the room to
    split each pair's keys over several waves).
    """
    import torch

    NB, Hkv, bs, D = k_pool.shape
    total, Hq, Dq = q.shape
    B = cu_q.shape[0] - 1
    if Dq != D or v_pool.shape != (NB, Hkv, D, bs) or out.shape != q.shape:
        raise ILPCError(EINVAL, "paged_prefill_attn: inconsistent Q/K/V/out shapes")
    if block_tables.dim() != 2 or block_tables.shape[0] != B or seq_lens.shape[0] != B:
        raise ILPCError(EINVAL, "paged_prefill_attn: inconsistent batch shapes")
    if workspace is None:
        shape = (B, int(max_q_len), Hq, Hkv, D)
        need = _ws_bytes.get(shape)
        if need is None:
            need = _ws_bytes[shape] = attn_workspace_bytes(*shape)
        workspace = attn_workspace(q.device, stream, need)
    ws_ptr, ws_bytes = _dev(workspace, torch.uint8, "workspace", 1), workspace.numel()
    args = (_dev(q, torch.bfloat16, "q", 3), _dev(k_pool, torch.bfloat16, "k_pool", 4),
            _dev(v_pool, torch.bfloat16, "v_pool", 4), NB,
            _dev(block_tables, torch.int32, "block_tables", 2), block_tables.shape[1],
            _dev(cu_q, torch.int32, "cu_q", 1), _dev(seq_lens, torch.int32, "seq_lens", 1), B,
            int(max_q_len), Hq, Hkv, D, bs, float(scale), _dev(out, torch.bfloat16, "out", 3),
            ws_ptr, ws_bytes, _stream(stream))
    _check(load().ilpc_paged_prefill_attn(*args))


def paged_prefill_attn_noalloc(q, k_pool, v_pool, block_tables, cu_q, seq_lens, max_q_len: int, scale: float,
                               out, stream=None):
    """paged_prefill_attn with the library's static device scratch as its
    workspace: the call allocates nothing.  Calls that may overlap on one GPU
    must not be issued (they share that scratch)."""
    import torch

    NB, Hkv, bs, D = k_pool.shape
    total, Hq, Dq = q.shape
    B = cu_q.shape[0] - 1
    if Dq != D or v_pool.shape != (NB, Hkv, D, bs) or out.shape != q.shape:
        raise ILPCError(EINVAL, "paged_prefill_attn_noalloc: inconsistent Q/K/V/out shapes")
    if block_tables.dim() != 2 or block_tables.shape[0] != B or seq_lens.shape[0] != B:
        raise ILPCError(EINVAL, "paged_prefill_attn_noalloc: inconsistent batch shapes")
    args = (_dev(q, torch.bfloat16, "q", 3), _dev(k_pool, torch.bfloat16, "k_pool", 4),
            _dev(v_pool, torch.bfloat16, "v_pool", 4), NB,
            _dev(block_tables, torch.int32, "block_tables", 2), block_tables.shape[1],
            _dev(cu_q, torch.int32, "cu_q", 1), _dev(seq_lens, torch.int32, "seq_lens", 1), B,
            int(max_q_len), Hq, Hkv, D, bs, float(scale), _dev(out, torch.bfloat16, "out", 3), _stream(stream))
    _check(load().ilpc_paged_prefill_attn_noalloc(*args))


NOALLOC_SCRATCH_BYTES = 256 + (8 << 20)


def decode_split(B, Hkv, max_blocks) -> int:
    """Key ranges per (request, kv head) the decode kernel uses by default."""
    n = _i32()
    _check(load().ilpc_decode_split(B, Hkv, max_blocks, ctypes.byref(n)))
    return int(n.value)


def decode_workspace_bytes(B, max_q_len, Hq, Hkv, D, n_split) -> int:
    n = ctypes.c_size_t()
    _check(load().ilpc_decode_workspace_bytes(B, max_q_len, Hq, Hkv, D, n_split, ctypes.byref(n)))
    return int(n.value)


def paged_decode_attn(q, k_pool, v_pool, block_tables, cu_q, seq_lens, max_q_len: int, scale: float, out,
                      stream=None, n_split: int = 1, workspace=None):
    """The decode kernel alone (max_q_len * Hq / Hkv <= 32): same semantics as
    paged_prefill_attn, which picks it by itself (unsplit) for such batches
    when they have at least one (request, kv head) pair per compute unit.

    n_split > 1 cuts every pair's keys into that many ranges (0: the
    library's choice, decode_split()); `workspace` is then a uint8 device
    tensor of at least decode_workspace_bytes() bytes, allocated here when
    omitted (an allocation: pass one in under graph capture).
    """
    import torch

    NB, Hkv, bs, D = k_pool.shape
    total, Hq, Dq = q.shape
    B = cu_q.shape[0] - 1
    if Dq != D or v_pool.shape != (NB, Hkv, D, bs) or out.shape != q.shape:
        raise ILPCError(EINVAL, "paged_decode_attn: inconsistent Q/K/V/out shapes")
    if block_tables.dim() != 2 or block_tables.shape[0] != B or seq_lens.shape[0] != B:
        raise ILPCError(EINVAL, "paged_decode_attn: inconsistent batch shapes")
    args = (_dev(q, torch.bfloat16, "q", 3), _dev(k_pool, torch.bfloat16, "k_pool", 4),
            _dev(v_pool, torch.bfloat16, "v_pool", 4), NB,
            _dev(block_tables, torch.int32, "block_tables", 2), block_tables.shape[1],
            _dev(cu_q, torch.int32, "cu_q", 1), _dev(seq_lens, torch.int32, "seq_lens", 1), B,
            int(max_q_len), Hq, Hkv, D, bs, float(scale), _dev(out, torch.bfloat16, "out", 3))
    if n_split == 0:
        n_split = decode_split(B, Hkv, block_tables.shape[1])
    need = decode_workspace_bytes(B, int(max_q_len), Hq, Hkv, D, n_split) if n_split >= 1 else 0
    if workspace is None and need:
        workspace = torch.empty(need, dtype=torch.uint8, device=q.device)
    ws_ptr, ws_bytes = (None, 0) if workspace is None else (_dev(workspace, torch.uint8, "workspace", 1),
                                                           workspace.numel())
    _check(load().ilpc_paged_decode_attn(*args, int(n_split), ws_ptr, ws_bytes, _stream(stream)))


def attn_cascade_workspace_bytes(B, max_q_len, Hq, Hkv, D) -> int:
    n = ctypes.c_size_t()
    _check(load().ilpc_attn_cascade_workspace_bytes(B, max_q_len, Hq, Hkv, D, ctypes.byref(n)))
    return int(n.value)


def paged_prefill_attn_cascade(q, k_pool, v_pool, block_tables, cu_q, seq_lens, max_q_len: int,
                               shared_len: int, scale: float, out, workspace, stream=None):
    """Attention split at a shared prefix of `shared_len` keys (see the C header).

    `workspace` is a uint8 device tensor of attn_cascade_workspace_bytes()
    bytes whose first 128 bytes are zero before the first call.
    """
    import torch

    NB, Hkv, bs, D = k_pool.shape
    total, Hq, Dq = q.shape
    B = cu_q.shape[0] - 1
    if Dq != D or v_pool.shape != (NB, Hkv, D, bs) or out.shape != q.shape:
        raise ILPCError(EINVAL, "paged_prefill_attn_cascade: inconsistent Q/K/V/out shapes")
    if block_tables.dim() != 2 or block_tables.shape[0] != B or seq_lens.shape[0] != B:
        raise ILPCError(EINVAL, "paged_prefill_attn_cascade: inconsistent batch shapes")
    args = (_dev(q, torch.bfloat16, "q", 3), _dev(k_pool, torch.bfloat16, "k_pool", 4),
            _dev(v_pool, torch.bfloat16, "v_pool", 4), NB,
            _dev(block_tables, torch.int32, "block_tables", 2), block_tables.shape[1],
            _dev(cu_q, torch.int32, "cu_q", 1), _dev(seq_lens, torch.int32, "seq_lens", 1), B,
            int(max_q_len), Hq, Hkv, D, bs, int(shared_len), float(scale),
            _dev(out, torch.bfloat16, "out", 3), _dev(workspace, torch.uint8, "workspace", 1),
            workspace.numel(), _stream(stream))
    _check(load().ilpc_paged_prefill_attn_cascade(*args))
