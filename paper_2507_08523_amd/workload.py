"""Seeded synthetic log-parsing prompt batches and their Q/K/V inputs.

A log-parsing prompt is a common instruction, k in-context demonstrations and
the queried log (InferLog, section 2.1.1, prompt format).  The paper measures
on Loghub-2k; these seeded token streams stand in for it with the shapes of
each named workload (token ids uniform in [0, 32000)).

This module holds none of the method's arithmetic -- no block keys, no cache
matching, no attention.  It only builds inputs:

* token streams of the measured batch, plus the warm batch that is registered
  into the cache before it;
* content-addressed K/V: every distinct full-block *token prefix* owns one
  [16, Hkv, D] K and V slab (a model's K/V of a token depends only on the
  tokens up to it, so requests sharing a prefix share those values exactly);
  the tail of each prompt (partial last block and decode tokens) gets slabs of
  its own;
* Q for every position of every prompt, so a query row does not depend on how
  much of its prompt happened to be cached.

Prefix identity is decided by exact token equality (a dictionary keyed by the
parent prefix and the block's tokens).
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

VOCAB = 32000
BLOCK = 16


@dataclass(frozen=True)
class WorkloadSpec:
    """Shape and structure of one synthetic batch (one attention layer)."""

    name: str
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    n_prompts: int
    instr_len: int
    n_demos: int
    demo_len: int
    pool_size: int
    query_len: tuple  # (lo, hi), inclusive, drawn uniformly per prompt
    q_std: float = 1.0
    kv_std: float = 1.0
    decode_steps: int = 0
    warm: str = "shared"          # "shared" | "none" | "own_prefix"
    own_prefix_len: int = 0       # for warm == "own_prefix"
    shared_demos: int | None = None  # leading demos common to all prompts; rest private
    # ICL stream (n_templates > 0): template-labelled candidate demonstrations,
    # a stream of `history` requests served before the measured batch
    n_templates: int = 0
    logs_per_template: int = 0
    history: int = 0
    seed: int = 0

    @property
    def group(self) -> int:
        return self.n_q_heads // self.n_kv_heads

    @property
    def scale(self) -> float:
        return 1.0 / float(np.sqrt(self.head_dim))


def _sweep(pct: int, m: int | None, warm: str) -> WorkloadSpec:
    return WorkloadSpec(name=f"sweep{pct}", n_q_heads=32, n_kv_heads=8, head_dim=128,
                        n_prompts=128, instr_len=256, n_demos=12, demo_len=60, pool_size=12,
                        query_len=(48, 48), shared_demos=(m if m is not None else 0), warm=warm,
                        seed=300 + pct)


SPECS: dict[str, WorkloadSpec] = {
    # 4 prompts sharing one 64-token cached prefix, each with a 32-token suffix
    "tiny": WorkloadSpec(name="tiny", n_q_heads=4, n_kv_heads=1, head_dim=64, n_prompts=4,
                         instr_len=64, n_demos=0, demo_len=0, pool_size=0, query_len=(32, 32),
                         seed=100),
    # Llama-3-8B-shaped layer: 256 instr + 5 of 32 demos x 60 tokens + 48-token query
    "llama8b": WorkloadSpec(name="llama8b", n_q_heads=32, n_kv_heads=8, head_dim=128, n_prompts=64,
                            instr_len=256, n_demos=5, demo_len=60, pool_size=32, query_len=(48, 48),
                            seed=200),
    # Qwen2.5-7B-shaped layer: 512 instr + 8 of 64 demos x 80 tokens + 20..120-token query
    "qwen7b": WorkloadSpec(name="qwen7b", n_q_heads=28, n_kv_heads=4, head_dim=128, n_prompts=256,
                           instr_len=512, n_demos=8, demo_len=80, pool_size=64, query_len=(20, 120),
                           q_std=1.0 / float(np.sqrt(128.0)), seed=210),
    # hit-rate sweep on Llama shapes: 128 prompts of 1024 tokens, m leading demos shared
    "sweep0": _sweep(0, 0, "none"),
    "sweep25": _sweep(25, 0, "shared"),
    "sweep50": _sweep(50, 4, "shared"),
    "sweep75": _sweep(75, 8, "shared"),
    "sweep100": _sweep(100, 12, "shared"),
    # the same fully shared batch generating 32 output tokens per prompt (the
    # short template each log query is parsed into)
    "sweep100_decode": WorkloadSpec(**{**_sweep(100, 12, "shared").__dict__, "name": "sweep100_decode",
                                       "decode_steps": 32}),
    # large context: 16 of 128 demos x 128 tokens + 64-token query, then 32 decode steps
    "large": WorkloadSpec(name="large", n_q_heads=64, n_kv_heads=8, head_dim=128, n_prompts=512,
                          instr_len=0, n_demos=16, demo_len=128, pool_size=128, query_len=(64, 64),
                          decode_steps=32, seed=400),
    "large_prefixwarm": WorkloadSpec(name="large_prefixwarm", n_q_heads=64, n_kv_heads=8,
                                     head_dim=128, n_prompts=512, instr_len=0, n_demos=16,
                                     demo_len=128, pool_size=128, query_len=(64, 64),
                                     warm="own_prefix", own_prefix_len=2048, seed=400),
}


# Log-parsing request stream with template-labelled demonstrations, on the
# Llama-3-8B-shaped layer: 200 candidate logs (40 templates x 5 logs), 5
# demonstrations per request, 2000 requests (the size of one Loghub-2k dataset),
# the last 64 of which form the measured batch.
_ICL = dict(n_q_heads=32, n_kv_heads=8, head_dim=128, n_prompts=64, instr_len=256, n_demos=5,
            demo_len=60, pool_size=200, query_len=(48, 48), warm="history", n_templates=40,
            logs_per_template=5, history=1936, seed=500)
SPECS["icl_llama8b"] = WorkloadSpec(name="icl_llama8b", **_ICL)

# Weights of the template draw of an ICL stream, hottest first; every other
# template weighs TAIL_WEIGHT.  Drawing 5 distinct templates of 40 by successive
# weighted sampling without replacement, these put the five hottest templates
# into 36.2%, 27.2%, 24.7%, 21.2% and 17.1% of requests, the hotspot
# selection frequencies InferLog reports (section 2.2.2, hotspot demonstrations).
HOT_WEIGHTS = (1.0, 0.7075, 0.6350, 0.5327, 0.4240)
TAIL_WEIGHT = 0.2563


@dataclass
class IclStream:
    """The demonstration sets a kNN selector would pick for a request stream.

    templates, demos: int32 [R, n_demos] in selection order (the order the
    selector emits, least similar first); demonstration d is candidate log d,
    of template d // logs_per_template, with tokens demo_tokens[d].
    """

    spec: WorkloadSpec
    instr: np.ndarray
    demo_tokens: np.ndarray
    templates: np.ndarray
    demos: np.ndarray
    queries: list

    def prompts(self, templates=None, demos=None):
        """Instruction + demonstrations (in the given order) + query, per request."""
        d = self.demos if demos is None else np.asarray(demos)
        return [np.concatenate([self.instr, *self.demo_tokens[d[r]], self.queries[r]]).astype(np.int32)
                for r in range(len(self.queries))]


def icl_stream(spec: WorkloadSpec | str) -> IclStream:
    """Seeded stand-in for kNN demonstration selection over a request stream.

    Per request: n_demos distinct templates drawn by weighted sampling without
    replacement (hot templates per HOT_WEIGHTS), one candidate log of each drawn
    uniformly, the set in a fresh random order (similarity to each query log
    differs), then a query log of uniform random tokens.
    """
    if isinstance(spec, str):
        spec = SPECS[spec]
    T, m, k = spec.n_templates, spec.logs_per_template, spec.n_demos
    if T < k or m < 1 or spec.pool_size != T * m:
        raise ValueError("ICL stream needs n_templates >= n_demos and pool_size = n_templates * logs")
    rng = np.random.default_rng(spec.seed)
    instr = rng.integers(0, VOCAB, spec.instr_len, dtype=np.int64).astype(np.int32)
    demo_tokens = rng.integers(0, VOCAB, (T * m, spec.demo_len), dtype=np.int64).astype(np.int32)
    w = np.full(T, TAIL_WEIGHT)
    w[:min(T, len(HOT_WEIGHTS))] = HOT_WEIGHTS[:T]
    R = spec.history + spec.n_prompts
    # successive sampling without replacement == top-k of log-weight + Gumbel noise
    key = np.log(w)[None, :] + rng.gumbel(size=(R, T))
    chosen = np.argsort(-key, axis=1, kind="stable")[:, :k]
    order = np.argsort(rng.random((R, k)), axis=1)
    templates = np.take_along_axis(chosen, order, axis=1).astype(np.int32)
    demos = (templates * m + rng.integers(0, m, (R, k))).astype(np.int32)
    lo, hi = spec.query_len
    queries = [rng.integers(0, VOCAB, int(rng.integers(lo, hi + 1)), dtype=np.int64).astype(np.int32)
               for _ in range(R)]
    return IclStream(spec=spec, instr=instr, demo_tokens=demo_tokens, templates=templates, demos=demos,
                     queries=queries)


def cache_op_stream(seed: int, n_steps: int = 60, n_pieces: int = 5):
    """Seeded operations on a prefix cache with a block lifecycle.

    ("match", prompts): 1-3 prompts, each 1-3 shared pieces of 8-49 tokens in a
    random order plus a private tail of 1-19 tokens; ("release", u): finish a
    fraction u of the requests still held; ("touch", ids): 4 block ids in
    [-1, 40).
    """
    rng = np.random.default_rng(seed)
    pieces = [rng.integers(0, VOCAB, int(rng.integers(8, 50))).astype(np.int32) for _ in range(n_pieces)]
    ops = []
    for _ in range(n_steps):
        u = rng.random()
        if u < 0.55:
            prompts = []
            for _ in range(int(rng.integers(1, 4))):
                order = rng.permutation(n_pieces)[:int(rng.integers(1, 4))]
                tail = rng.integers(0, VOCAB, int(rng.integers(1, 20))).astype(np.int32)
                prompts.append(np.concatenate([pieces[i] for i in order] + [tail]))
            ops.append(("match", prompts))
        elif u < 0.9:
            ops.append(("release", float(rng.random())))
        else:
            ops.append(("touch", [int(x) for x in rng.integers(-1, 40, 4)]))
    return ops


def scaled_spec(name: str, n_prompts: int, **over) -> WorkloadSpec:
    """A named workload with fewer prompts (same per-prompt structure)."""
    base = SPECS[name]
    d = dict(base.__dict__)
    d.update(over)
    d["n_prompts"] = n_prompts
    d["name"] = f"{base.name}[{n_prompts}]"
    return WorkloadSpec(**d)


@dataclass
class Workload:
    """Token streams and content-addressed slab maps of one seeded batch."""

    spec: WorkloadSpec
    prompts: list            # measured batch: list of int32 arrays
    warm: list               # batch registered before the measured one
    warm_src: list           # prompt each warm sequence is a prefix of
    slab_ids: list           # per prompt: int64 array, slab of each logical block
    n_slabs: int
    q_offsets: np.ndarray    # per prompt: first row of its positions in the Q table
    tensors: dict = field(default_factory=dict)

    @property
    def seq_lens(self) -> np.ndarray:
        return np.array([len(p) for p in self.prompts], dtype=np.int32)

    # -- tensors -----------------------------------------------------------
    def materialize(self, device="cpu"):
        """Draw K/V slabs and the Q table (bf16) on ``device`` from the seed."""
        import torch

        sp = self.spec
        dev = torch.device(device)
        out = {}
        for i, nm in enumerate(("k", "v")):
            g = torch.Generator(device=dev)
            g.manual_seed(sp.seed * 1000 + 1 + i)
            out[nm] = _randn_bf16((self.n_slabs * BLOCK, sp.n_kv_heads, sp.head_dim),
                                  sp.kv_std, g, dev)
        g = torch.Generator(device=dev)
        g.manual_seed(sp.seed * 1000 + 7)
        n_q = int(self.q_offsets[-1])
        out["q"] = _randn_bf16((n_q, sp.n_q_heads, sp.head_dim), sp.q_std, g, dev)
        self.tensors = out
        return out

    def kv_rows(self, r: int, positions: np.ndarray) -> np.ndarray:
        """Slab-table row of request r's K/V at absolute ``positions``."""
        positions = np.asarray(positions, dtype=np.int64)
        return self.slab_ids[r][positions // BLOCK] * BLOCK + positions % BLOCK

    def dense_kv(self, r: int, length: int):
        """Request r's K and V for positions 0..length-1, [length, Hkv, D]."""
        import torch

        idx = torch.from_numpy(self.kv_rows(r, np.arange(length)))
        idx = idx.to(self.tensors["k"].device)
        return self.tensors["k"][idx], self.tensors["v"][idx]

    def q_rows(self, r: int, start: int, stop: int):
        """Request r's Q for positions start..stop-1, [stop-start, Hq, D]."""
        o = int(self.q_offsets[r])
        return self.tensors["q"][o + start:o + stop]

    def packed_rows(self, items, with_q=True):
        """Rows of positions start..stop-1 of prompt r for each (r, start, stop).

        Returns a dict with q [sum n, Hq, D] (if ``with_q``), k_new, v_new
        [sum n, Hkv, D], cu int32 [n_items+1] and max_len.
        """
        import torch

        n = np.array([stop - start for (_, start, stop) in items], dtype=np.int64)
        cu = np.zeros(len(items) + 1, dtype=np.int32)
        cu[1:] = np.cumsum(n)
        kv_idx = [self.kv_rows(r, np.arange(a, b)) for (r, a, b) in items]
        kv_idx = np.concatenate(kv_idx) if kv_idx else np.zeros(0, np.int64)
        dev = self.tensors["k"].device
        kv_i = torch.from_numpy(kv_idx.astype(np.int64)).to(dev)
        out = {"k_new": self.tensors["k"][kv_i].contiguous(),
               "v_new": self.tensors["v"][kv_i].contiguous(),
               "cu": cu, "max_len": int(n.max()) if len(n) else 0}
        if with_q:
            q_idx = [self.q_offsets[r] + np.arange(a, b) for (r, a, b) in items]
            q_idx = np.concatenate(q_idx) if q_idx else np.zeros(0, np.int64)
            q_i = torch.from_numpy(q_idx.astype(np.int64)).to(dev)
            out["q"] = self.tensors["q"][q_i].contiguous()
        return out

    def packed_suffix(self, cached_len):
        """Q / K_new / V_new of every request's positions cached_len[r]..L_r-1."""
        L = self.seq_lens
        P = np.asarray(cached_len, dtype=np.int64)
        return self.packed_rows([(r, int(P[r]), int(L[r])) for r in range(len(L))])

    def packed_warm(self, cached_len):
        """K_new / V_new of the warm batch's uncached positions."""
        P = np.asarray(cached_len, dtype=np.int64)
        return self.packed_rows([(self.warm_src[w], int(P[w]), len(self.warm[w]))
                                 for w in range(len(self.warm))], with_q=False)

    def decode_inputs(self, step: int):
        """Q row and new K/V row of every request at position L_r + step."""
        import torch

        sp = self.spec
        assert 0 <= step < sp.decode_steps
        L = self.seq_lens.astype(np.int64)
        kv_idx = np.array([self.kv_rows(r, np.array([L[r] + step]))[0] for r in range(len(L))],
                          dtype=np.int64)
        q_idx = self.q_offsets[:-1] + L + step
        dev = self.tensors["k"].device
        kv_i = torch.from_numpy(kv_idx).to(dev)
        q_i = torch.from_numpy(q_idx.astype(np.int64)).to(dev)
        return {"q": self.tensors["q"][q_i].contiguous(),
                "k_new": self.tensors["k"][kv_i].contiguous(),
                "v_new": self.tensors["v"][kv_i].contiguous()}


def _randn_bf16(shape, std, gen, dev):
    import torch

    out = torch.empty(shape, dtype=torch.bfloat16, device=dev)
    flat = out.view(-1)
    n = flat.numel()
    chunk = 1 << 28
    for s in range(0, n, chunk):
        e = min(n, s + chunk)
        x = torch.randn(e - s, generator=gen, device=dev, dtype=torch.float32)
        if std != 1.0:
            x.mul_(std)
        flat[s:e] = x.to(torch.bfloat16)
    return out


def build(spec: WorkloadSpec | str, demos=None) -> Workload:
    """Token streams, warm batch and slab maps for ``spec`` (no tensors yet).

    For an ICL stream, ``demos`` (int32 [history + n_prompts, n_demos]) are the
    demonstration ids each request finally carries, in order; by default the
    selector's own sets and order.
    """
    if isinstance(spec, str):
        spec = SPECS[spec]
    if spec.n_templates:
        st = icl_stream(spec)
        everything = st.prompts(demos=demos)
        return _from_prompts(spec, everything[spec.history:], everything[:spec.history])
    rng = np.random.default_rng(spec.seed)
    instr = rng.integers(0, VOCAB, spec.instr_len, dtype=np.int64).astype(np.int32)
    pool = rng.integers(0, VOCAB, (spec.pool_size, spec.demo_len), dtype=np.int64).astype(np.int32)
    distinct_first = rng.permutation(VOCAB)[: spec.n_prompts].astype(np.int32)
    prompts = []
    for r in range(spec.n_prompts):
        parts = [instr]
        if spec.shared_demos is None:
            order = rng.permutation(spec.pool_size)[: spec.n_demos]
            parts += [pool[i] for i in order]
        else:
            m = spec.shared_demos
            parts += [pool[i] for i in range(m)]
            private = rng.integers(0, VOCAB, ((spec.n_demos - m) * spec.demo_len,), dtype=np.int64)
            private = private.astype(np.int32)
            if private.size:
                private[0] = distinct_first[r]  # sharing stops exactly at the first private demo
            parts.append(private)
        lo, hi = spec.query_len
        q_len = int(rng.integers(lo, hi + 1))
        parts.append(rng.integers(0, VOCAB, q_len, dtype=np.int64).astype(np.int32))
        prompts.append(np.concatenate(parts).astype(np.int32))
    return _from_prompts(spec, prompts, None)


def _from_prompts(spec: WorkloadSpec, prompts: list, history) -> Workload:
    """Content addressing and warm batch of a measured batch ``prompts``.

    ``history`` (warm mode "history"): earlier requests whose full blocks are
    all in the cache when the measured batch arrives; the warm batch is then,
    per measured prompt, its longest run of leading full blocks that some
    earlier request holds token for token.
    """
    # content addressing: one node per distinct full-block token prefix
    node_of: dict = {}
    full_nodes = []
    for p in prompts:
        parent = -1
        nodes = []
        for b in range(len(p) // BLOCK):
            key = (parent, p[b * BLOCK:(b + 1) * BLOCK].tobytes())
            nid = node_of.get(key)
            if nid is None:
                nid = len(node_of)
                node_of[key] = nid
            nodes.append(nid)
            parent = nid
        full_nodes.append(nodes)
    n_slabs = len(node_of)
    slab_ids = []
    for r, p in enumerate(prompts):
        n_total = -(-(len(p) + spec.decode_steps) // BLOCK)
        n_tail = n_total - len(full_nodes[r])
        tail = list(range(n_slabs, n_slabs + n_tail))
        n_slabs += n_tail
        slab_ids.append(np.array(full_nodes[r] + tail, dtype=np.int64))

    # warm batch
    warm, warm_src = [], []
    if spec.warm == "shared":
        count: dict = {}
        for nodes in full_nodes:
            for nid in set(nodes):
                count[nid] = count.get(nid, 0) + 1
        seen = set()
        for r, nodes in enumerate(full_nodes):
            s = 0
            while s < len(nodes) and count[nodes[s]] >= 2:
                s += 1
            if s and nodes[s - 1] not in seen:
                seen.add(nodes[s - 1])
                warm.append(prompts[r][: s * BLOCK].copy())
                warm_src.append(r)
    elif spec.warm == "history":
        held: dict = {}   # (parent node, block tokens) -> node, over the history
        for p in history:
            parent = -1
            for b in range(len(p) // BLOCK):
                parent = held.setdefault((parent, p[b * BLOCK:(b + 1) * BLOCK].tobytes()), len(held))
        seen = set()
        for r, p in enumerate(prompts):
            s, parent = 0, -1
            while s < len(p) // BLOCK:
                parent = held.get((parent, p[s * BLOCK:(s + 1) * BLOCK].tobytes()))
                if parent is None:
                    break
                s += 1
            if s and full_nodes[r][s - 1] not in seen:
                seen.add(full_nodes[r][s - 1])
                warm.append(p[: s * BLOCK].copy())
                warm_src.append(r)
    elif spec.warm == "own_prefix":
        warm = [p[: spec.own_prefix_len].copy() for p in prompts]
        warm_src = list(range(len(prompts)))
    elif spec.warm != "none":
        raise ValueError(f"unknown warm mode {spec.warm}")

    lens = np.array([len(p) + spec.decode_steps for p in prompts], dtype=np.int64)
    q_offsets = np.zeros(len(prompts) + 1, dtype=np.int64)
    q_offsets[1:] = np.cumsum(lens)
    return Workload(spec=spec, prompts=prompts, warm=warm, warm_src=warm_src, slab_ids=slab_ids,
                    n_slabs=n_slabs, q_offsets=q_offsets)
