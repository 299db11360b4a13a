"""Benchmark of the prefix-cached prefill hot path on one MI355X.

One step = one pass of the whole path over one batch of synthetic
log-parsing prompts (inputs already resident in HBM):

    prefix match (host C++)  ->  one pinned H2D copy of the batch metadata
    ->  kv_append (HIP)  ->  paged prefill attention (HIP)
    [-> decode steps, for workloads that have them: kv_append of one token per
        prompt + attention with one query per prompt, 32 times]

Every step starts from the same cache state: the step takes a checkpoint
before matching and rolls the cache back after its metadata is staged (the
rollback is extra host work inside the step, nothing is skipped).

Prints ONE JSON line.  ``value`` is new-query tokens per second over the timed
steps (prefill suffix tokens + decode tokens).  ``roofline`` is for the
dominant kernel, the prefill attention launch, timed with HIP events on the
stream it runs on.  ``cpu_baseline`` times the fp64 oracle on a bounded
sample of the same workload on the host cores.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload large] [--prompts N] [--cascade | --single] [--no-pair]

The default workload is ``large``: 512 prompts of 2112 tokens (16 demonstrations
of 128 tokens + a 64-token query; 64 q / 8 kv heads, head_dim 128), whose
prefill is followed by 32 decode steps -- the largest configuration that fits
one GPU.  The roofline of the prefill launch is
t_roof = max(FLOPs / 2.5 PFLOP/s, unique bytes / 8 TB/s), unique bytes
counting each physical K/V block once; logical bytes (K/V once per request)
are reported beside them.  ``--flush-mib N`` writes N MiB of device memory
before every step, so HBM-bound launches do not find the previous step's data
in the caches.

The attention runs split at the prefix every prompt of the batch shares
(ilpc_paged_prefill_attn_cascade) where the library's rule
(ilpc_prefer_shared_split) expects that to be faster than the single pass --
long shared prefixes with a short own part per prompt, as in ``sweep100`` --
and as the single pass elsewhere; ``config.attention`` says which ran.
``--cascade`` forces the split, ``--single`` the single pass.

``--rope BASE`` rotates the new tokens' K and Q at their positions inside the
append (ilpc_rope_kv_append; the warm prefix is rotated the same way).
``--chunk-tokens N`` runs the prefill as scheduler steps of at most N new
tokens (append + attention per step); the attention timing and ``roofline``
then cover all steps.  ``--graph`` (decode workloads) captures the 32 decode
steps once as a HIP graph with all their metadata on the device, and every
timed step replays it; with ``--chunk-tokens`` it also captures the
scheduler steps of the chunked prefill as one graph.  ``--prompts N`` keeps the workload's shapes with N
prompts (``large --prompts 16``: decode steps of a small batch, whose
attention splits each request's keys over several waves).

ICL stream workloads (``icl_llama8b``): 2000 log-parsing requests whose
demonstrations a selector picks with hot templates.  Before the timed steps the
whole stream passes the ICL table (prefix-aware refinement, host C++) in
arrival order, 64 requests per call; the earlier requests' blocks fill the
cache and the last 64 requests are the measured batch.  ``config`` adds the
stream's prefix-cache hit rate with and without refinement.  ``--no-pair``
measures the batch in the selector's order.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import subprocess
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "prefix-cached prefill attn: query tokens/s, TFLOP/s & GB/s vs MI355X roofline"
PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 matrix peak
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E peak
KERNEL_SRC = os.path.join(ROOT, "paper_2507_08523_amd", "csrc", "paged_attn.hip")


def workload_work(wl, cached_len, tables):
    """Algorithmic FLOPs and bytes of one prefill attention launch.

    FLOPs count the visible (query, key) pairs only: 4 * Hq * D per pair (the
    QK^T and PV products).  Logical bytes read every request's K/V context
    once per request (shared prefix blocks once per request that holds them)
    plus Q in and O out.  Unique bytes count each physical K/V block once, at
    the largest number of its 16 slots any request reads, plus Q and O.
    """
    sp = wl.spec
    L = wl.seq_lens.astype(np.float64)
    P = np.asarray(cached_len, dtype=np.float64)
    S = L - P
    pairs = float(np.sum(S * P + S * (S + 1) / 2))   # visible (query, key) pairs
    flops = 4.0 * sp.n_q_heads * sp.head_dim * pairs
    per_token = 4.0 * sp.n_kv_heads * sp.head_dim           # K + V of one token, bf16
    kv_bytes = float(np.sum(per_token * L))
    qo_bytes = float(np.sum(4.0 * sp.n_q_heads * sp.head_dim * S))     # Q in + O out, bf16
    Li = wl.seq_lens.astype(np.int64)
    nb = (Li + 15) // 16
    ids = np.concatenate([tables[r, :nb[r]] for r in range(len(Li))]).astype(np.int64)
    fill = np.concatenate([np.minimum(16, Li[r] - 16 * np.arange(nb[r])) for r in range(len(Li))])
    slots = np.zeros(int(ids.max()) + 1 if ids.size else 0, np.int64)
    np.maximum.at(slots, ids, fill)
    unique_kv = float(slots.sum()) * per_token
    return {"pairs": pairs, "flops": flops, "logical_bytes": kv_bytes + qo_bytes,
            "unique_bytes": unique_kv + qo_bytes, "query_tokens": int(S.sum())}


def kernel_source_sha() -> str:
    """Hash of the attention kernel's code: `//` comments, trailing blanks and
    empty lines are left out, so a comment edit does not orphan the counter
    summaries taken on the same code (the source has no block comments and
    no `//` inside string literals)."""
    lines = []
    with open(KERNEL_SRC, encoding="utf-8") as f:
        for line in f:
            code = line.split("//", 1)[0].rstrip()
            if code:
                lines.append(code)
    return hashlib.sha256("\n".join(lines).encode()).hexdigest()[:16]


def traffic_from_profile(workload_name: str):
    """Measured HBM bytes per launch from the committed counter summary, or
    None when there is none or the kernel source changed since it was taken."""
    path = os.path.join(ROOT, "profiles", f"paged_attn_{workload_name}_traffic.txt")
    if not os.path.exists(path):
        return None
    fields = {}
    with open(path) as f:
        for line in f:
            if line.startswith("#") or ":" not in line:
                continue
            k, v = line.split(":", 1)
            fields[k.strip()] = v.strip()
    if fields.get("kernel_source_sha") != kernel_source_sha():
        return None
    return float(fields["hbm_bytes_per_launch"]) if "hbm_bytes_per_launch" in fields else None


def traffic_key(args, split: bool) -> str:
    """Name of the counter summary that matches this run's attention launches:
    the workload's own for the single pass (RoPE and graph replay change
    neither the prefill launch nor its inputs), ``<workload>_cascade`` for the
    shared-prefix split (``split``), ``<workload>_chunk<N>`` for chunked
    prefill and ``<workload>_nopair`` for an unrefined ICL stream."""
    key = args.workload
    if split:
        key += "_cascade"
    if args.chunk_tokens:
        key += f"_chunk{args.chunk_tokens}"
    if args.no_pair:
        key += "_nopair"
    return key


def host_cpu():
    """The host's processor as lscpu reports it, and the CPUs this process may use."""
    info = {"nproc": os.cpu_count(), "affinity_cpus": len(os.sched_getaffinity(0))}
    try:
        out = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=20).stdout
    except (OSError, subprocess.SubprocessError):
        return info
    keep = {"Model name": "model", "CPU(s)": "cpus", "Thread(s) per core": "threads_per_core",
            "Core(s) per socket": "cores_per_socket", "Socket(s)": "sockets"}
    for ln in out.splitlines():
        k, _, v = ln.partition(":")
        if k.strip() in keep:
            info[keep[k.strip()]] = v.strip()
    return info


def cpu_baseline(wl, cached_len, work, n_tokens, budget_s: float, decode_budget_s: float):
    """Time the fp64 oracle on the host cores and extrapolate it to the step.

    Prefix match of the whole batch (timed in full), prefill attention of
    requests in a seeded order until ``budget_s`` (passing over the batch again
    if it is done first), and, for workloads with decode steps, seeded
    (request, step) decode queries until ``decode_budget_s``.  The attention
    parts are scaled to the whole step by FLOP ratio (their cost is
    proportional to the visible pairs); the result is query tokens per second
    of the whole step, prefill and decode tokens, like ``value``.
    """
    from threadpoolctl import threadpool_info

    from oracle.attn_ref import decode_step_ref, prefill_attention_ref
    from oracle.prefix_ref import PrefixCacheRef

    sp = wl.spec
    ref = PrefixCacheRef(1 << 30, 1 << 30)
    if wl.warm:
        ref.match(wl.warm)
    dec = sp.decode_steps
    reserve = [dec] * len(wl.prompts) if dec else None
    t0 = time.perf_counter()
    c_ref, _, _ = ref.match(wl.prompts, reserve=reserve)
    t_match = time.perf_counter() - t0
    assert np.array_equal(c_ref, cached_len)
    per_pair = 4.0 * sp.n_q_heads * sp.head_dim
    rng = np.random.default_rng(0)
    order = rng.permutation(len(wl.prompts))
    t_attn, flops_done, tokens, done = 0.0, 0.0, 0, 0
    for i in range(len(order) * 1000):
        r = int(order[i % len(order)])
        L, P = int(wl.seq_lens[r]), int(cached_len[r])
        k, v = wl.dense_kv(r, L)
        q = wl.q_rows(r, P, L).float().cpu().numpy().astype(np.float64)
        k = k.float().cpu().numpy().astype(np.float64)
        v = v.float().cpu().numpy().astype(np.float64)
        t0 = time.perf_counter()
        prefill_attention_ref(q, k, v, sp.scale)
        t_attn += time.perf_counter() - t0
        S = L - P
        flops_done += per_pair * (S * P + S * (S + 1) / 2)
        tokens += S
        done += 1
        if t_attn >= budget_s:
            break
    t_prefill = t_attn * work["flops"] / flops_done
    sample = (f"fp64 oracle: prefix match of all {len(wl.prompts)} prompts ({t_match * 1e3:.1f} ms, timed in full); "
              f"prefill attention of {done} request passes in a seeded order ({tokens} query tokens, "
              f"{t_attn:.1f} s) scaled by FLOP ratio {work['flops'] / flops_done:.3g} to the batch "
              f"({t_prefill:.1f} s)")
    t_decode = 0.0
    if dec:
        L_all = wl.seq_lens.astype(np.int64)
        total = per_pair * float(np.sum(dec * (L_all + 1) + dec * (dec - 1) / 2))
        t_dec, f_dec, n_dec = 0.0, 0.0, 0
        picks = rng.permutation(len(wl.prompts))
        for r in picks:
            r = int(r)
            s = int(rng.integers(0, dec))
            n = int(L_all[r]) + s + 1
            k, v = wl.dense_kv(r, n)
            qd = wl.q_rows(r, n - 1, n)[0].float().cpu().numpy().astype(np.float64)
            k = k.float().cpu().numpy().astype(np.float64)
            v = v.float().cpu().numpy().astype(np.float64)
            t0 = time.perf_counter()
            decode_step_ref(qd, k, v, sp.scale)
            t_dec += time.perf_counter() - t0
            f_dec += per_pair * n
            n_dec += 1
            if t_dec >= decode_budget_s:
                break
        t_decode = t_dec * total / f_dec
        sample += (f"; {n_dec} decode queries at seeded (request, step) ({t_dec:.2f} s) scaled by FLOP ratio "
                   f"{total / f_dec:.3g} to {dec} steps x {len(wl.prompts)} prompts ({t_decode:.1f} s)")
    t_step = t_match + t_prefill + t_decode
    threads = max([i.get("num_threads", 1) for i in threadpool_info() if i.get("user_api") == "blas"] + [1])
    return {"value": round(n_tokens / t_step, 2), "unit": "query tokens/s", "cores": int(threads),
            "kind": "oracle", "extrapolated": bool(work["flops"] > flops_done or dec > 0),
            "est_step_s": round(t_step, 6), "sample": sample, "host": host_cpu()}


def icl_stream_workload(name: str, pair: bool):
    """The measured batch of an ICL request stream, demonstrations refined by
    the ICL table (or in the selector's order), and the stream's hit rates."""
    from paper_2507_08523_amd import workload
    from paper_2507_08523_amd.pipeline import ICL_TABLE_CAPACITY, pair_refine_stream, stream_hit_rate

    sp = workload.SPECS[name]
    st = workload.icl_stream(sp)
    R = len(st.templates)
    naive = stream_hit_rate(st.prompts(), sp.n_prompts)
    info = {"stream_requests": R, "pair": pair, "stream_hit_rate_naive": round(naive["hit_rate"], 4)}
    demos = None
    if pair:
        t0 = time.perf_counter()
        _, demos, pmc = pair_refine_stream(st, ICL_TABLE_CAPACITY, sp.n_prompts)
        dt = time.perf_counter() - t0
        refined = stream_hit_rate(st.prompts(demos=demos), sp.n_prompts)
        info.update({"icl_table_capacity": ICL_TABLE_CAPACITY,
                     "stream_hit_rate": round(refined["hit_rate"], 4),
                     "hit_rate_gain": round(refined["hit_rate"] / naive["hit_rate"], 3),
                     "mean_pmc": round(float(pmc.mean()), 3),
                     "pair_us_per_request": round(dt / R * 1e6, 3)})
    return info, workload.build(sp, demos=demos)


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="large")
    ap.add_argument("--prompts", type=int, default=0,
                    help="run the workload's shapes with this many prompts (0: its own count)")
    ap.add_argument("--cpu-budget", type=float, default=12.0, help="seconds of oracle prefill attention to time")
    ap.add_argument("--cpu-decode-budget", type=float, default=2.0,
                    help="seconds of oracle decode queries to time (workloads with decode steps)")
    ap.add_argument("--flush-mib", type=int, default=0,
                    help="before every step, write this many MiB of device memory (evicts the MALL "
                         "and L2 between steps; the write is inside the step time, outside the "
                         "kernel timings)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-pair", action="store_true",
                    help="ICL stream workloads: serve the selector's demonstration order unrefined")
    ap.add_argument("--chunk-tokens", type=int, default=0,
                    help="prefill in scheduler steps of at most this many new tokens (0: one pass)")
    ap.add_argument("--rope", type=float, default=0.0, metavar="BASE",
                    help="rotate new K and Q with RoPE of this base inside the append (0: off)")
    ap.add_argument("--graph", action="store_true",
                    help="replay the decode steps (decode workloads) and the chunked prefill steps "
                         "(--chunk-tokens) as captured HIP graphs")
    ap.add_argument("--cascade", action="store_true",
                    help="split the attention at the prefix every prompt shares, whatever the library's "
                         "rule says (by default the split runs where ilpc_prefer_shared_split picks it)")
    ap.add_argument("--single", action="store_true",
                    help="run the single pass even where the library's rule picks the shared-prefix split")
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="run one plain device copy of this many MiB first (counter calibration)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (got --gpus {args.gpus}); the path needs no collective "
              "and every box here has one GPU", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2507_08523_amd import ilpc, workload
    from paper_2507_08523_amd.pipeline import (ChunkGraph, DecodeGraph, PagedPrefixCache, chunk_schedule,
                                               max_blocks_of, pool_blocks_needed, prefer_shared_split, rope_inv_freq,
                                               shared_prefix_len)

    ilpc.load()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream(dev)

    if args.calib_copy_mib:
        n = args.calib_copy_mib << 20
        a = torch.empty(n, dtype=torch.uint8, device=dev)
        b = torch.empty_like(a)
        b.copy_(a)
        torch.cuda.synchronize()
        del a, b

    icl = None
    if workload.SPECS[args.workload].n_templates:
        if args.prompts:
            print("--prompts does not apply to ICL stream workloads", file=sys.stderr)
            sys.exit(2)
        icl, wl = icl_stream_workload(args.workload, not args.no_pair)
    elif args.prompts:
        wl = workload.build(workload.scaled_spec(args.workload, args.prompts))
    else:
        wl = workload.build(args.workload)
    wl.materialize(dev)
    sp = wl.spec
    pc = PagedPrefixCache(sp.n_kv_heads, sp.head_dim, pool_blocks_needed(wl), max_blocks_of(wl),
                          max(len(wl.prompts), len(wl.warm), 1), 20, dev)

    if args.cascade and (args.rope or args.chunk_tokens or args.single):
        print("--cascade does not combine with --rope, --chunk-tokens or --single", file=sys.stderr)
        sys.exit(2)
    if args.graph and (args.cascade or (args.rope and sp.decode_steps)):
        print("--graph does not combine with --cascade, nor with --rope on decode workloads", file=sys.stderr)
        sys.exit(2)
    inv_freq = torch.from_numpy(rope_inv_freq(sp.head_dim, args.rope)).to(dev) if args.rope else None

    # warm pass (untimed): registers the shared prefix blocks and their K/V
    if wl.warm:
        c, t = pc.match(wl.warm)
        rows = wl.packed_warm(c)
        b = pc.upload_prefill(c, t, [len(p) for p in wl.warm])
        if args.rope:
            pc.append_rope(b, rows["k_new"], rows["v_new"], inv_freq)
        else:
            pc.append(b, rows["k_new"], rows["v_new"])
        torch.cuda.synchronize()
        del rows

    tokens = np.concatenate(wl.prompts).astype(np.int32)
    cu_tok = np.zeros(len(wl.prompts) + 1, np.int32)
    cu_tok[1:] = np.cumsum(wl.seq_lens)
    dec = sp.decode_steps
    reserve = np.full(len(wl.prompts), dec, np.int32) if dec else None

    # rehearsal: learn the cached lengths, gather the suffix inputs (resident in HBM)
    mark = pc.cache.checkpoint()
    cached, tables = pc.match(packed=(tokens, cu_tok), reserve=reserve)
    pc.cache.rollback(mark)
    rows = wl.packed_suffix(cached)
    q, k_new, v_new = rows["q"], rows["k_new"], rows["v_new"]
    out = torch.empty_like(q)
    q_rot = torch.empty_like(q) if args.rope else None
    n_chunks = len(chunk_schedule(wl.seq_lens - cached, args.chunk_tokens)) if args.chunk_tokens else 1
    # the shared-prefix split: forced by --cascade, else where the library's
    # rule picks it (the single pass with --single, RoPE, chunked steps or graphs)
    shared_len = shared_prefix_len(cached, tables)
    auto = not (args.single or args.rope or args.chunk_tokens or args.graph)
    L = wl.seq_lens.astype(np.int32)
    heads = (sp.n_q_heads, sp.n_kv_heads)
    split_prefill = args.cascade or (auto and prefer_shared_split(L, int((L - cached).max()), *heads, shared_len))
    split_decode = bool(dec) and (args.cascade or (auto and prefer_shared_split(L + dec, 1, *heads, shared_len)))
    cascade_ws = decode_ws = None
    if split_prefill or split_decode:
        n_ws = ilpc.attn_cascade_workspace_bytes(len(wl.prompts), int((wl.seq_lens - cached).max()),
                                                 sp.n_q_heads, sp.n_kv_heads, sp.head_dim)
        cascade_ws = torch.zeros(n_ws, dtype=torch.uint8, device=dev)
        decode_ws = torch.zeros(ilpc.attn_cascade_workspace_bytes(len(wl.prompts), 1, sp.n_q_heads,
                                                                  sp.n_kv_heads, sp.head_dim),
                                dtype=torch.uint8, device=dev)
    dec_in = [wl.decode_inputs(s) for s in range(dec)]
    dec_out = [torch.empty_like(d["q"]) for d in dec_in]
    dec_rot = [torch.empty_like(d["q"]) for d in dec_in] if args.rope else None
    cu_dec = np.arange(len(L) + 1, dtype=np.int32)
    dgraph = cgraph = None
    if args.graph and args.chunk_tokens:
        # all scheduler steps of the chunked prefill as one graph (its eager
        # pass also leaves the prefill's K/V in the pools)
        cgraph = ChunkGraph(pc, cached, tables, L, q, k_new, v_new, out, sp.scale, args.chunk_tokens, inv_freq,
                            q_rot)
        torch.cuda.synchronize()
    if args.graph and dec:
        # the prefill's K/V must be in the pools before the eager pass of the capture
        b = pc.upload_prefill(cached, tables, L, stream)
        pc.append(b, k_new, v_new, stream)
        torch.cuda.synchronize()
        dgraph = DecodeGraph(pc, tables, L, dec_in, dec_out, sp.scale)
        torch.cuda.synchronize()
    work = workload_work(wl, cached, tables)
    n_tokens = work["query_tokens"] + dec * len(L)

    n_ev = args.steps + args.warmup
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(n_ev)]
    # decode attention launches, timed apart from their appends and uploads
    n_dev = dec if dgraph is None else 0
    dev_ev = [[(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
               for _ in range(n_dev)] for _ in range(n_ev)]
    flush = torch.empty(args.flush_mib << 20, dtype=torch.uint8, device=dev) if args.flush_mib else None
    host_s = []

    def step(i):
        e = ev[i]
        if flush is not None:
            flush.fill_(i & 0xFF)
        h0 = time.perf_counter()
        m = pc.cache.checkpoint()
        c, t = pc.match(packed=(tokens, cu_tok), reserve=reserve)
        b = None if args.chunk_tokens else pc.upload_prefill(c, t, L, stream)
        pc.cache.rollback(m)
        host_s.append(time.perf_counter() - h0)
        e[0].record(stream)
        if cgraph is not None:   # every scheduler step, replayed as one graph
            assert np.array_equal(t, tables), "block tables changed since the capture"
            e[1].record(stream)
            cgraph.replay()
        elif args.chunk_tokens:   # appends and attention interleave, chunk by chunk
            e[1].record(stream)
            pc.prefill_chunked(c, t, L, q, k_new, v_new, out, sp.scale, args.chunk_tokens, stream,
                               inv_freq, q_rot)
        else:
            if args.rope:
                pc.append_rope(b, k_new, v_new, inv_freq, q, q_rot, stream)
            else:
                pc.append(b, k_new, v_new, stream)
            e[1].record(stream)
            if split_prefill:
                pc.attend_cascade(b, q, out, sp.scale, shared_len, cascade_ws, stream)
            else:
                pc.attend(b, q_rot if args.rope else q, out, sp.scale, stream)
        e[2].record(stream)
        if dgraph is not None:
            assert np.array_equal(t, tables), "block tables changed since the capture"
            dgraph.replay()
        for s in range(dec if dgraph is None else 0):
            bd = pc.upload(t, cu_dec, L + s + 1, L + s, stream)
            qd = dec_in[s]["q"]
            if args.rope:
                pc.append_rope(bd, dec_in[s]["k_new"], dec_in[s]["v_new"], inv_freq, qd, dec_rot[s], stream)
                qd = dec_rot[s]
            else:
                pc.append(bd, dec_in[s]["k_new"], dec_in[s]["v_new"], stream)
            dev_ev[i][s][0].record(stream)
            if split_decode:
                pc.attend_cascade(bd, qd, dec_out[s], sp.scale, shared_len, decode_ws, stream)
            else:
                pc.attend(bd, qd, dec_out[s], sp.scale, stream)
            dev_ev[i][s][1].record(stream)
        e[3].record(stream)
        return c

    for i in range(args.warmup):
        c = step(i)
    torch.cuda.synchronize()
    assert np.array_equal(c, cached), "cached lengths changed between steps"
    host_s.clear()
    t0 = time.perf_counter()
    for i in range(args.warmup, n_ev):
        step(i)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0

    timed = ev[args.warmup:]
    attn_ms = float(np.mean([e[1].elapsed_time(e[2]) for e in timed]))
    append_ms = float(np.mean([e[0].elapsed_time(e[1]) for e in timed]))
    decode_ms = float(np.mean([e[2].elapsed_time(e[3]) for e in timed])) if dec else 0.0
    ms_per_step = elapsed * 1e3 / args.steps
    tflops = work["flops"] / (attn_ms * 1e-3) / 1e12
    gbs = work["logical_bytes"] / (attn_ms * 1e-3) / 1e9
    unique_gbs = work["unique_bytes"] / (attn_ms * 1e-3) / 1e9
    # roofline of the prefill launch: t_roof = max(FLOPs / MFMA peak, unique bytes / HBM peak);
    # the launch is bound by whichever term is larger
    t_mfma = work["flops"] / (PEAK_BF16_TFLOPS * 1e12)
    t_hbm = work["unique_bytes"] / (PEAK_HBM_GBS * 1e9)
    traffic = None if args.prompts else traffic_from_profile(traffic_key(args, split_prefill))
    if t_mfma >= t_hbm:
        roof = {"bound": "mfma", "achieved": round(tflops, 2), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                "frac": round(tflops / PEAK_BF16_TFLOPS, 4), "traffic": traffic}
    else:
        roof = {"bound": "hbm", "achieved": round(unique_gbs, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                "frac": round(unique_gbs / PEAK_HBM_GBS, 4), "traffic": traffic}
    attn = {"launch_us": round(attn_ms * 1e3, 2), "tflops": round(tflops, 2),
            "mfma_frac": round(tflops / PEAK_BF16_TFLOPS, 4),
            "flops": work["flops"], "logical_bytes": work["logical_bytes"], "unique_bytes": work["unique_bytes"],
            "logical_gbs": round(gbs, 1), "logical_hbm_frac": round(gbs / PEAK_HBM_GBS, 4),
            "unique_gbs": round(unique_gbs, 1), "t_mfma_us": round(t_mfma * 1e6, 2),
            "t_unique_hbm_us": round(t_hbm * 1e6, 2), "roofline_frac": round(max(t_mfma, t_hbm) / (attn_ms * 1e-3), 4),
            "kernel_sha": kernel_source_sha()}
    decode = None
    if n_dev:
        per = np.array([[a.elapsed_time(b) for (a, b) in e] for e in dev_ev[args.warmup:]])   # [steps, dec] ms
        Ld = wl.seq_lens.astype(np.float64)
        kv = 4.0 * sp.n_kv_heads * sp.head_dim
        qo = 4.0 * sp.n_q_heads * sp.head_dim * len(Ld)
        bytes_step = np.array([kv * float(np.sum(Ld + s + 1)) + qo for s in range(dec)])
        us = per.mean(axis=0) * 1e3
        dgbs = float(np.mean(bytes_step / (us * 1e-6) / 1e9))
        decode = {"attn_us_per_step": round(float(us.mean()), 2), "bytes_per_step": float(bytes_step.mean()),
                  "logical_gbs": round(dgbs, 1), "hbm_frac": round(dgbs / PEAK_HBM_GBS, 4),
                  "flush_mib": args.flush_mib}

    line = {
        "metric": METRIC,
        "value": round(n_tokens * args.steps / elapsed, 1),
        "unit": "query tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": sp.name, "prompts": len(wl.prompts), "q_heads": sp.n_q_heads,
                   "kv_heads": sp.n_kv_heads, "head_dim": sp.head_dim, "block": 16,
                   "query_tokens": work["query_tokens"], "decode_steps": dec,
                   "cached_fraction": round(float(cached.sum() / wl.seq_lens.sum()), 4),
                   "attention": {"prefill": "shared-prefix split" if split_prefill else "single pass",
                                 **({"decode": "shared-prefix split" if split_decode else "single pass"}
                                    if dec else {}),
                                 "shared_len": shared_len,
                                 "chosen_by": "--cascade" if args.cascade else ("library rule" if auto else "flags")},
                   **({"chunk_tokens": args.chunk_tokens, "chunks": n_chunks} if args.chunk_tokens else {}),
                   **({"rope_base": args.rope} if args.rope else {}),
                   **({"decode_graph": True} if dgraph is not None else {}),
                   **({"chunk_graph": True} if cgraph is not None else {}),
                   **({"flush_mib": args.flush_mib} if args.flush_mib else {}),
                   **(icl or {})},
        "roofline": {**roof, **({"scope": f"all {n_chunks} chunked steps: appends, attention and the "
                                         "host's per-step metadata copies"} if args.chunk_tokens else {})},
        "attn": attn,
        **({"decode_attn": decode} if decode else {}),
        "breakdown_ms": {"host_match_upload": round(float(np.mean(host_s)) * 1e3, 4),
                         "kv_append": round(append_ms, 4), "attention": round(attn_ms, 4),
                         "decode_steps": round(decode_ms, 4)},
    }
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(wl, cached, work, n_tokens, args.cpu_budget,
                                            args.cpu_decode_budget)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
