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

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload llama8b] [--prompts N] [--cascade] [--no-pair]

``--cascade`` runs the prefill attention split at the prefix every prompt of
the batch shares (ilpc_paged_prefill_attn_cascade).

``--rope BASE`` rotates the new tokens' K and Q at their positions inside the
append (ilpc_rope_kv_append; the warm prefix is rotated the same way).
``--chunk-tokens N`` runs the prefill as scheduler steps of at most N new
tokens (append + attention per step); the attention timing and ``roofline``
then cover all steps.  ``--graph`` (decode workloads) captures the 32 decode
steps once as a HIP graph with all their metadata on the device, and every
timed step replays it.  ``--prompts N`` keeps the workload's shapes with N
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


def workload_work(wl, cached_len):
    """Algorithmic FLOPs and bytes of one prefill attention launch."""
    sp = wl.spec
    L = wl.seq_lens.astype(np.float64)
    P = np.asarray(cached_len, dtype=np.float64)
    S = L - P
    pairs = float(np.sum(S * P + S * (S + 1) / 2))   # visible (query, key) pairs
    flops = 4.0 * sp.n_q_heads * sp.head_dim * pairs
    kv_bytes = float(np.sum(4.0 * sp.n_kv_heads * sp.head_dim * L))   # K + V context, bf16
    qo_bytes = float(np.sum(4.0 * sp.n_q_heads * sp.head_dim * S))     # Q in + O out, bf16
    return {"pairs": pairs, "flops": flops, "logical_bytes": kv_bytes + qo_bytes,
            "query_tokens": int(S.sum())}


def kernel_source_sha() -> str:
    with open(KERNEL_SRC, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


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


def cpu_baseline(wl, cached_len, budget_s: float):
    """Time the fp64 oracle (prefix match of the whole batch + attention of
    requests in a seeded order, passing over the batch again while the budget
    lasts) on the host cores."""
    from threadpoolctl import threadpool_info

    from oracle.attn_ref import prefill_attention_ref
    from oracle.prefix_ref import PrefixCacheRef

    ref = PrefixCacheRef(1 << 30, 1 << 30)
    if wl.warm:
        ref.match(wl.warm)
    t0 = time.perf_counter()
    c_ref, _, _ = ref.match(wl.prompts)
    t_match = time.perf_counter() - t0
    assert np.array_equal(c_ref, cached_len)
    rng = np.random.default_rng(0)
    order = rng.permutation(len(wl.prompts))
    t_attn, tokens, done = 0.0, 0, 0
    for i in range(len(order) * 1000):
        r = order[i % len(order)]
        L, P = int(wl.seq_lens[r]), int(cached_len[r])
        k, v = wl.dense_kv(int(r), L)
        q = wl.q_rows(int(r), P, L).float().cpu().numpy().astype(np.float64)
        k = k.float().cpu().numpy().astype(np.float64)
        v = v.float().cpu().numpy().astype(np.float64)
        t0 = time.perf_counter()
        prefill_attention_ref(q, k, v, wl.spec.scale)
        t_attn += time.perf_counter() - t0
        tokens += L - P
        done += 1
        if t_attn >= budget_s:
            break
    total_q = int(np.sum(wl.seq_lens - cached_len))
    sec_per_token = t_match / total_q + t_attn / tokens
    threads = max([i.get("num_threads", 1) for i in threadpool_info() if i.get("user_api") == "blas"] + [1])
    return {"value": 1.0 / sec_per_token, "unit": "query tokens/s", "cores": int(threads),
            "kind": "oracle",
            "sample": (f"fp64 oracle: prefix match of all {len(wl.prompts)} prompts ({t_match*1e3:.1f} ms) + "
                       f"attention of {done} requests of the {len(wl.prompts)} in a seeded order, "
                       f"repeated once the batch is done ({tokens} query tokens, {t_attn:.1f} s); "
                       f"host nproc={os.cpu_count()}")}


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
    ap.add_argument("--workload", default="llama8b")
    ap.add_argument("--prompts", type=int, default=0,
                    help="run the workload's shapes with this many prompts (0: its own count)")
    ap.add_argument("--cpu-budget", type=float, default=12.0, help="seconds of oracle attention to time")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-pair", action="store_true",
                    help="ICL stream workloads: serve the selector's demonstration order unrefined")
    ap.add_argument("--chunk-tokens", type=int, default=0,
                    help="prefill in scheduler steps of at most this many new tokens (0: one pass)")
    ap.add_argument("--rope", type=float, default=0.0, metavar="BASE",
                    help="rotate new K and Q with RoPE of this base inside the append (0: off)")
    ap.add_argument("--graph", action="store_true",
                    help="decode workloads: replay the decode steps as one captured HIP graph")
    ap.add_argument("--cascade", action="store_true",
                    help="split the prefill attention at the prefix every prompt shares")
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="run one plain device copy of this many MiB first (counter calibration)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (got --gpus {args.gpus}); the path needs no collective "
              "and every box here has one GPU", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2507_08523_amd import ilpc, workload
    from paper_2507_08523_amd.pipeline import (DecodeGraph, PagedPrefixCache, chunk_schedule, max_blocks_of,
                                               pool_blocks_needed, rope_inv_freq, shared_prefix_len)

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

    if args.cascade and (args.rope or args.chunk_tokens):
        print("--cascade does not combine with --rope or --chunk-tokens", file=sys.stderr)
        sys.exit(2)
    if args.graph and (args.cascade or args.rope):
        print("--graph does not combine with --cascade or --rope", file=sys.stderr)
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
    shared_len, cascade_ws = 0, None
    if args.cascade:
        shared_len = shared_prefix_len(cached, tables)
        n_ws = ilpc.attn_cascade_workspace_bytes(len(wl.prompts), int((wl.seq_lens - cached).max()),
                                                 sp.n_q_heads, sp.n_kv_heads, sp.head_dim)
        cascade_ws = torch.zeros(n_ws, dtype=torch.uint8, device=dev)
        decode_ws = torch.zeros(ilpc.attn_cascade_workspace_bytes(len(wl.prompts), 1, sp.n_q_heads,
                                                                  sp.n_kv_heads, sp.head_dim),
                                dtype=torch.uint8, device=dev)
    L = wl.seq_lens.astype(np.int32)
    dec_in = [wl.decode_inputs(s) for s in range(dec)]
    dec_out = [torch.empty_like(d["q"]) for d in dec_in]
    dec_rot = [torch.empty_like(d["q"]) for d in dec_in] if args.rope else None
    cu_dec = np.arange(len(L) + 1, dtype=np.int32)
    dgraph = None
    if args.graph and dec:
        # the prefill's K/V must be in the pools before the eager pass of the capture
        b = pc.upload_prefill(cached, tables, L, stream)
        pc.append(b, k_new, v_new, stream)
        torch.cuda.synchronize()
        dgraph = DecodeGraph(pc, tables, L, dec_in, dec_out, sp.scale)
        torch.cuda.synchronize()
    work = workload_work(wl, cached)
    n_tokens = work["query_tokens"] + dec * len(L)

    n_ev = args.steps + args.warmup
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(n_ev)]
    host_s = []

    def step(i):
        e = ev[i]
        h0 = time.perf_counter()
        m = pc.cache.checkpoint()
        c, t = pc.match(packed=(tokens, cu_tok), reserve=reserve)
        b = None if args.chunk_tokens else pc.upload_prefill(c, t, L, stream)
        pc.cache.rollback(m)
        host_s.append(time.perf_counter() - h0)
        e[0].record(stream)
        if args.chunk_tokens:   # appends and attention interleave, chunk by chunk
            e[1].record(stream)
            pc.prefill_chunked(c, t, L, q, k_new, v_new, out, sp.scale, args.chunk_tokens, stream,
                               inv_freq, q_rot)
        else:
            if args.rope:
                pc.append_rope(b, k_new, v_new, inv_freq, q, q_rot, stream)
            else:
                pc.append(b, k_new, v_new, stream)
            e[1].record(stream)
            if args.cascade:
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
            if args.cascade:
                pc.attend_cascade(bd, qd, dec_out[s], sp.scale, shared_len, decode_ws, stream)
            else:
                pc.attend(bd, qd, dec_out[s], sp.scale, stream)
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
    # the prefill launch is bound by whichever roofline limit is higher for it
    t_mfma = work["flops"] / (PEAK_BF16_TFLOPS * 1e12)
    t_hbm = work["logical_bytes"] / (PEAK_HBM_GBS * 1e9)
    traffic = None if args.prompts else traffic_from_profile(args.workload)
    if t_mfma >= t_hbm:
        roof = {"bound": "mfma", "achieved": round(tflops, 2), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                "frac": round(tflops / PEAK_BF16_TFLOPS, 4), "traffic": traffic}
    else:
        roof = {"bound": "hbm", "achieved": round(gbs, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                "frac": round(gbs / PEAK_HBM_GBS, 4), "traffic": traffic}

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
                   **({"cascade_shared_len": shared_len} if args.cascade else {}),
                   **({"chunk_tokens": args.chunk_tokens, "chunks": n_chunks} if args.chunk_tokens else {}),
                   **({"rope_base": args.rope} if args.rope else {}),
                   **({"decode_graph": True} if dgraph is not None else {}),
                   **(icl or {})},
        "roofline": {**roof, **({"scope": f"all {n_chunks} chunked steps: appends, attention and the "
                                         "host's per-step metadata copies"} if args.chunk_tokens else {})},
        "attn": {"launch_us": round(attn_ms * 1e3, 2), "tflops": round(tflops, 2),
                 "logical_gbs": round(gbs, 1), "flops": work["flops"], "logical_bytes": work["logical_bytes"],
                 "kernel_sha": kernel_source_sha()},
        "breakdown_ms": {"host_match_upload": round(float(np.mean(host_s)) * 1e3, 4),
                         "kv_append": round(append_ms, 4), "attention": round(attn_ms, 4),
                         "decode_steps": round(decode_ms, 4)},
    }
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(wl, cached, args.cpu_budget)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
