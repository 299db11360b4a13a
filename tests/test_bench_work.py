"""The benchmark's algorithmic work model (CPU only): visible pairs, FLOPs,
logical and unique bytes of a prefill launch, checked against brute-force
counts over the host prefix match's block tables."""
import os

import numpy as np
import pytest

from paper_2507_08523_amd import ilpc, workload

import bench


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(ilpc.LIB_PATH):
        pytest.fail("libilpc.so is not built: run `python -m paper_2507_08523_amd.build`")
    return ilpc.load()


def _match(wl):
    cache = ilpc.PrefixCache(1 << 20, 22)
    mb = max(-(-(len(p) + wl.spec.decode_steps) // 16) for p in wl.prompts)
    if wl.warm:
        cache.match(wl.warm, max_blocks=max(-(-len(p) // 16) for p in wl.warm))
    res = [wl.spec.decode_steps] * len(wl.prompts) if wl.spec.decode_steps else None
    c, t, _ = cache.match(wl.prompts, reserve=res, max_blocks=mb)
    return c, t


def _brute(wl, c, t):
    sp = wl.spec
    pairs = 0
    slots = {}
    for r, p in enumerate(wl.prompts):
        L, P = len(p), int(c[r])
        for i in range(P, L):          # query at absolute position i sees keys 0..i
            pairs += i + 1
        for pos in range(L):           # every key slot the request reads
            b = int(t[r, pos // 16])
            slots.setdefault(b, set()).add(pos % 16)
    kv_tok = 4 * sp.n_kv_heads * sp.head_dim
    qo = 4 * sp.n_q_heads * sp.head_dim * int(sum(len(p) for p in wl.prompts) - c.sum())
    logical = kv_tok * sum(len(p) for p in wl.prompts) + qo
    unique = kv_tok * sum(max(s) + 1 for s in slots.values()) + qo
    return pairs, logical, unique


@pytest.mark.parametrize("spec", [workload.SPECS["tiny"], workload.scaled_spec("llama8b", 12),
                                  workload.scaled_spec("sweep100", 6), workload.scaled_spec("large", 3),
                                  workload.scaled_spec("qwen7b", 5)])
def test_work_model_matches_brute_force(lib, spec):
    wl = workload.build(spec)
    c, t = _match(wl)
    w = bench.workload_work(wl, c, t)
    pairs, logical, unique = _brute(wl, c, t)
    assert w["pairs"] == pairs
    assert w["flops"] == 4 * spec.n_q_heads * spec.head_dim * pairs
    assert w["logical_bytes"] == logical
    assert w["unique_bytes"] == unique
    assert w["unique_bytes"] <= w["logical_bytes"]


def test_sweep100_unique_bytes_count_the_shared_prefix_once(lib):
    # 128 prompts share 976 tokens (61 blocks); each has 3 private blocks of
    # its 48-token query: logical bytes read the prefix 128 times, unique once
    wl = workload.build("sweep100")
    c, t = _match(wl)
    w = bench.workload_work(wl, c, t)
    kv_tok = 4 * 8 * 128
    qo = 4 * 32 * 128 * 128 * 48
    assert w["logical_bytes"] == kv_tok * 128 * 1024 + qo
    assert w["unique_bytes"] == kv_tok * (976 + 128 * 48) + qo
    assert abs(w["unique_bytes"] / 1e6 - 130) < 1 and abs(w["logical_bytes"] / 1e6 - 638) < 1


def test_kernel_hash_ignores_comments_only(tmp_path, monkeypatch):
    # the counter summaries are keyed on the kernel's code: a comment edit
    # keeps the hash, a code edit changes it
    import bench

    src = tmp_path / "k.hip"
    src.write_text("int f(int x) {  // doubles\n  return 2 * x;\n}\n")
    monkeypatch.setattr(bench, "KERNEL_SRC", str(src))
    h0 = bench.kernel_source_sha()
    src.write_text("// a new header line\nint f(int x) {  // twice x\n\n  return 2 * x;   \n}\n")
    assert bench.kernel_source_sha() == h0
    src.write_text("int f(int x) {\n  return 3 * x;\n}\n")
    assert bench.kernel_source_sha() != h0


def test_traffic_summary_matches_the_launch_variant():
    # a run reports measured traffic only from the summary of the same
    # launches: the shared-prefix split, chunked steps and an unrefined ICL
    # batch each have their own
    import argparse

    import bench

    def key(split=False, **kw):
        a = dict(workload="sweep100", cascade=False, chunk_tokens=0, no_pair=False, rope=0.0, graph=False)
        a.update(kw)
        return bench.traffic_key(argparse.Namespace(**a), split)

    assert key() == "sweep100"
    assert key(rope=5e5, graph=True) == "sweep100"
    assert key(split=True) == "sweep100_cascade"
    assert key(workload="llama8b", chunk_tokens=1024) == "llama8b_chunk1024"
    assert key(workload="icl_llama8b", no_pair=True) == "icl_llama8b_nopair"


def test_committed_summaries_name_the_current_kernel_code(monkeypatch):
    # every counter or trace summary under profiles/ names the code hash of
    # the kernel source it was taken on; after a code change the summaries
    # must be taken again (bench.py then reports traffic as unmeasured)
    import re

    import bench

    root = bench.ROOT

    def sha(name):
        monkeypatch.setattr(bench, "KERNEL_SRC", os.path.join(root, "paper_2507_08523_amd", "csrc", name))
        return bench.kernel_source_sha()

    current = {"paged_attn.hip": sha("paged_attn.hip"), "decode_attn.hip": sha("decode_attn.hip")}
    prof = os.path.join(root, "profiles")
    checked = 0
    for fname in sorted(os.listdir(prof)):
        text = open(os.path.join(prof, fname), encoding="utf-8").read()
        src = "decode_attn.hip" if fname.startswith("decode_attn") else "paged_attn.hip"
        found = re.findall(r"kernel code hash ([0-9a-f]{16})", text)
        found += re.findall(r"^kernel_source_sha: ([0-9a-f]{16})$", text, re.M)
        found += re.findall(r"^\w+ \| ([0-9a-f]{16}) \|", text, re.M)
        assert found, f"{fname} names no kernel code hash"
        assert set(found) == {current[src]}, (fname, set(found), current[src])
        checked += 1
    assert checked >= 20
