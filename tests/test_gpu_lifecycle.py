"""GPU: a request stream through an LRU prefix cache on a pool small enough to
evict, with kv_append and paged attention after every batch checked against
the fp64 oracle.

Blocks are released, cached, evicted and handed to later requests, which
append their own K/V into them; a later hit must read exactly the K/V of its
token prefix.  K/V are content-addressed (one slab per distinct full-block
token prefix of the stream, private slabs for partial blocks), so a block
handed out while still referenced, or a stale hit, shows up as an error.
"""
import sys

import numpy as np
import pytest
import torch

from oracle.attn_ref import prefill_attention_ref
from oracle.lifecycle_ref import LruPrefixCacheRef
from paper_2507_08523_amd import ilpc
from paper_2507_08523_amd.pipeline import PagedPrefixCache
from paper_2507_08523_amd.workload import cache_op_stream

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


class StreamKV:
    """Bf16 K/V of every position of a stream's prompts, by token prefix."""

    def __init__(self, Hkv, D, seed):
        self.Hkv, self.D, self.seed = Hkv, D, seed
        self.node = {}      # (parent node, block tokens) -> node id
        self.slab = {}      # node id -> (k, v) [16, Hkv, D] bf16 on the CPU
        self.n_private = 0

    def _draw(self, nid):
        if nid not in self.slab:
            g = torch.Generator().manual_seed(self.seed * 1_000_003 + nid)
            kv = torch.randn((2, BLOCK, self.Hkv, self.D), generator=g).to(torch.bfloat16)
            self.slab[nid] = (kv[0], kv[1])
        return self.slab[nid]

    def dense(self, prompt):
        """K, V [L, Hkv, D] of one prompt."""
        L = len(prompt)
        parent, ks, vs = -1, [], []
        for b in range(-(-L // BLOCK)):
            if (b + 1) * BLOCK <= L:
                key = (parent, prompt[b * BLOCK:(b + 1) * BLOCK].tobytes())
                parent = self.node.setdefault(key, len(self.node))
                nid = parent
            else:   # partial block: private to this request
                self.n_private += 1
                nid = -self.n_private
            k, v = self._draw(nid)
            ks.append(k)
            vs.append(v)
        return torch.cat(ks)[:L], torch.cat(vs)[:L]


@pytest.mark.parametrize("seed,n_blocks,Hq,Hkv,D", [(0, 40, 8, 2, 128), (1, 24, 4, 1, 64),
                                                     (2, 64, 16, 4, 128)])
def test_stream_with_eviction_against_oracle(seed, n_blocks, Hq, Hkv, D):
    dev = torch.device("cuda")
    max_blocks = 12
    pc = PagedPrefixCache(Hkv, D, n_blocks, max_blocks, 4, 8, dev, lru=True)
    ref = LruPrefixCacheRef(n_blocks)
    kv = StreamKV(Hkv, D, seed)
    rng = np.random.default_rng(300 + seed)
    scale = 1.0 / np.sqrt(D)
    live = []
    worst, tot, cnt, n_batches, n_hit_rows = 0.0, 0.0, 0, 0, 0
    for op, arg in cache_op_stream(seed, n_steps=70):
        if op == "match":
            try:
                c_ref, t_ref, _ = ref.match(arg, max_blocks=max_blocks)
            except Exception:
                with pytest.raises(ilpc.ILPCError):
                    pc.match(arg)
                continue
            c, t = pc.match(arg)
            assert np.array_equal(c, c_ref) and np.array_equal(t, t_ref)
            L = np.array([len(p) for p in arg], np.int32)
            dense = [kv.dense(p) for p in arg]
            qs = [torch.randn((int(L[r] - c[r]), Hq, D), generator=torch.Generator().manual_seed(
                int(rng.integers(1 << 30)))).to(torch.bfloat16) for r in range(len(arg))]
            k_new = torch.cat([dense[r][0][int(c[r]):] for r in range(len(arg))]).to(dev)
            v_new = torch.cat([dense[r][1][int(c[r]):] for r in range(len(arg))]).to(dev)
            q = torch.cat(qs).to(dev)
            out = torch.empty_like(q)
            print(f"[lifecycle] seed {seed} batch {n_batches}: L={L.tolist()} P={c.tolist()} "
                  f"usage={pc.cache.usage()}", flush=True)
            b = pc.upload_prefill(c, t, L)
            pc.append(b, k_new, v_new)
            pc.attend(b, q, out, scale)
            torch.cuda.synchronize()
            row = 0
            for r in range(len(arg)):
                S = int(L[r] - c[r])
                want = prefill_attention_ref(qs[r].float().numpy(), dense[r][0].float().numpy(),
                                             dense[r][1].float().numpy(), scale)
                got = out[row:row + S].float().cpu().numpy()
                err = np.abs(got - want)
                worst = max(worst, float(err.max()))
                tot += float(err.sum())
                cnt += err.size
                row += S
            n_batches += 1
            n_hit_rows += int(c.sum())
            live.extend(t)
        elif op == "release":
            k = int(round(arg * len(live)))
            picks = set(rng.permutation(len(live))[:k].tolist())
            rows = np.array([live[i] for i in sorted(picks)], np.int32).reshape(len(picks), max_blocks)
            pc.release(rows)
            ref.release(rows)
            live = [x for i, x in enumerate(live) if i not in picks]
        else:
            ids = [x for x in arg if x < n_blocks]
            pc.cache.touch(ids)
            ref.touch(ids)
        assert pc.cache.usage() == ref.usage()
    mean = tot / max(cnt, 1)
    ev = pc.cache.usage()[3]
    print(f"[lifecycle] seed {seed}: {n_batches} batches, {n_hit_rows} cached rows, {ev} evictions, "
          f"max_abs={worst:.3e} mean_abs={mean:.3e}", flush=True)
    sys.stdout.flush()
    assert n_batches >= 10 and n_hit_rows > 0 and ev > 0
    assert worst <= MAX_ABS and mean <= MEAN_ABS
