"""Pins of the attention oracle against facts outside itself.

* brute force: pure-Python loops over (query, head, key) with math.exp;
* library routine: torch's CPU float64 scaled_dot_product_attention with an
  explicit boolean causal mask and K/V heads repeated per group;
* closed forms: a query that sees one key returns that key's V row; Q = 0
  gives the running mean of V; constant V gives V;
* invariants: suffix rows of a prefix-cached prefill equal the same rows of the
  full prefill (section 2.1.2: a token's KV depends only on its prefix);
  grouped-query attention equals multi-head attention on repeated K/V;
  the output is linear in V; a decode step equals the last prefill row.
"""
import math

import numpy as np
import pytest
import torch

from oracle.attn_ref import decode_step_ref, prefill_attention_ref


def _rand(rng, *shape):
    # bf16-exact values, as the GPU path receives them
    x = torch.from_numpy(rng.standard_normal(shape).astype(np.float32)).to(torch.bfloat16)
    return x.double().numpy()


@pytest.mark.parametrize("S,L,Hq,Hkv,D", [(1, 1, 2, 1, 3), (3, 7, 4, 2, 3), (5, 5, 6, 3, 2),
                                          (4, 9, 4, 1, 5)])
def test_matches_pure_python_loops(S, L, Hq, Hkv, D):
    rng = np.random.default_rng(10 + S * L)
    q, k, v = _rand(rng, S, Hq, D), _rand(rng, L, Hkv, D), _rand(rng, L, Hkv, D)
    scale = 0.37
    got = prefill_attention_ref(q, k, v, scale)
    G = Hq // Hkv
    for t in range(S):
        pos = L - S + t
        for h in range(Hq):
            g = h // G
            w = []
            for j in range(pos + 1):
                w.append(math.exp(scale * sum(q[t, h, d] * k[j, g, d] for d in range(D))))
            tot = sum(w)
            for d in range(D):
                ref = sum(w[j] * v[j, g, d] for j in range(pos + 1)) / tot
                assert abs(got[t, h, d] - ref) < 1e-12 * max(1.0, abs(ref))


@pytest.mark.parametrize("S,L,Hq,Hkv,D", [(37, 101, 8, 2, 64), (16, 16, 4, 4, 128),
                                          (1, 50, 7, 1, 32)])
def test_matches_torch_sdpa_float64(S, L, Hq, Hkv, D):
    rng = np.random.default_rng(S + L + D)
    q, k, v = _rand(rng, S, Hq, D), _rand(rng, L, Hkv, D), _rand(rng, L, Hkv, D)
    scale = 1.0 / math.sqrt(D)
    got = prefill_attention_ref(q, k, v, scale)
    G = Hq // Hkv
    qt = torch.from_numpy(q).permute(1, 0, 2)                       # [Hq, S, D]
    kt = torch.from_numpy(k).permute(1, 0, 2).repeat_interleave(G, 0)
    vt = torch.from_numpy(v).permute(1, 0, 2).repeat_interleave(G, 0)
    pos = torch.arange(S) + (L - S)
    mask = torch.arange(L)[None, :] <= pos[:, None]
    ref = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, attn_mask=mask, scale=scale)
    np.testing.assert_allclose(got, ref.permute(1, 0, 2).numpy(), rtol=0, atol=1e-12)


def test_single_visible_key_returns_its_value():
    rng = np.random.default_rng(5)
    L = 12
    q, k, v = _rand(rng, L, 4, 16), _rand(rng, L, 2, 16), _rand(rng, L, 2, 16)
    got = prefill_attention_ref(q, k, v, 0.25)
    assert np.array_equal(got[0, :2], np.stack([v[0, 0], v[0, 0]]))
    assert np.array_equal(got[0, 2:], np.stack([v[0, 1], v[0, 1]]))


def test_zero_query_gives_running_mean():
    rng = np.random.default_rng(6)
    S, L = 9, 20
    k, v = _rand(rng, L, 1, 8), _rand(rng, L, 1, 8)
    got = prefill_attention_ref(np.zeros((S, 2, 8)), k, v, 1.0)
    for t in range(S):
        pos = L - S + t
        np.testing.assert_allclose(got[t, 0], v[: pos + 1, 0].mean(axis=0), atol=1e-14)
        np.testing.assert_allclose(got[t, 1], v[: pos + 1, 0].mean(axis=0), atol=1e-14)


def test_constant_values_pass_through():
    rng = np.random.default_rng(7)
    q, k = _rand(rng, 6, 4, 8), _rand(rng, 10, 2, 8)
    v = np.broadcast_to(np.arange(8.0)[None, None, :], (10, 2, 8)).copy()
    got = prefill_attention_ref(q, k, v, 0.5)
    np.testing.assert_allclose(got, np.broadcast_to(np.arange(8.0), got.shape), atol=1e-13)


def test_prefix_cached_rows_equal_full_prefill_rows():
    rng = np.random.default_rng(8)
    L, P = 70, 48
    q_full, k, v = _rand(rng, L, 8, 32), _rand(rng, L, 2, 32), _rand(rng, L, 2, 32)
    full = prefill_attention_ref(q_full, k, v, 0.2)
    cached = prefill_attention_ref(q_full[P:], k, v, 0.2)
    np.testing.assert_allclose(cached, full[P:], atol=1e-14)


def test_gqa_equals_mha_on_repeated_kv():
    rng = np.random.default_rng(9)
    q, k, v = _rand(rng, 11, 6, 16), _rand(rng, 30, 2, 16), _rand(rng, 30, 2, 16)
    gqa = prefill_attention_ref(q, k, v, 0.3)
    mha = prefill_attention_ref(q, np.repeat(k, 3, axis=1), np.repeat(v, 3, axis=1), 0.3)
    np.testing.assert_allclose(gqa, mha, atol=1e-14)


def test_linear_in_values():
    rng = np.random.default_rng(11)
    q, k = _rand(rng, 7, 4, 16), _rand(rng, 19, 2, 16)
    v1, v2 = _rand(rng, 19, 2, 16), _rand(rng, 19, 2, 16)
    a = prefill_attention_ref(q, k, v1, 0.3) + prefill_attention_ref(q, k, v2, 0.3)
    np.testing.assert_allclose(prefill_attention_ref(q, k, v1 + v2, 0.3), a, atol=1e-13)


def test_decode_step_equals_last_prefill_row():
    rng = np.random.default_rng(12)
    q, k, v = _rand(rng, 25, 8, 32), _rand(rng, 25, 1, 32), _rand(rng, 25, 1, 32)
    np.testing.assert_allclose(decode_step_ref(q[-1], k, v, 0.17),
                               prefill_attention_ref(q, k, v, 0.17)[-1], atol=1e-14)


def test_oracle_on_workload_inputs_is_finite_and_bounded():
    from paper_2507_08523_amd import workload

    wl = workload.build("tiny")
    wl.materialize("cpu")
    sp = wl.spec
    for r in range(len(wl.prompts)):
        L = len(wl.prompts[r])
        k, v = wl.dense_kv(r, L)
        q = wl.q_rows(r, 64, L)
        out = prefill_attention_ref(q.float().numpy(), k.float().numpy(), v.float().numpy(), sp.scale)
        assert np.isfinite(out).all()
        # a convex combination of V rows stays inside their range
        vv = v.float().numpy()
        assert (out <= vv.max(axis=0)[None] + 1e-12).all() and (out >= vv.min(axis=0)[None] - 1e-12).all()
