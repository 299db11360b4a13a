"""Oracle: dense float64 causal grouped-query attention (test infrastructure).

What is computed (InferLog, section 2.1.2): prefill runs the whole prompt
through the model in one parallel pass; with prefix caching only the
cache-missing suffix is computed, and it attends to the reused KV of the
cached prefix plus its own freshly stored KV (section 3.2.2).  Because a
token's K/V depends only on the tokens before it (section 2.1.2), the result
is by definition the suffix rows of ordinary causal attention over the whole
prompt -- which is what this module writes out, on the request's dense K/V.
It never sees a paged pool or a block table.

Readings taken where the paper is silent: softmax scale passed in (1/sqrt(D)
in every workload); absolute positions with the suffix bottom-right aligned
(query t of a request with L keys and S queries sits at position L - S + t and
sees keys 0..L-S+t); grouped-query heads in contiguous groups
(kv head = q head // (Hq / Hkv)); K arrives with positions already applied.

Inputs are the exact bf16 values (as any float array); arithmetic is float64.
"""
from __future__ import annotations

import numpy as np


def prefill_attention_ref(q, k, v, scale: float) -> np.ndarray:
    """Causal GQA attention of S suffix queries over L keys of one request.

    q: [S, Hq, D]; k, v: [L, Hkv, D] with S <= L.  Returns float64 [S, Hq, D].
    """
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    S, Hq, D = q.shape
    L, Hkv, Dk = k.shape
    assert Dk == D and v.shape == k.shape and 1 <= S <= L and Hq % Hkv == 0
    G = Hq // Hkv
    pos = (L - S) + np.arange(S)                     # absolute query positions
    visible = np.arange(L)[None, :] <= pos[:, None]  # [S, L] causal mask
    out = np.empty((S, Hq, D), dtype=np.float64)
    for h in range(Hq):
        g = h // G
        scores = scale * (q[:, h, :] @ k[:, g, :].T)           # [S, L]
        scores = np.where(visible, scores, -np.inf)
        scores = scores - scores.max(axis=1, keepdims=True)
        p = np.exp(scores)
        p = p / p.sum(axis=1, keepdims=True)
        out[:, h, :] = p @ v[:, g, :]
    return out


def decode_step_ref(q_row, k, v, scale: float) -> np.ndarray:
    """One decode query (the newest token, position L-1) over keys 0..L-1.

    q_row: [Hq, D]; k, v: [L, Hkv, D].  Equals the last row of a prefill of
    length L.  Returns float64 [Hq, D].
    """
    q_row = np.asarray(q_row)
    return prefill_attention_ref(q_row[None], k, v, scale)[0]
