"""Oracle: rotary position embedding of key and query rows (test infrastructure).

What is computed: InferLog section 2.1.2 notes that the cached KV carries
each token's position, so the new tokens of a prompt are encoded at their
absolute positions (cached prefix length + offset) before their keys join the
reused ones.  The models the paper serves (Llama-3, Qwen2.5) encode positions
with rotary embeddings (Su et al., "RoFormer", 2021): the vector is split into
two-dimensional pairs, and pair i of the row at position m is turned by the
angle m * theta_i.

Readings (the paper does not spell the encoding out):

* pairs are (i, i + D/2) for i < D/2, the "rotate-half" arrangement of the
  Llama and Qwen checkpoints;
* theta_i is given as a table (fp32 values, e.g. base^(-2i/D)); scaled
  variants are a different table, not a different rotation;
* angles and the rotation are taken in float64 from those table values.

Plain numpy float64, no blocking.
"""
from __future__ import annotations

import numpy as np


def rope(x, positions, inv_freq) -> np.ndarray:
    """Rotate rows ``x`` [n, H, D] at ``positions`` [n]; returns float64 [n, H, D]."""
    x = np.asarray(x, dtype=np.float64)
    n, H, D = x.shape
    half = D // 2
    theta = np.asarray(inv_freq, dtype=np.float64).reshape(half)
    ang = np.asarray(positions, dtype=np.float64).reshape(n, 1) * theta.reshape(1, half)  # [n, D/2]
    c = np.cos(ang)[:, None, :]
    s = np.sin(ang)[:, None, :]
    lo, hi = x[..., :half], x[..., half:]
    return np.concatenate([lo * c - hi * s, hi * c + lo * s], axis=-1)
