"""Pins of the rotary-embedding oracle (oracle/rope_ref.py).

* position 0 is the identity;
* a pair is a complex number turned by e^{i m theta} (RoFormer's complex
  form), computed here with numpy complex128 -- a different formulation from
  the oracle's cos/sin arithmetic;
* RoFormer's defining property: the dot product of a rotated query and key
  depends only on the distance of their positions;
* rotations compose (m then m' equals m + m') and keep each pair's length.
"""
import numpy as np
import pytest

from oracle.rope_ref import rope


def _inv_freq(D, base=10000.0):
    return (base ** (-np.arange(0, D, 2, dtype=np.float64) / D)).astype(np.float32)


@pytest.mark.parametrize("D", [2, 8, 64, 128])
def test_complex_form(D):
    rng = np.random.default_rng(D)
    x = rng.standard_normal((7, 3, D))
    pos = rng.integers(0, 5000, 7)
    f = _inv_freq(D)
    z = x[..., :D // 2] + 1j * x[..., D // 2:]
    z = z * np.exp(1j * pos[:, None, None] * f.astype(np.float64)[None, None, :])
    want = np.concatenate([z.real, z.imag], axis=-1)
    np.testing.assert_allclose(rope(x, pos, f), want, rtol=0, atol=1e-12)


def test_position_zero_is_identity():
    x = np.random.default_rng(1).standard_normal((4, 2, 64))
    np.testing.assert_array_equal(rope(x, np.zeros(4), _inv_freq(64)), x)


def test_dot_product_depends_only_on_distance():
    rng = np.random.default_rng(2)
    D = 128
    f = _inv_freq(D, 500000.0)
    q, k = rng.standard_normal((1, 1, D)), rng.standard_normal((1, 1, D))
    for m, n, t in [(5, 2, 100), (900, 17, 3), (0, 0, 2048)]:
        a = np.sum(rope(q, [m], f) * rope(k, [n], f))
        b = np.sum(rope(q, [m + t], f) * rope(k, [n + t], f))
        assert abs(a - b) < 1e-9
    # and it does depend on the distance
    a = np.sum(rope(q, [10], f) * rope(k, [0], f))
    b = np.sum(rope(q, [11], f) * rope(k, [0], f))
    assert abs(a - b) > 1e-3


def test_composition_and_pair_norms():
    rng = np.random.default_rng(3)
    D = 64
    f = _inv_freq(D)
    x = rng.standard_normal((5, 4, D))
    a, b = rng.integers(0, 3000, 5), rng.integers(0, 3000, 5)
    np.testing.assert_allclose(rope(rope(x, a, f), b, f), rope(x, a + b, f), atol=1e-9)
    y = rope(x, a, f)
    np.testing.assert_allclose(y[..., :D // 2] ** 2 + y[..., D // 2:] ** 2,
                               x[..., :D // 2] ** 2 + x[..., D // 2:] ** 2, rtol=1e-12)
