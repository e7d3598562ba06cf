"""Pins of the oracle's rotary encoding and key re-alignment (oracle/rope.py)."""
import numpy as np
import pytest

from oracle import rope


def _complex_form(x, pos, w):
    """Independent formulation: pair (x_i, x_{i+D/2}) as a complex number times exp(j p w_i)."""
    half = x.shape[-1] // 2
    z = x[..., :half] + 1j * x[..., half:]
    z = z * np.exp(1j * np.asarray(pos, dtype=np.float64)[..., None] * w)
    return np.concatenate([z.real, z.imag], axis=-1)


def test_inv_freq_hand_values():
    np.testing.assert_allclose(rope.inv_freq(4, 1e4), [1.0, 1e-2], rtol=1e-15)
    w = rope.inv_freq(128, 1e6)
    assert w[0] == 1.0
    np.testing.assert_allclose(w[-1], 1e6 ** (-126 / 128), rtol=1e-15)
    assert np.all(np.diff(w) < 0)


def test_quarter_and_half_turn_by_hand():
    w = np.array([1.0])                               # D = 2: a single pair at unit frequency
    np.testing.assert_allclose(rope.rotate(np.array([3.0, 4.0]), np.pi / 2, w), [-4.0, 3.0], atol=1e-15)
    np.testing.assert_allclose(rope.rotate(np.array([3.0, 4.0]), np.pi, w), [-3.0, -4.0], atol=1e-15)
    # pair i of D = 4 uses dims (i, i + 2)
    w4 = rope.inv_freq(4, 100.0)                       # [1, 0.1]
    y = rope.rotate(np.array([1.0, 0.0, 0.0, 0.0]), 2.0, w4)
    np.testing.assert_allclose(y, [np.cos(2.0), 0.0, np.sin(2.0), 0.0], atol=1e-15)
    y = rope.rotate(np.array([0.0, 1.0, 0.0, 0.0]), 2.0, w4)
    np.testing.assert_allclose(y, [0.0, np.cos(0.2), 0.0, np.sin(0.2)], atol=1e-15)


@pytest.mark.parametrize("D,theta", [(64, 1e4), (128, 1e6)])
def test_matches_complex_exponential(D, theta):
    rng = np.random.default_rng(0)
    x = rng.standard_normal((300, 4, D))
    pos = rng.integers(-40000, 40000, size=(300, 1)).astype(np.float64)
    w = rope.inv_freq(D, theta)
    np.testing.assert_allclose(rope.rotate(x, pos, w), _complex_form(x, pos, w), rtol=0, atol=1e-12)


def test_zero_turn_is_identity_exactly():
    rng = np.random.default_rng(1)
    x = rng.standard_normal((50, 8, 128))
    np.testing.assert_array_equal(rope.rotate(x, 0, rope.inv_freq(128, 1e6)), x)


@pytest.mark.parametrize("D,theta", [(64, 1e4), (128, 1e6)])
def test_composition_on_keys_from_pre_encoding_values(D, theta):
    """R(p + delta) k_raw == R(delta) R(p) k_raw (keys recomputed from pre-RoPE values)."""
    rng = np.random.default_rng(2)
    w = rope.inv_freq(D, theta)
    k_raw = rng.standard_normal((400, 2, D))
    p = np.arange(400, dtype=np.float64)[:, None]           # source positions 0..399
    for delta in (1, 17, 1024, 4095, 30000, -250):
        a = rope.rotate(rope.rotate(k_raw, p, w), delta, w)
        b = rope.rotate(k_raw, p + delta, w)
        # float64 angles carry 2^-53 relative rounding: the bound scales with the angle
        tol = 2.0 ** -50 * (400 + abs(delta)) * np.abs(k_raw).max()
        np.testing.assert_allclose(a, b, rtol=0, atol=max(tol, 1e-13))


def test_isometry_per_pair():
    rng = np.random.default_rng(3)
    D = 128
    x = rng.standard_normal((100, D))
    y = rope.rotate(x, rng.integers(-5000, 5000, 100), rope.inv_freq(D, 1e6))
    n0 = np.hypot(x[:, :D // 2], x[:, D // 2:])
    n1 = np.hypot(y[:, :D // 2], y[:, D // 2:])
    np.testing.assert_allclose(n0, n1, rtol=1e-13)


def test_relative_position_property():
    """<R(m) q, R(n) k> depends on m - n only."""
    rng = np.random.default_rng(4)
    D = 64
    w = rope.inv_freq(D, 1e4)
    q, k = rng.standard_normal(D), rng.standard_normal(D)
    ref = rope.rotate(q, 7, w) @ k
    for m in (7, 100, 2000, 12345):
        n = m - 7
        np.testing.assert_allclose(rope.rotate(q, m, w) @ rope.rotate(k, n, w), ref, rtol=1e-10)
