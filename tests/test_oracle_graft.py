"""Pins of the oracle's composite cache (oracle/graft.py)."""
import numpy as np
import pytest

from oracle import graft, numerics, rope


def _encoded_source(n, H, D, theta, dtype, seed=0, scale=1.0):
    """A source sequence: pre-encoding keys k_raw and their stored (encoded, rounded) form."""
    rng = np.random.default_rng(seed)
    k_raw = rng.standard_normal((n, H, D)) * scale
    w = rope.inv_freq(D, theta)
    stored = numerics.round_to(rope.rotate(k_raw, np.arange(n)[:, None], w), dtype)
    return k_raw, stored, w


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_graft_at_original_offsets_reproduces_source_exactly(dtype):
    D, H = 64, 2
    _, stored, w = _encoded_source(300, H, D, 1e4, dtype)
    v = numerics.round_to(np.random.default_rng(9).standard_normal((300, H, D)), dtype)
    cuts = [0, 64, 150, 151, 300]
    items = []
    for a, b in zip(cuts[:-1], cuts[1:]):                 # segment cut at source offset a
        items.append((a, a, numerics.encode(stored[a:b], dtype), numerics.encode(v[a:b], dtype)))
    items = items[::-1]                                   # order of the call must not matter
    K, V, written = graft.compose(320, H, D, items, w, dtype)
    np.testing.assert_array_equal(K[:300], stored)
    np.testing.assert_array_equal(V[:300], v)
    assert written[:300].all() and not written[300:].any()


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("dst", [0, 1, 777, 4000, 31000])
def test_graft_equals_encoding_at_target(dtype, dst):
    """A segment captured at positions 0..n-1 and grafted at dst carries R(dst + j) k_raw."""
    D, H, n = 128, 2, 200
    k_raw, stored, w = _encoded_source(n, H, D, 1e6, dtype, seed=dst, scale=0.5)
    got = graft.graft_keys(numerics.encode(stored, dtype), dst, w, dtype)
    exact = rope.rotate(k_raw, (dst + np.arange(n))[:, None], w)
    # error budget: the capture rounding of each pair member (<= ulp/2 each), turned by a
    # rotation (|cos| + |sin| <= sqrt 2), plus the final rounding (<= ulp/2 of the result)
    xs = numerics.decode(numerics.encode(stored, dtype), dtype)
    u_in = numerics.ulp(xs, dtype)
    half = D // 2
    u_pair = np.maximum(u_in[..., :half], u_in[..., half:])
    u_pair = np.concatenate([u_pair, u_pair], axis=-1)
    bound = 0.5 * numerics.ulp(got, dtype) + 0.5 * np.sqrt(2.0) * u_pair
    assert np.all(np.abs(got - exact) <= bound * (1 + 1e-9) + 1e-12 * np.abs(exact))
    if dtype == "f32":
        rel = np.abs(got - exact).max() / np.abs(exact).max()
        assert rel < 1e-6


def test_graft_composition_before_rounding():
    D = 64
    w = rope.inv_freq(D, 1e4)
    x = np.random.default_rng(1).standard_normal((50, 2, D))
    for d1, d2 in ((3, 5), (100, -40), (-7, -9), (1000, 2000)):
        a = rope.rotate(rope.rotate(x, d1, w), d2, w)
        tol = 2.0 ** -50 * (abs(d1) + abs(d2)) * np.abs(x).max()     # float64 angle rounding
        np.testing.assert_allclose(a, rope.rotate(x, d1 + d2, w), rtol=0, atol=max(tol, 1e-13))


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_values_copied_and_norms_kept(dtype):
    rng = np.random.default_rng(2)
    D = 128
    k = numerics.encode(rng.standard_normal((40, 8, D)), dtype)
    v = numerics.encode(rng.standard_normal((40, 8, D)), dtype)
    w = rope.inv_freq(D, 1e6)
    K, V, _ = graft.compose(100, 8, D, [(50, 0, k, v)], w, dtype)
    np.testing.assert_array_equal(V[50:90], numerics.decode(v, dtype))
    kd = numerics.decode(k, dtype)
    n0 = np.hypot(kd[..., :D // 2], kd[..., D // 2:])
    n1 = np.hypot(K[50:90, :, :D // 2], K[50:90, :, D // 2:])
    rel = 2.0 ** -8 if dtype == "bf16" else 2.0 ** -23
    assert np.all(np.abs(n1 - n0) <= 2 * rel * n0 + 1e-30)
    assert not K[:50].any() and not K[90:].any()


def test_overlapping_compose_rejected():
    k = np.zeros((4, 1, 4), dtype=np.float32)
    with pytest.raises(ValueError):
        graft.compose(10, 1, 4, [(0, 0, k, k), (3, 0, k, k)], rope.inv_freq(4, 1e4), "f32")


def test_fresh_encoding_matches_complex_form():
    rng = np.random.default_rng(3)
    D = 64
    w = rope.inv_freq(D, 1e4)
    x = rng.standard_normal((10, 4, D))
    pos = np.arange(100, 110)
    got = graft.encode_fresh(numerics.encode(x, "f32"), pos, w, "f32")
    z = (x[..., :32] + 1j * x[..., 32:]) * np.exp(1j * pos[:, None, None] * w)
    exact = np.concatenate([z.real, z.imag], axis=-1)
    assert np.abs(got - exact).max() <= 2e-6
