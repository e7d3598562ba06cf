"""Pins of the oracle's storage rounding (oracle/numerics.py)."""
import numpy as np
import pytest
import torch

from oracle import numerics


def _torch_bf16_bits(x32: np.ndarray) -> np.ndarray:
    t = torch.from_numpy(np.ascontiguousarray(x32, dtype=np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16)


def test_bf16_matches_torch_on_random_fp32():
    rng = np.random.default_rng(0)
    bits = rng.integers(0, 2**32, size=200_000, dtype=np.uint64).astype(np.uint32)
    x = bits.view(np.float32)
    x = x[np.isfinite(x) & (np.abs(x) < 3.38e38)]
    got = numerics.bf16_bits(numerics.bf16_round(x.astype(np.float64)))
    np.testing.assert_array_equal(got, _torch_bf16_bits(x))


def test_bf16_matches_torch_on_ties_and_subnormals():
    rng = np.random.default_rng(1)
    hi = rng.integers(0, 2**16, size=50_000, dtype=np.uint64).astype(np.uint32)
    hi = hi[(hi & 0x7F80) != 0x7F80]                          # finite
    hi = hi[(hi & 0x7FFF) < 0x7F7F]                           # rounding up stays finite
    ties = (hi << 16) | 0x8000                                # exactly half-way
    below = (hi << 16) | 0x7FFF
    above = (hi << 16) | 0x8001
    sub = rng.integers(1, 2**23, size=5000, dtype=np.uint64).astype(np.uint32)  # fp32 subnormals
    allb = np.concatenate([ties, below, above, sub, sub | 0x80000000]).astype(np.uint32)
    x = allb.view(np.float32)
    got = numerics.bf16_bits(numerics.bf16_round(x.astype(np.float64)))
    np.testing.assert_array_equal(got, _torch_bf16_bits(x))


def test_bf16_fp64_inputs_pick_nearest_neighbour():
    """Single rounding from float64: x between consecutive bf16 values a < b."""
    rng = np.random.default_rng(2)
    kb = rng.integers(0x0080, 0x7F00, size=4000).astype(np.uint16)   # positive normals
    a = numerics.bf16_value(kb)
    b = numerics.bf16_value(kb + 1)
    for t in (0.0, 0.25, 0.5 - 2**-30, 0.5, 0.5 + 2**-30, 0.75, 1.0):
        x = a + t * (b - a)
        got = numerics.bf16_round(x)
        if t < 0.5:
            exp = a
        elif t > 0.5:
            exp = b
        else:
            exp = np.where(kb % 2 == 0, a, b)        # tie: even mantissa
        np.testing.assert_array_equal(got, exp)
        np.testing.assert_array_equal(numerics.bf16_round(-x), -exp)


def test_bf16_double_rounding_case():
    """A float64 just above a bf16 half-way point must round up; via fp32 it would tie down."""
    a = numerics.bf16_value(np.array([0x3F80], dtype=np.uint16))[0]   # 1.0
    half = 2.0 ** -8                                                  # half of the bf16 step at 1.0
    x = a + half + 2.0 ** -40                                         # fp32 rounds this to the tie
    assert np.float32(x) == np.float32(a + half)
    assert numerics.bf16_round(np.array([x]))[0] == a + 2 * half


def test_f32_round_is_ieee():
    rng = np.random.default_rng(3)
    x = rng.standard_normal(10000) * 10.0 ** rng.integers(-30, 30, 10000)
    np.testing.assert_array_equal(numerics.round_to(x, "f32"), x.astype(np.float32).astype(np.float64))


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_encode_decode_roundtrip(dtype):
    rng = np.random.default_rng(4)
    x = rng.standard_normal(1000)
    e = numerics.encode(x, dtype)
    np.testing.assert_array_equal(numerics.decode(e, dtype), numerics.round_to(x, dtype))
    step = numerics.ulp(numerics.round_to(x, dtype), dtype)
    assert np.all(np.abs(numerics.round_to(x, dtype) - x) <= 0.5 * step * (1 + 1e-12))


def test_ulp_values():
    assert numerics.ulp(np.array([1.0]), "bf16")[0] == 2.0 ** -7
    assert numerics.ulp(np.array([1.0]), "f32")[0] == 2.0 ** -23
    assert numerics.ulp(np.array([0.75]), "bf16")[0] == 2.0 ** -8
