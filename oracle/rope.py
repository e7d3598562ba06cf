"""Rotary position encoding and re-alignment of cached keys (oracle).

Reading of the paper (it names no positional scheme, App. B.1 runs the coder
model through HuggingFace Transformers): keys and queries carry the rotary
encoding of the Qwen2.5-Coder family in its "rotate-half" layout.  Dimension
``i`` and ``i + D/2`` form a pair that turns by the angle ``p * w_i`` at token
position ``p``, with ``w_i = theta ** (-2 i / D)``, ``i = 0 .. D/2 - 1``:

    y_i       = x_i       * cos(p w_i) - x_{i+D/2} * sin(p w_i)
    y_{i+D/2} = x_{i+D/2} * cos(p w_i) + x_i       * sin(p w_i)

A cached function module is reused wherever the new program places it (Sec.
4.1, two-tier code cache; the EPIC baseline of App. A.5 likewise re-aligns
cached key-value states to their new positions).  A key stored
encoded at source position ``p_src`` and grafted at target position ``p_dst``
is therefore turned by the delta ``p_dst - p_src``: since the rotations
compose, ``R(delta) R(p_src) k = R(p_dst) k``.  Values carry no position and
are copied unchanged.

The angle is the float64 product ``p * w_i`` (``w_i`` the float64 power), and
cos/sin are float64; this is the definition, not an fp32 approximation.

Pins (tests/test_oracle_rope.py): equality with the complex-exponential form
``(x_i + j x_{i+D/2}) * exp(j p w_i)`` (numpy complex exp), R(0) = I exactly,
R(a) R(b) = R(a + b) on keys recomputed from pre-encoding values (<= 1e-12),
isometry per pair, the relative-position property of dot products, and a
hand-worked quarter-turn.
"""
from __future__ import annotations

import numpy as np


def inv_freq(head_dim: int, theta: float) -> np.ndarray:
    """w_i = theta ** (-2 i / D), i = 0 .. D/2 - 1 (float64)."""
    if head_dim % 2:
        raise ValueError("head_dim must be even")
    i = np.arange(head_dim // 2, dtype=np.float64)
    return np.power(float(theta), -2.0 * i / float(head_dim))


def rotate(x, pos, w) -> np.ndarray:
    """Turn every rotary pair of ``x[..., D]`` by ``pos * w_i``.

    ``pos`` broadcasts against ``x[..., 0]`` (one position per row); it may be
    negative (a delta).  float64 in, float64 out.
    """
    x = np.asarray(x, dtype=np.float64)
    half = x.shape[-1] // 2
    ang = np.asarray(pos, dtype=np.float64)[..., None] * np.asarray(w, dtype=np.float64)
    c, s = np.cos(ang), np.sin(ang)
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)
