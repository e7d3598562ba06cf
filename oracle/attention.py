"""Causal grouped-query attention over the grafted cache (oracle).

Only the new span's tokens are computed; they attend over the cached states
before them (Sec. 4.2, Eq. 6; App. B.1, cache-patching), and every decode step
attends to the whole cache built so far.  Reading of what the paper leaves open (the
model is a Qwen2.5-Coder checkpoint run through HuggingFace Transformers,
Sec. 5.1 and App. B.1): standard scaled-dot-product softmax attention, scale
``1 / sqrt(D)``, no soft-capping, bias or window; grouped-query heads with
query head ``hq`` reading key/value head ``hq // g`` (``g = Hq / Hkv``); the
causal mask is by *position*: a query at position ``p`` sees every cached
position ``<= p`` (grafted or fresh), and nothing else.

For query row ``q`` (already rotary-encoded at ``p`` and rounded to the storage
dtype) and key/value head ``h``:

    s_j = (q . k_j) / sqrt(D),   j = 0 .. p
    a_j = exp(s_j - max_i s_i) / sum_i exp(s_i - max_i s_i)
    o   = sum_j a_j v_j

evaluated in float64, one query row and one head at a time.

Pins (tests/test_oracle_attention.py): torch's scaled_dot_product_attention
on CPU in float64 with an explicit boolean mask; rows of weights sum to 1
(V = 1 gives O = 1); one visible key gives its value; Q = 0 gives the mean of
the visible values; invariance under a common shift of all positions;
causality; a decode step equals the last row of the equivalent prefill; g = 1
is multi-head attention; a needle placed through a graft is found.
"""
from __future__ import annotations

import numpy as np


def attend_row(q, p: int, K, V, written) -> np.ndarray:
    """One query token: ``q [Hq][D]`` at position ``p`` -> ``o [Hq][D]`` (float64)."""
    q = np.asarray(q, dtype=np.float64)
    Hq, D = q.shape
    Hkv = K.shape[1]
    g = Hq // Hkv
    if not written[:p + 1].all():
        raise ValueError(f"unwritten position below {p}")
    out = np.empty((Hq, D))
    for h in range(Hkv):                      # the g query heads of kv head h
        keys = K[:p + 1, h, :]
        vals = V[:p + 1, h, :]
        s = q[h * g:(h + 1) * g] @ keys.T / np.sqrt(D)          # [g][p + 1]
        e = np.exp(s - s.max(axis=1, keepdims=True))
        a = e / e.sum(axis=1, keepdims=True)
        out[h * g:(h + 1) * g] = a @ vals
    return out


def attend(q, positions, K, V, written) -> np.ndarray:
    """Query tokens ``q [n][Hq][D]`` at ``positions [n]`` -> ``[n][Hq][D]``."""
    q = np.asarray(q, dtype=np.float64)
    return np.stack([attend_row(q[t], int(p), K, V, written) for t, p in enumerate(positions)]) \
        if len(positions) else np.zeros((0,) + q.shape[1:])

