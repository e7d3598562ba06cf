"""The composite (grafted) cache of one sequence at one layer (oracle).

Cache-stitching injects the KV states of the retrieved function interfaces,
concatenated, as context of the generation (Sec. 4.2, Eq. 4); each entry of
the two-tier cache holds the KV states of one function (Sec. 4.1, Eq. 2).
Here a library segment ``s`` of ``len_s`` tokens, stored encoded at source
positions ``src_pos0_s .. src_pos0_s + len_s - 1``, is grafted at offset
``o_s``: token ``j`` lands at position ``o_s + j``, its key turned by
``delta_s = o_s - src_pos0_s`` and rounded to the storage dtype, its value
copied bit for bit.  Fresh (patch) tokens at position ``p`` store their key
encoded at ``p`` (rounded) and their value as given.  The cached segments are
never recomputed (Sec. 4.2, Eq. 6 reuses the prefix KV states as they are).

All arithmetic is float64; results are storage-rounded float64 arrays.

Pins (tests/test_oracle_graft.py): grafting segments cut from one encoded
source sequence back at their original offsets reproduces that sequence
exactly; a graft by delta equals encoding the pre-encoding keys at the target
position (<= 1e-12 before rounding); graft by d1 then d2 equals graft by
d1 + d2; values are copied exactly; per-pair norms are kept.
"""
from __future__ import annotations

from typing import Iterable, Tuple

import numpy as np

from . import numerics, rope


def graft_keys(k_lib, delta: int, w, dtype: str) -> np.ndarray:
    """Keys of one segment ``[len][Hkv][D]`` turned by ``delta`` and rounded."""
    x = numerics.decode(k_lib, dtype)
    return numerics.round_to(rope.rotate(x, delta, w), dtype)


def graft_values(v_lib, dtype: str) -> np.ndarray:
    return numerics.decode(v_lib, dtype)


def encode_fresh(x, positions, w, dtype: str) -> np.ndarray:
    """Rotary-encode fresh query or key rows ``[n][H][D]`` at their positions."""
    v = numerics.decode(x, dtype)
    pos = np.asarray(positions, dtype=np.float64).reshape(-1, 1)
    return numerics.round_to(rope.rotate(v, pos, w), dtype)


def compose(max_tokens: int, n_kv_heads: int, head_dim: int,
            items: Iterable[Tuple[int, int, np.ndarray, np.ndarray]], w, dtype: str):
    """Graft ``items = [(dst, src_pos0, k_lib, v_lib), ...]`` into an empty cache.

    Returns ``(K, V, written)`` with ``K, V`` float64 ``[max_tokens][Hkv][D]``.
    """
    K = np.zeros((max_tokens, n_kv_heads, head_dim))
    V = np.zeros((max_tokens, n_kv_heads, head_dim))
    written = np.zeros(max_tokens, dtype=bool)
    for dst, src_pos0, k_lib, v_lib in items:
        n = k_lib.shape[0]
        if written[dst:dst + n].any():
            raise ValueError("overlapping spans")
        K[dst:dst + n] = graft_keys(k_lib, dst - src_pos0, w, dtype)
        V[dst:dst + n] = graft_values(v_lib, dtype)
        written[dst:dst + n] = True
    return K, V, written


def place_fresh(K, V, written, positions, k, v, w, dtype: str) -> None:
    """Store fresh keys (encoded at their positions) and values, in place."""
    positions = np.asarray(positions, dtype=np.int64)
    if written[positions].any():
        raise ValueError("position already written")
    K[positions] = encode_fresh(k, positions, w, dtype)
    V[positions] = numerics.decode(v, dtype)
    written[positions] = True
