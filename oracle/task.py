"""One grafting task at one layer, end to end (oracle).

The order is the one of cache-stitching followed by patching and decoding
(Alg. 1 (B), ``stitch`` then ``patch``; Sec. 4.2, Eq. 4 and Eq. 6):

1. graft the retrieved segments into an empty cache (``graft.compose``);
2. store the fresh patch tokens' keys and values at their positions and
   attend each fresh query over every position up to its own
   (``graft.place_fresh``, ``attention.attend``);
3. for every decode step, append one token at the current length and attend
   it over the whole cache;
4. cache-patching (``patch_layer``): keep a prefix of the cache, prefill a new
   span over it and decode after it.

Inputs are storage arrays (fp32 or bf16 bits) exactly as the library receives
them; outputs are float64.
"""
from __future__ import annotations

from typing import Dict, List, Sequence, Tuple

import numpy as np

from . import attention, graft, rope


def run_layer(n_q_heads: int, n_kv_heads: int, head_dim: int, theta: float, dtype: str,
              max_tokens: int,
              items: Sequence[Tuple[int, int, np.ndarray, np.ndarray]],
              fresh_pos, fresh_q, fresh_k, fresh_v,
              dec_q: Sequence[np.ndarray] = (), dec_k: Sequence[np.ndarray] = (),
              dec_v: Sequence[np.ndarray] = ()) -> Dict[str, np.ndarray]:
    """Run graft -> patch prefill -> decode for one sequence at one layer.

    ``items``: ``[(dst, src_pos0, k_lib [len][Hkv][D], v_lib), ...]``.
    ``fresh_*``: positions ``[n]`` and q ``[n][Hq][D]``, k/v ``[n][Hkv][D]``.
    ``dec_*``: one ``[Hq][D]`` / ``[Hkv][D]`` array per step.
    """
    w = rope.inv_freq(head_dim, theta)
    K, V, written = graft.compose(max_tokens, n_kv_heads, head_dim, items, w, dtype)
    out: Dict[str, np.ndarray] = {"K_graft": K.copy(), "V_graft": V.copy(),
                                  "written_graft": written.copy()}
    fresh_pos = np.asarray(fresh_pos, dtype=np.int64)
    if len(fresh_pos):
        graft.place_fresh(K, V, written, fresh_pos, fresh_k, fresh_v, w, dtype)
        q_enc = graft.encode_fresh(fresh_q, fresh_pos, w, dtype)
        out["prefill"] = attention.attend(q_enc, fresh_pos, K, V, written)
    else:
        out["prefill"] = np.zeros((0, n_q_heads, head_dim))
    dec_out: List[np.ndarray] = []
    dec_pos: List[int] = []
    for q, k, v in zip(dec_q, dec_k, dec_v):
        p = int(np.flatnonzero(written)[-1]) + 1
        graft.place_fresh(K, V, written, [p], k[None], v[None], w, dtype)
        q_enc = graft.encode_fresh(q[None], [p], w, dtype)[0]
        dec_out.append(attention.attend_row(q_enc, p, K, V, written))
        dec_pos.append(p)
    out["decode"] = np.stack(dec_out) if dec_out else np.zeros((0, n_q_heads, head_dim))
    out["decode_pos"] = np.asarray(dec_pos, dtype=np.int64)
    out["K"], out["V"], out["written"] = K, V, written
    return out


def patch_layer(state: Dict[str, np.ndarray], n_q_heads: int, head_dim: int, theta: float, dtype: str,
                keep: int, fresh_pos, fresh_q, fresh_k, fresh_v,
                dec_q: Sequence[np.ndarray] = (), dec_k: Sequence[np.ndarray] = (),
                dec_v: Sequence[np.ndarray] = ()) -> Dict[str, np.ndarray]:
    """Cache-patching on the result of ``run_layer`` (Sec. 4.2, Eq. 6; the
    patch step of Alg. 1): keep the prefix [0, keep) of the cache, prefill
    the new span (CoT tokens) at its positions over that prefix, then decode
    after it.  ``state`` is ``run_layer``'s output; its K, V, written arrays
    are not modified."""
    w = rope.inv_freq(head_dim, theta)
    K, V, written = state["K"].copy(), state["V"].copy(), state["written"].copy()
    written[keep:] = False                     # forget the error span and everything after it
    fresh_pos = np.asarray(fresh_pos, dtype=np.int64)
    out: Dict[str, np.ndarray] = {}
    graft.place_fresh(K, V, written, fresh_pos, fresh_k, fresh_v, w, dtype)
    out["prefill"] = attention.attend(graft.encode_fresh(fresh_q, fresh_pos, w, dtype), fresh_pos, K, V, written)
    dec_out: List[np.ndarray] = []
    for q, k, v in zip(dec_q, dec_k, dec_v):
        p = int(np.flatnonzero(written)[-1]) + 1
        graft.place_fresh(K, V, written, [p], k[None], v[None], w, dtype)
        dec_out.append(attention.attend_row(graft.encode_fresh(q[None], [p], w, dtype)[0], p, K, V, written))
    out["decode"] = np.stack(dec_out) if dec_out else np.zeros((0, n_q_heads, head_dim))
    out["K"], out["V"], out["written"] = K, V, written
    return out
