"""Helpers of the GPU tests: device reads, oracle references, tolerance checks."""
from __future__ import annotations

import ctypes
import os
import sys

import numpy as np
import torch

from oracle import graft as ograft, numerics, rope, task
from paper_2606_13097_amd import fcg, synth

_hip = None


def _rt():
    global _hip
    if _hip is None:
        _hip = ctypes.CDLL("libamdhip64.so.7")   # the runtime PyTorch already loaded
        _hip.hipMemcpy.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int]
        _hip.hipMemcpy.restype = ctypes.c_int
    return _hip


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def d2h(ptr: int, nbytes: int) -> np.ndarray:
    torch.cuda.synchronize()
    out = np.empty(nbytes, dtype=np.uint8)
    rc = _rt().hipMemcpy(out.ctypes.data, ptr, nbytes, 2)
    assert rc == 0, f"hipMemcpy failed: {rc}"
    return out


def storage_np(t: torch.Tensor) -> np.ndarray:
    t = t.detach().contiguous().cpu()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()


def to_device(a: np.ndarray, dtype: str) -> torch.Tensor:
    if dtype == "bf16":
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()


def read_cache(cache: fcg.Cache, w: synth.Workload, layer: int, seq: int, positions, lib=None) -> tuple:
    """K, V of (layer, seq) at ``positions`` as storage arrays [n][Hkv][D]; with ``lib``, the
    values of pages the cache maps onto that library are read from the library."""
    sh = w.shape
    H, D, es = sh.n_kv_heads, sh.head_dim, sh.elem_bytes
    npdt = np.float32 if sh.dtype == "f32" else np.uint16
    kp, vp = fcg.fcg_cache_device_ptrs(cache, layer)
    positions = np.asarray(positions)
    res = []
    for base in (kp, vp):
        if cache.page_size == 0:
            off = seq * H * cache.max_tokens * D * es
            raw = d2h(base + off, H * cache.max_tokens * D * es).view(npdt).reshape(H, cache.max_tokens, D)
            res.append(np.ascontiguousarray(raw[:, positions].transpose(1, 0, 2)))
        else:
            pt, _, _ = fcg.fcg_cache_export_layout(cache, seq, layer)
            P = cache.page_size
            pool = d2h(base, cache.n_pages * H * P * D * es).view(npdt).reshape(cache.n_pages, H, P, D)
            pages = pt[positions // P]
            assert (pages >= 0).all()
            res.append(np.ascontiguousarray(pool[pages, :, positions % P]))
    if cache.page_size and lib is not None:
        alias = fcg.fcg_cache_export_v_alias(cache, seq)[positions // cache.page_size]
        hit = alias >= 0
        if hit.any():
            cap = lib.capacity
            _, lv = fcg.fcg_lib_device_ptrs(lib, layer)
            slab = d2h(lv, H * cap * D * es).view(npdt).reshape(H, cap, D)
            toks = alias[hit] + positions[hit] % cache.page_size
            res[1][hit] = slab[:, toks].transpose(1, 0, 2)
    return res[0], res[1]


def oracle_items(w: synth.Workload, seq: int, layer: int):
    m = w.graft_seq == seq
    return [(int(d), int(w.lib_src_pos0[g]), synth.lib_segment(w, int(g), layer, "k"),
             synth.lib_segment(w, int(g), layer, "v")) for g, d in zip(w.graft_seg[m], w.graft_dst[m])]


def oracle_run(w: synth.Workload, seq: int, layer: int, n_decode: int, q_mult: float = 1.0):
    """Oracle graft -> prefill -> decode for one sequence and layer, inputs from the host generator."""
    sh = w.shape
    pos, rows = w.fresh_of_seq(seq)
    fq = synth.fresh_tokens(w, seq, layer, "q", rows)
    if q_mult != 1.0:
        fq = scale_storage(fq, q_mult, sh.dtype)
    fk = synth.fresh_tokens(w, seq, layer, "k", rows)
    fv = synth.fresh_tokens(w, seq, layer, "v", rows)
    steps = np.arange(n_decode)
    dq = synth.decode_tokens(w, seq, layer, "q", steps) if n_decode else []
    if n_decode and q_mult != 1.0:
        dq = scale_storage(dq, q_mult, sh.dtype)
    dk = synth.decode_tokens(w, seq, layer, "k", steps) if n_decode else []
    dv = synth.decode_tokens(w, seq, layer, "v", steps) if n_decode else []
    return task.run_layer(sh.n_q_heads, sh.n_kv_heads, sh.head_dim, sh.rope_theta, sh.dtype, w.max_tokens,
                          oracle_items(w, seq, layer), pos, fq, fk, fv, list(dq), list(dk), list(dv))


def scale_storage(x: np.ndarray, mult: float, dtype: str) -> np.ndarray:
    """Multiply storage values by a power of two (exact)."""
    return numerics.encode(numerics.decode(x, dtype) * mult, dtype)


# bf16 keeps 8 significant bits: one round-to-nearest step changes a value x by
# at most U_BF16 * |x|
U_BF16 = 2.0 ** -8
# Roundings on the bf16 attention path whose error scales with the output element:
# its own storage rounding, and one bf16 intermediate (the probabilities of the PV
# product -- when one key dominates, the output is that key's value times its
# rounded weight -- or a bf16 split partial the merge reads).  The first of these
# bounds a single rounding by U_BF16 |o|; the bar admits two.  (The remaining
# roundings of a spread attention average out inside the absolute 2e-2.)
C_ATTN = 2 * U_BF16
ABS_ATTN = 2e-2          # max-abs bar on bf16 attention outputs
FRO_ATTN = 1e-2          # relative Frobenius bar (2e-2 max-abs is vacuous for near-uniform attention)

# Observed errors of every check of the session, printed in pytest's terminal
# summary (tests/conftest.py) so that the margins appear in the log of passing runs.
STATS: list = []


def _record(kind: str, what: str, **fields) -> None:
    test = os.environ.get("PYTEST_CURRENT_TEST", "").split(" ")[0]
    STATS.append(dict(kind=kind, what=what, test=test, **fields))


def check_attn(got_storage: np.ndarray, ref: np.ndarray, dtype: str, what: str) -> dict:
    """fp32: normwise 1e-5 per head.  bf16: per element |got - ref| <= 2e-2 + C_ATTN |ref|,
    and relative Frobenius 1e-2 over the tensor.

    The absolute 2e-2 is the bar on bf16 attention outputs; the per-element term
    covers the roundings that scale with the element itself (C_ATTN), which matter
    once outputs reach magnitudes of several units (x8 outlier channels, peaked
    attention onto one large value).
    """
    got = numerics.decode(got_storage, dtype)
    assert got.shape == ref.shape, (got.shape, ref.shape)
    assert np.isfinite(got).all(), f"{what}: non-finite output"
    if dtype == "f32":
        worst = 0.0
        for h in range(ref.shape[-2]):
            den = np.abs(ref[..., h, :]).max()
            err = np.abs(got[..., h, :] - ref[..., h, :]).max()
            worst = max(worst, err / den if den > 0 else err)
            assert err <= 1e-5 * den, f"{what}: head {h} normwise error {err / den:.3e} > 1e-5"
        _record("attn-f32", what, normwise=worst)
        return {"normwise": worst}
    diff = np.abs(got - ref)
    bar = ABS_ATTN + C_ATTN * np.abs(ref)
    use = float((diff / bar).max()) if diff.size else 0.0
    err = float(diff.max()) if diff.size else 0.0
    fro = float(np.linalg.norm(got - ref) / max(np.linalg.norm(ref), 1e-30))
    # the smallest per-element coefficient this check needed beyond the absolute bar
    need_c = float(np.max((diff - ABS_ATTN) / np.maximum(np.abs(ref), 1e-30), initial=0.0))
    st = {"max_abs": err, "fro": fro, "bar_use": use, "need_c": max(need_c, 0.0),
          "max_ref": float(np.abs(ref).max()) if ref.size else 0.0}
    _record("attn-bf16", what, **st)
    assert use <= 1.0, (f"{what}: |got - ref| exceeds 2e-2 + {C_ATTN:.4g} |ref| (worst element at "
                        f"{use:.3f} of its bar, max-abs {err:.3e})")
    assert fro <= FRO_ATTN, f"{what}: relative Frobenius error {fro:.3e} > {FRO_ATTN}"
    return st


def check_keys(got_storage: np.ndarray, ref_rounded: np.ndarray, dtype: str, what: str) -> None:
    """Grafted / appended keys.

    fp32: normwise 1e-5.  bf16: |got - ref| <= ulp(ref) + 2^-20 * |pair|, per element.  The
    kernel turns a pair (x_i, x_{i+D/2}) in fp32 with fp32 cos/sin: its result is within
    about 2^-22 (|x_i| + |x_{i+D/2}|) of the exact value (cos/sin, product and fma roundings),
    and the pair norm is kept by the turn; rounding that to bf16 can land one bf16 step away
    from the rounding of the exact value.  A component much smaller than its pair can
    therefore differ by more than one of its own ulps; the pair-norm term covers that.
    """
    got = numerics.decode(got_storage, dtype)
    if dtype == "f32":
        den = np.abs(ref_rounded).max()
        err = np.abs(got - ref_rounded).max()
        _record("keys-f32", what, normwise=float(err / den) if den > 0 else float(err))
        assert err <= 1e-5 * den, f"{what}: normwise error {err / den:.3e}"
    else:
        half = ref_rounded.shape[-1] // 2
        pair = np.hypot(ref_rounded[..., :half], ref_rounded[..., half:])
        pair = np.concatenate([pair, pair], axis=-1)
        tol = numerics.ulp(ref_rounded, dtype) + 2.0 ** -20 * pair
        bad = np.abs(got - ref_rounded) > tol
        n_off = int((got != ref_rounded).sum())
        _record("keys-bf16", what, off_rounding=n_off, n=int(got.size), outside_bar=int(bad.sum()))
        assert not bad.any(), f"{what}: {int(bad.sum())} keys outside one ulp + 2^-20 |pair|"
        assert n_off <= 0.01 * got.size, f"{what}: {n_off} of {got.size} keys differ from the oracle's rounding"
