"""Thin Python binding of libfcg.so (C ABI in include/fcg.h).

Argument marshalling only: every step of the grafting path runs in the HIP
kernels of libfcg.so.  Functions carry the C names.  Device tensors are torch
tensors on the GPU (only their ``data_ptr`` is passed); host index arrays are
anything ``numpy.asarray(..., int32)`` accepts.  A failing call raises
``FcgError`` with the status and the library's message.

If libfcg.so is missing this module raises at import: there is no fallback.
"""
from __future__ import annotations

import ctypes as C
import os
from typing import Optional, Sequence

import numpy as np
# PyTorch ships its own libamdhip64 (soname libamdhip64.so.7).  Loading torch
# first makes the dynamic linker bind libfcg.so to that same runtime, so
# torch's streams and allocations and libfcg's kernels share one HIP runtime.
import torch  # noqa: F401

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libfcg.so")

FCG_F32, FCG_BF16 = 0, 1
FCG_LAYOUT_ONLY = 1
FCG_ALIAS_V = 2
STATUS = ["FCG_OK", "FCG_EINVAL", "FCG_ERANGE", "FCG_EOVERLAP", "FCG_EHOLE", "FCG_ENOMEM", "FCG_ESTATE",
          "FCG_EHIP"]
FCG_OK, FCG_EINVAL, FCG_ERANGE, FCG_EOVERLAP, FCG_EHOLE, FCG_ENOMEM, FCG_ESTATE, FCG_EHIP = range(8)

# every symbol include/fcg.h declares
EXPORTS = [
    "fcg_lib_create", "fcg_lib_add_segment", "fcg_lib_segment_info", "fcg_lib_device_ptrs", "fcg_lib_destroy",
    "fcg_lib_host_reserve", "fcg_lib_offload", "fcg_lib_reload", "fcg_lib_segment_state", "fcg_lib_update_residency",
    "fcg_cache_create", "fcg_cache_reset", "fcg_cache_truncate", "fcg_cache_export_layout", "fcg_cache_export_v_alias",
    "fcg_cache_device_ptrs",
    "fcg_cache_destroy", "fcg_graft", "fcg_patch_prefill", "fcg_decode", "fcg_decode_noalloc", "fcg_status_string",
    "fcg_last_error",
    "fcg_cache_timing", "fcg_cache_timing_read",
    "fcg_locality_create", "fcg_locality_record", "fcg_locality_set_ppl", "fcg_locality_scores",
    "fcg_locality_residency", "fcg_locality_destroy",
]
FCG_TIME_GRAFT, FCG_TIME_PREFILL_ATTN, FCG_TIME_PREFILL, FCG_TIME_DECODE, FCG_TIME_DECODE_ATTN = range(5)


class FcgError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{STATUS[status] if 0 <= status < len(STATUS) else status}: {msg}")
        self.status = status


class ModelDesc(C.Structure):
    _fields_ = [("n_layers", C.c_int32), ("n_q_heads", C.c_int32), ("n_kv_heads", C.c_int32),
                ("head_dim", C.c_int32), ("rope_theta", C.c_double), ("dtype", C.c_int32),
                ("rope_style", C.c_int32)]


def model_desc(n_layers, n_q_heads, n_kv_heads, head_dim, rope_theta, dtype) -> ModelDesc:
    dt = {"f32": FCG_F32, "bf16": FCG_BF16}.get(dtype, dtype)
    return ModelDesc(n_layers, n_q_heads, n_kv_heads, head_dim, float(rope_theta), int(dt), 0)


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run `python -m paper_2606_13097_amd.build`")
    lib = C.CDLL(LIB_PATH)
    P, I32, I64, U32 = C.c_void_p, C.c_int32, C.c_int64, C.c_uint32
    PI32, PI64 = C.POINTER(C.c_int32), C.POINTER(C.c_int64)
    sig = {
        "fcg_lib_create": [C.POINTER(ModelDesc), I64, I32, U32, C.POINTER(P)],
        "fcg_lib_add_segment": [P, I32, I32, P, P, P, PI32],
        "fcg_lib_segment_info": [P, I32, PI64, PI32, PI32],
        "fcg_lib_device_ptrs": [P, I32, C.POINTER(P), C.POINTER(P)],
        "fcg_lib_destroy": [P],
        "fcg_lib_host_reserve": [P, I64],
        "fcg_lib_offload": [P, I32, P],
        "fcg_lib_reload": [P, I32, P],
        "fcg_lib_segment_state": [P, I32, PI32, PI32],
        "fcg_lib_update_residency": [P, P, I64, C.c_double, P, PI32, PI32],
        "fcg_cache_create": [C.POINTER(ModelDesc), I32, I32, I32, I32, U32, C.POINTER(P)],
        "fcg_cache_reset": [P, I32],
        "fcg_cache_truncate": [P, I32, I32, P],
        "fcg_cache_export_v_alias": [P, I32, P],
        "fcg_cache_export_layout": [P, I32, I32, P, PI32, P],
        "fcg_cache_device_ptrs": [P, I32, C.POINTER(P), C.POINTER(P)],
        "fcg_cache_destroy": [P],
        # int32 arrays go as plain addresses (ndarray.ctypes.data): no pointer objects per call
        "fcg_graft": [P, P, I32, P, P, P, P],
        "fcg_patch_prefill": [P, I32, I32, P, P, P, P, P, P, P],
        "fcg_decode": [P, I32, I32, P, P, P, P, P, P, P],
        "fcg_decode_noalloc": [P, I32, I32, P, P, P, P, P, P, P],
        "fcg_cache_timing": [P, I32],
        "fcg_cache_timing_read": [P, I32, PI32, C.POINTER(C.c_double)],
        "fcg_locality_create": [I32, I32, C.c_double, C.c_double, C.c_double, C.POINTER(P)],
        "fcg_locality_record": [P, I32, P],
        "fcg_locality_set_ppl": [P, I32, C.c_double],
        "fcg_locality_scores": [P, P],
        "fcg_locality_residency": [P, I64, P, P],
        "fcg_locality_destroy": [P],
    }
    for name, args in sig.items():
        f = getattr(lib, name)
        f.argtypes = args
        f.restype = C.c_int
    lib.fcg_status_string.argtypes = [C.c_int]
    lib.fcg_status_string.restype = C.c_char_p
    lib.fcg_last_error.argtypes = []
    lib.fcg_last_error.restype = C.c_char_p
    return lib


_L = _load()


def _check(status: int) -> None:
    if status != FCG_OK:
        raise FcgError(status, _L.fcg_last_error().decode())


def _i32(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a, dtype=np.int32))


def _p(a: np.ndarray):
    return a.ctypes.data if a.size else None


_SMALL = 64  # int32 arrays up to this length go as ctypes arrays


def _i32_small(a):
    """An int32 array argument as (ctypes array or None, length).  Building a small
    ctypes array costs well under a microsecond; an ndarray's ``.ctypes.data``
    costs about two, and a decode call passes two such arrays."""
    vals = a.tolist() if isinstance(a, np.ndarray) else [int(x) for x in a]
    n = len(vals)
    return ((C.c_int32 * n)(*vals) if n else None), n


def _dptr(t) -> Optional[int]:
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _current_stream() -> Optional[int]:
    """Raw handle of torch's current stream on the current device (None without a GPU)."""
    import torch
    if not torch.cuda.is_available():
        return None
    raw = getattr(torch._C, "_cuda_getCurrentRawStream", None)   # no Stream object per call
    if raw is not None:
        return raw(torch.cuda.current_device())
    return torch.cuda.current_stream().cuda_stream


def _stream(stream) -> Optional[int]:
    if stream is None:
        return _current_stream()
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


class Library:
    """Handle of a segment library (``fcg_lib``)."""

    h = None

    def __init__(self, desc: ModelDesc, capacity_tokens: int, max_segments: int, flags: int = 0):
        h = C.c_void_p()
        _check(_L.fcg_lib_create(C.byref(desc), int(capacity_tokens), int(max_segments), int(flags), C.byref(h)))
        self.h, self.desc = h, desc
        self._lib = _L   # kept for close(), which may run while the interpreter tears down globals
        self.capacity = int(capacity_tokens)

    def close(self):
        if self.h:
            self._lib.fcg_lib_destroy(self.h)
            self.h = None

    __del__ = close


class Cache:
    """Handle of a composite cache (``fcg_cache``)."""

    h = None

    def __init__(self, desc: ModelDesc, n_seqs: int, max_tokens: int, page_size: int = 0, n_pages: int = 0,
                 flags: int = 0):
        h = C.c_void_p()
        _check(_L.fcg_cache_create(C.byref(desc), int(n_seqs), int(max_tokens), int(page_size), int(n_pages),
                                   int(flags), C.byref(h)))
        self.h, self.desc = h, desc
        self._lib = _L   # kept for close(), which may run while the interpreter tears down globals
        self.n_seqs, self.max_tokens, self.page_size, self.n_pages = n_seqs, max_tokens, page_size, n_pages
        self.n_lp = -(-max_tokens // page_size) if page_size else 0

    def close(self):
        if self.h:
            self._lib.fcg_cache_destroy(self.h)
            self.h = None

    __del__ = close


def fcg_lib_create(desc: ModelDesc, capacity_tokens: int, max_segments: int, flags: int = 0) -> Library:
    return Library(desc, capacity_tokens, max_segments, flags)


def fcg_lib_add_segment(lib: Library, length: int, src_pos0: int, k=None, v=None, stream=None) -> int:
    sid = C.c_int32()
    _check(_L.fcg_lib_add_segment(lib.h, int(length), int(src_pos0), _dptr(k), _dptr(v),
                                  _stream(stream) if k is not None else None, C.byref(sid)))
    return sid.value


def fcg_lib_segment_info(lib: Library, seg_id: int):
    off, n, src = C.c_int64(), C.c_int32(), C.c_int32()
    _check(_L.fcg_lib_segment_info(lib.h, int(seg_id), C.byref(off), C.byref(n), C.byref(src)))
    return off.value, n.value, src.value


def fcg_lib_device_ptrs(lib: Library, layer: int):
    k, v = C.c_void_p(), C.c_void_p()
    _check(_L.fcg_lib_device_ptrs(lib.h, int(layer), C.byref(k), C.byref(v)))
    return k.value, v.value


def fcg_lib_destroy(lib: Library) -> None:
    lib.close()


def fcg_lib_host_reserve(lib: Library, host_tokens: int) -> None:
    _check(_L.fcg_lib_host_reserve(lib.h, int(host_tokens)))


def fcg_lib_offload(lib: Library, seg: int, stream=None) -> None:
    _check(_L.fcg_lib_offload(lib.h, int(seg), _stream(stream)))


def fcg_lib_reload(lib: Library, seg: int, stream=None) -> None:
    _check(_L.fcg_lib_reload(lib.h, int(seg), _stream(stream)))


def fcg_lib_segment_state(lib: Library, seg: int):
    """-> (in device memory, has a host copy)."""
    a, b = C.c_int32(), C.c_int32()
    _check(_L.fcg_lib_segment_state(lib.h, int(seg), C.byref(a), C.byref(b)))
    return bool(a.value), bool(b.value)


def fcg_lib_update_residency(lib: Library, loc: "Locality", budget_bytes: int = -1, ppl_threshold: float = 0.0,
                             stream=None):
    """The update step: offload / reload segments by locality under a byte budget -> (offloaded, reloaded)."""
    a, b = C.c_int32(), C.c_int32()
    _check(_L.fcg_lib_update_residency(lib.h, loc.h, int(budget_bytes), float(ppl_threshold),
                                       _stream(stream), C.byref(a), C.byref(b)))
    return a.value, b.value


def fcg_cache_create(desc: ModelDesc, n_seqs: int, max_tokens: int, page_size: int = 0, n_pages: int = 0,
                     flags: int = 0) -> Cache:
    return Cache(desc, n_seqs, max_tokens, page_size, n_pages, flags)


def fcg_cache_reset(cache: Cache, seq: int) -> None:
    _check(_L.fcg_cache_reset(cache.h, int(seq)))


def fcg_cache_truncate(cache: Cache, seq: int, pos: int, stream=None) -> None:
    """Keep positions [0, pos) of ``seq`` in every layer (cache-patching reuses that prefix)."""
    _check(_L.fcg_cache_truncate(cache.h, int(seq), int(pos), _stream(stream)))


def fcg_cache_export_v_alias(cache: Cache, seq: int) -> np.ndarray:
    """-> int32 [n_lp]: library token of each logical page's first position, -1 = own values."""
    out = np.zeros(max(cache.n_lp, 1), dtype=np.int32)
    _check(_L.fcg_cache_export_v_alias(cache.h, int(seq), out.ctypes.data))
    return out[:cache.n_lp]


def fcg_cache_export_layout(cache: Cache, seq: int, layer: int):
    """-> (page_table int32 [n_lp] or None, seq_len, written uint8 [max_tokens])."""
    pt = np.zeros(max(cache.n_lp, 1), dtype=np.int32)
    n = C.c_int32()
    wr = np.zeros(cache.max_tokens, dtype=np.uint8)
    _check(_L.fcg_cache_export_layout(cache.h, int(seq), int(layer), _p(pt) if cache.page_size else None,
                                      C.byref(n), wr.ctypes.data))
    return (pt[:cache.n_lp] if cache.page_size else None), n.value, wr


def fcg_cache_device_ptrs(cache: Cache, layer: int):
    k, v = C.c_void_p(), C.c_void_p()
    _check(_L.fcg_cache_device_ptrs(cache.h, int(layer), C.byref(k), C.byref(v)))
    return k.value, v.value


def fcg_cache_destroy(cache: Cache) -> None:
    cache.close()


def fcg_graft(cache: Cache, lib: Library, seq: Sequence[int], seg: Sequence[int], dst: Sequence[int],
              stream=None) -> None:
    s, g, d = _i32(seq), _i32(seg), _i32(dst)
    if not (s.size == g.size == d.size):
        raise ValueError("seq, seg and dst differ in length")
    _check(_L.fcg_graft(cache.h, lib.h, int(s.size), _p(s), _p(g), _p(d), _stream(stream)))


def fcg_patch_prefill(cache: Cache, layer: int, seq, pos, q, k, v, out, stream=None) -> None:
    s, p = _i32(seq), _i32(pos)
    if s.size != p.size:
        raise ValueError("seq and pos differ in length")
    _check(_L.fcg_patch_prefill(cache.h, int(layer), int(s.size), _p(s), _p(p), _dptr(q), _dptr(k), _dptr(v),
                                _dptr(out), _stream(stream) if q is not None else None))


def _decode_call(fn, cache: Cache, layer: int, seqs, q, k, v, out, stream) -> np.ndarray:
    if len(seqs) > _SMALL:
        s = _i32(seqs)
        pos = np.zeros(max(s.size, 1), dtype=np.int32)
        _check(fn(cache.h, int(layer), int(s.size), _p(s), _dptr(q), _dptr(k), _dptr(v), _dptr(out), pos.ctypes.data,
                  _stream(stream) if q is not None else None))
        return pos[:s.size]
    # one step of a small batch: the per-call marshalling is a visible part of the step
    s, n = _i32_small(seqs)
    pos = (C.c_int32 * max(n, 1))()
    _check(fn(cache.h, int(layer), n, s, _dptr(q), _dptr(k), _dptr(v), _dptr(out), pos,
              _stream(stream) if q is not None else None))
    return np.frombuffer(pos, dtype=np.int32, count=n)


def fcg_decode(cache: Cache, layer: int, seqs, q, k, v, out, stream=None) -> np.ndarray:
    return _decode_call(_L.fcg_decode, cache, layer, seqs, q, k, v, out, stream)


def fcg_decode_noalloc(cache: Cache, layer: int, seqs, q, k, v, out, stream=None) -> np.ndarray:
    """fcg_decode through the entry point that allocates nothing (static device scratch)."""
    return _decode_call(_L.fcg_decode_noalloc, cache, layer, seqs, q, k, v, out, stream)


def fcg_cache_timing(cache: Cache, enable: bool) -> None:
    _check(_L.fcg_cache_timing(cache.h, int(bool(enable))))


def fcg_cache_timing_read(cache: Cache, kind: int):
    """-> (number of recorded intervals, their summed duration in ms)."""
    n, ms = C.c_int32(), C.c_double()
    _check(_L.fcg_cache_timing_read(cache.h, int(kind), C.byref(n), C.byref(ms)))
    return n.value, ms.value


class Locality:
    """Handle of a locality scorer (``fcg_locality``)."""

    h = None

    def __init__(self, n_funcs: int, window: int = 20, alpha: float = 0.4, beta: float = 0.3, gamma: float = 0.3):
        h = C.c_void_p()
        _check(_L.fcg_locality_create(int(n_funcs), int(window), float(alpha), float(beta), float(gamma),
                                      C.byref(h)))
        self.h, self.n_funcs = h, int(n_funcs)
        self._lib = _L

    def close(self):
        if self.h:
            self._lib.fcg_locality_destroy(self.h)
            self.h = None

    __del__ = close


def fcg_locality_record(loc: Locality, func_ids) -> None:
    a = np.ascontiguousarray(func_ids, dtype=np.int32)
    _check(_L.fcg_locality_record(loc.h, len(a), a.ctypes.data if len(a) else None))


def fcg_locality_set_ppl(loc: Locality, func: int, ppl: float) -> None:
    _check(_L.fcg_locality_set_ppl(loc.h, int(func), float(ppl)))


def fcg_locality_scores(loc: Locality) -> np.ndarray:
    out = np.zeros(loc.n_funcs, dtype=np.float64)
    _check(_L.fcg_locality_scores(loc.h, out.ctypes.data))
    return out


def fcg_locality_residency(loc: Locality, budget: int, cost) -> np.ndarray:
    c = np.ascontiguousarray(cost, dtype=np.int64)
    if len(c) != loc.n_funcs:
        raise ValueError("one cost per function")
    out = np.zeros(loc.n_funcs, dtype=np.uint8)
    _check(_L.fcg_locality_residency(loc.h, int(budget), c.ctypes.data, out.ctypes.data))
    return out


def fcg_status_string(status: int) -> str:
    return _L.fcg_status_string(int(status)).decode()


def fcg_last_error() -> str:
    return _L.fcg_last_error().decode()
