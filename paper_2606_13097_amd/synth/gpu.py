"""Device half of the seeded input generator: binding of libfcg_synth.so.

``fill`` writes the same bits as ``paper_2606_13097_amd.synth.tensor_values``
into a strided device region; it is how multi-gigabyte segment libraries and
the bench's inputs are created in place.
"""
from __future__ import annotations

import ctypes as C
import os

import torch  # bind to PyTorch's HIP runtime before loading the library

from . import TAGS

_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libfcg_synth.so")
if not os.path.exists(_PATH):
    raise ImportError(f"{_PATH} is not built; run `python -m paper_2606_13097_amd.build`")
_L = C.CDLL(_PATH)
_L.fcg_synth_fill.argtypes = [C.c_void_p, C.c_int, C.c_uint64, C.c_int, C.c_int, C.c_int, C.c_int, C.c_int,
                              C.c_int, C.c_int, C.c_int, C.c_int64, C.c_int64, C.c_int64, C.c_float, C.c_double,
                              C.c_void_p]
_L.fcg_synth_fill.restype = C.c_int


def fill(dst_ptr: int, dtype: str, seed: int, tag: str, layer0: int, n_layers: int, item: int, row0: int,
         n_rows: int, n_heads: int, head_dim: int, stride_layer: int, stride_head: int, stride_row: int,
         scale: float, outlier_rate: float = 0.0, stream=None) -> None:
    """Element (l, r, h, d) -> dst[l*stride_layer + h*stride_head + r*stride_row + d]."""
    if stream is None:
        stream = torch.cuda.current_stream().cuda_stream
    if tag in ("fresh_q", "dec_q"):
        outlier_rate = 0.0          # outlier pairs live in K and V only
    rc = _L.fcg_synth_fill(C.c_void_p(dst_ptr), 0 if dtype == "f32" else 1, seed, TAGS[tag], layer0, n_layers, item,
                           row0, n_rows, n_heads, head_dim, stride_layer, stride_head, stride_row, scale,
                           outlier_rate, C.c_void_p(stream))
    if rc != 0:
        raise RuntimeError(f"fcg_synth_fill failed with HIP error {rc}")


def fill_rows(t: torch.Tensor, dtype: str, seed: int, tag: str, layer: int, item: int, row0: int, scale: float,
              outlier_rate: float = 0.0) -> None:
    """Fill a contiguous ``[n_rows][n_heads][D]`` device tensor with rows row0 .. of (tag, layer, item)."""
    assert t.is_cuda and t.is_contiguous() and t.dim() == 3
    n, H, D = t.shape
    fill(t.data_ptr(), dtype, seed, tag, layer, 1, item, row0, n, H, D, 0, D, H * D, scale, outlier_rate)
