"""Set up a synthetic grafting workload on the GPU and drive the hot path.

A ``Workload`` (paper_2606_13097_amd.synth) fixes the model shape, the
segment library and every task's graft / patch / decode plan.  ``GpuSetup``
builds the library in HBM (values written in place by the device twin of the
generator), creates the composite cache, and calls the C ABI:

    fcg_graft  -> fcg_patch_prefill (per layer) -> fcg_decode (per step, per layer)

which is the order of cache-stitching followed by patching and decoding
(Alg. 1 (B); Sec. 4.2, Eq. 4 and Eq. 6).
"""
from __future__ import annotations

from typing import Optional

import numpy as np
import torch

from . import fcg, synth
from .synth import gpu as synth_gpu

TORCH_DTYPE = {"f32": torch.float32, "bf16": torch.bfloat16}


class GpuSetup:
    def __init__(self, w: synth.Workload, device: str = "cuda", n_caches: int = 1, cache_flags: int = 0,
                 lib_spare_tokens: int = 0):
        self.w = w
        sh = w.shape
        self.desc = fcg.model_desc(sh.n_layers, sh.n_q_heads, sh.n_kv_heads, sh.head_dim, sh.rope_theta, sh.dtype)
        self.device = device
        self.tdtype = TORCH_DTYPE[sh.dtype]
        cap = int(w.lib_lengths.sum()) + int(lib_spare_tokens)
        self.lib = fcg.Library(self.desc, cap, len(w.lib_lengths) + (8 if lib_spare_tokens else 0))
        self._fill_library()
        self.caches = [fcg.Cache(self.desc, w.n_seqs, w.max_tokens, w.page_size, w.n_pages, flags=cache_flags)
                       for _ in range(n_caches)]
        self.cache = self.caches[0]

    # -- library ---------------------------------------------------------------
    def _fill_library(self) -> None:
        w, sh = self.w, self.w.shape
        D, H, L = sh.head_dim, sh.n_kv_heads, sh.n_layers
        cap = self.lib.capacity
        k0, v0 = fcg.fcg_lib_device_ptrs(self.lib, 0)
        es = sh.elem_bytes
        for seg, (n, p0) in enumerate(zip(w.lib_lengths, w.lib_src_pos0)):
            sid = fcg.fcg_lib_add_segment(self.lib, int(n), int(p0))
            assert sid == seg
            off, _, _ = fcg.fcg_lib_segment_info(self.lib, sid)
            for which, base in (("k", k0), ("v", v0)):
                synth_gpu.fill(base + off * D * es, sh.dtype, w.seed, "lib_" + which, 0, L, seg, 0, int(n), H, D,
                               H * cap * D, cap * D, D, w.kv_scale, w.outlier_rate)
        torch.cuda.synchronize()

    # -- inputs ----------------------------------------------------------------
    def fresh_inputs(self, layer: int):
        """q [n][Hq][D], k, v [n][Hkv][D] of the plan's fresh tokens (plan order)."""
        w, sh = self.w, self.w.shape
        n = len(w.fresh_pos)
        out = []
        for which, H, scale in (("q", sh.n_q_heads, w.q_scale), ("k", sh.n_kv_heads, w.kv_scale),
                                ("v", sh.n_kv_heads, w.kv_scale)):
            t = torch.empty((n, H, sh.head_dim), dtype=self.tdtype, device=self.device)
            for s in range(w.n_seqs):
                idx = np.flatnonzero(w.fresh_seq == s)
                if idx.size == 0:
                    continue
                # the plan lists a sequence's fresh tokens contiguously, rows 0 .. n_s - 1
                assert np.array_equal(idx, np.arange(idx[0], idx[0] + idx.size))
                assert np.array_equal(w.fresh_row[idx], np.arange(idx.size))
                synth_gpu.fill_rows(t[idx[0]:idx[0] + idx.size], sh.dtype, w.seed, "fresh_" + which, layer, s, 0,
                                    scale, w.outlier_rate)
            out.append(t)
        return out

    def decode_inputs(self, layer: int, n_steps: Optional[int] = None):
        """q [steps][n_seqs][Hq][D], k, v [steps][n_seqs][Hkv][D] for every decode step."""
        w, sh = self.w, self.w.shape
        steps = w.n_decode if n_steps is None else n_steps
        out = []
        for which, H, scale in (("q", sh.n_q_heads, w.q_scale), ("k", sh.n_kv_heads, w.kv_scale),
                                ("v", sh.n_kv_heads, w.kv_scale)):
            t = torch.empty((steps, w.n_seqs, H, sh.head_dim), dtype=self.tdtype, device=self.device)
            D = sh.head_dim
            for s in range(w.n_seqs):
                base = t.data_ptr() + s * H * D * t.element_size()
                synth_gpu.fill(base, sh.dtype, w.seed, "dec_" + which, layer, 1, s, 0, steps, H, D, 0, D,
                               w.n_seqs * H * D, scale, w.outlier_rate)
            out.append(t)
        return out

    # -- hot path --------------------------------------------------------------
    def graft(self, cache: Optional[fcg.Cache] = None, stream=None) -> None:
        w = self.w
        fcg.fcg_graft(cache or self.cache, self.lib, w.graft_seq, w.graft_seg, w.graft_dst, stream)

    def prefill(self, layer: int, q, k, v, out, cache: Optional[fcg.Cache] = None, stream=None) -> None:
        w = self.w
        fcg.fcg_patch_prefill(cache or self.cache, layer, w.fresh_seq, w.fresh_pos, q, k, v, out, stream)

    def decode(self, layer: int, q, k, v, out, cache: Optional[fcg.Cache] = None, stream=None) -> np.ndarray:
        return fcg.fcg_decode(cache or self.cache, layer, np.arange(self.w.n_seqs), q, k, v, out, stream)

    def reset(self, cache: Optional[fcg.Cache] = None) -> None:
        for s in range(self.w.n_seqs):
            fcg.fcg_cache_reset(cache or self.cache, s)

    def close(self) -> None:
        for c in self.caches:
            c.close()
        self.lib.close()
