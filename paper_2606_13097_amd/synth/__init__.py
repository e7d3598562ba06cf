"""Seeded synthetic inputs for the grafting hot path (host half).

This module is the only code that both the GPU library's tests and the CPU
oracle's tests rely on.  It holds no arithmetic of the method itself: it
produces workload *plans* (segment lengths, which segments a task grafts and
at which offsets, which positions are fresh) and the *values* of every input
tensor (library K/V, fresh and decode Q/K/V).  The rotary encoding, the
grafting, the attention and every rounding step of the method live on the two
sides separately.

Values
------
Every element is drawn from SplitMix64 (Steele, Lea and Flood, "Fast
splittable pseudorandom number generators", OOPSLA 2014): for a stream key
``k`` the n-th output is ``mix64(k + n * GAMMA)`` with the published
``GAMMA = 0x9E3779B97F4A7C15`` and the published variant-13 finaliser
``mix64``.  The stream key of a seed is ``mix64(seed + GAMMA)``.

An element is addressed by the 61-bit counter
``c = (((tag * 2^8 + layer) * 2^16 + item) * 2^20 + row) * 2^13 + col``
(``col = head * head_dim + dim``).  It takes the three outputs
``n = 4c + 1, 4c + 2, 4c + 3``, splits each into four 16-bit fields and sums
the twelve fields ``h_j``.  The value is the Irwin-Hall approximation of a
standard normal,

    x = (sum_j h_j - 393210) / 65536,

i.e. ``sum_j (h_j + 1/2) / 65536 - 6``: twelve centred uniforms, variance 1
up to 2^-32.  The numerator is an integer below 2^19, so ``x`` is exact in
fp32, and so is ``x * scale`` for the power-of-two scales used here.  The
result is rounded to the storage dtype with round-to-nearest-even (bf16) or
kept (fp32).  A twin of this generator written in HIP
(``synth.hip``) fills large device buffers with the same bits.

Outlier channels (the 34B-class workload) are chosen per
``(layer, kv head, rotary pair i)``: the pair is an outlier when the top 53
bits of ``mix64(key + 4 * c_o * GAMMA)`` with
``c_o = counter(TAG_OUTLIER, layer, 0, head, i)`` fall below
``floor(rate * 2^53)``.  Both dims ``i`` and ``i + D/2`` of an outlier pair,
in K and in V, are multiplied by 8 (exact).

Library keys are drawn directly in their stored (already position-encoded)
form: a rotation of an isotropic Gaussian pair is again isotropic, so the
stored keys have the law of N(0, s^2) keys encoded at positions 0..len-1.

Plans
-----
Plans come from ``numpy.random.default_rng(seed)`` (PCG64).  The five
workloads follow the grafting scenarios of the paper: a task stitches a
system-prompt segment and retrieved function-interface segments (Sec. 4.1,
Eq. 2; Sec. 4.2, Eq. 4) and then prefills a short patch span and decodes
(Sec. 4.2, Eq. 6; App. B.1, fill-in-the-middle of at most 128 tokens).
"""
from __future__ import annotations

import dataclasses
from typing import List, Optional

import numpy as np

__all__ = [
    "GAMMA", "mix64", "stream_key", "counter", "normal_f32", "outlier_pairs",
    "tensor_values", "Shape", "Workload", "TAGS", "workload", "WORKLOADS",
    "bf16_bits_from_f32", "f32_from_bf16_bits",
]

GAMMA = np.uint64(0x9E3779B97F4A7C15)
_M1 = np.uint64(0xBF58476D1CE4E5B9)
_M2 = np.uint64(0x94D049BB133111EB)

# tensor tags of the element counter
TAGS = {
    "lib_k": 0, "lib_v": 1,
    "fresh_q": 2, "fresh_k": 3, "fresh_v": 4,
    "dec_q": 5, "dec_k": 6, "dec_v": 7,
    "outlier": 8,
}

_OUTLIER_FACTOR = 8.0


def mix64(z):
    """SplitMix64 finaliser (variant 13) on uint64 arrays (wrapping)."""
    z = np.asarray(z, dtype=np.uint64)
    with np.errstate(over="ignore"):
        z = (z ^ (z >> np.uint64(30))) * _M1
        z = (z ^ (z >> np.uint64(27))) * _M2
    return z ^ (z >> np.uint64(31))


def stream_key(seed: int) -> np.uint64:
    with np.errstate(over="ignore"):
        return mix64(np.uint64(seed) + GAMMA)[()]


def counter(tag, layer, item, row, col):
    """61-bit element counter; arguments broadcast."""
    tag = np.asarray(tag, dtype=np.uint64)
    layer = np.asarray(layer, dtype=np.uint64)
    item = np.asarray(item, dtype=np.uint64)
    row = np.asarray(row, dtype=np.uint64)
    col = np.asarray(col, dtype=np.uint64)
    for name, v, lim in (("tag", tag, 16), ("layer", layer, 256), ("item", item, 1 << 16),
                         ("row", row, 1 << 20), ("col", col, 1 << 13)):
        if v.size and int(v.max()) >= lim:
            raise ValueError(f"counter field {name} out of range (limit {lim})")
    return ((((tag << np.uint64(8) | layer) << np.uint64(16) | item) << np.uint64(20) | row)
            << np.uint64(13)) | col


def normal_f32(seed: int, c) -> np.ndarray:
    """Irwin-Hall(12) approximately-normal fp32 values for counters ``c``."""
    key = stream_key(seed)
    c = np.asarray(c, dtype=np.uint64)
    acc = np.zeros(c.shape, dtype=np.uint64)
    mask = np.uint64(0xFFFF)
    with np.errstate(over="ignore"):
        base = c * np.uint64(4)
        for j in (1, 2, 3):
            h = mix64(key + (base + np.uint64(j)) * GAMMA)
            acc += (h & mask) + ((h >> np.uint64(16)) & mask) + ((h >> np.uint64(32)) & mask) + (h >> np.uint64(48))
    num = acc.astype(np.int64) - 393210
    return num.astype(np.float32) * np.float32(1.0 / 65536.0)


_OUTLIER_RATE_BITS = 53


def outlier_pairs(seed: int, layer: int, n_heads: int, head_dim: int, rate: float) -> np.ndarray:
    """Boolean [n_heads][head_dim // 2]: rotary pairs scaled by 8."""
    half = head_dim // 2
    if rate <= 0.0:
        return np.zeros((n_heads, half), dtype=bool)
    thresh = np.uint64(int(np.floor(rate * float(1 << _OUTLIER_RATE_BITS))))
    h = np.arange(n_heads, dtype=np.uint64)[:, None]
    i = np.arange(half, dtype=np.uint64)[None, :]
    c = counter(TAGS["outlier"], layer, 0, h, i)
    key = stream_key(seed)
    with np.errstate(over="ignore"):
        d = mix64(key + (c * np.uint64(4)) * GAMMA)
    return (d >> np.uint64(64 - _OUTLIER_RATE_BITS)) < thresh


def bf16_bits_from_f32(x: np.ndarray) -> np.ndarray:
    """Round finite fp32 values to bf16 (nearest, ties to even); uint16 bits."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    lsb = (u >> np.uint64(16)) & np.uint64(1)
    r = (u + np.uint64(0x7FFF) + lsb) >> np.uint64(16)
    return r.astype(np.uint16)


def f32_from_bf16_bits(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def tensor_values(seed: int, tag: str, layer: int, item: int, rows, n_heads: int,
                  head_dim: int, scale: float, dtype: str,
                  outlier_rate: float = 0.0) -> np.ndarray:
    """Values of a ``[len(rows)][n_heads][head_dim]`` tensor slice.

    ``rows`` are the row indices (token index within a segment, token index of
    a fresh span, or decode step).  Returns float32 (``dtype == 'f32'``) or
    uint16 bf16 bits (``dtype == 'bf16'``).
    """
    rows = np.asarray(rows, dtype=np.uint64)
    col = np.arange(n_heads * head_dim, dtype=np.uint64)
    c = counter(TAGS[tag], layer, item, rows[:, None], col[None, :])
    x = normal_f32(seed, c).reshape(len(rows), n_heads, head_dim)
    if scale != 1.0:
        x = x * np.float32(scale)
    if outlier_rate > 0.0 and tag != "fresh_q" and tag != "dec_q":
        m = outlier_pairs(seed, layer, n_heads, head_dim, outlier_rate)
        m = np.concatenate([m, m], axis=1)
        x = np.where(m[None, :, :], x * np.float32(_OUTLIER_FACTOR), x).astype(np.float32)
    if dtype == "f32":
        return np.ascontiguousarray(x, dtype=np.float32)
    if dtype == "bf16":
        return bf16_bits_from_f32(x)
    raise ValueError(f"unknown dtype {dtype!r}")


# ----------------------------------------------------------------------------
# Workload plans
# ----------------------------------------------------------------------------

@dataclasses.dataclass(frozen=True)
class Shape:
    n_layers: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    rope_theta: float
    dtype: str  # "f32" or "bf16"

    @property
    def group(self) -> int:
        return self.n_q_heads // self.n_kv_heads

    @property
    def elem_bytes(self) -> int:
        return 4 if self.dtype == "f32" else 2

    @property
    def token_bytes(self) -> int:
        """K+V bytes of one token over all layers."""
        return 2 * self.n_layers * self.n_kv_heads * self.head_dim * self.elem_bytes


@dataclasses.dataclass
class Workload:
    name: str
    shape: Shape
    seed: int
    lib_lengths: np.ndarray          # int32 [n_lib]
    lib_src_pos0: np.ndarray         # int32 [n_lib]
    kv_scale: float
    q_scale: float
    outlier_rate: float
    n_seqs: int
    page_size: int                   # 0 = contiguous
    max_tokens: int                  # per sequence
    graft_seq: np.ndarray            # int32 [n_items]
    graft_seg: np.ndarray            # int32 [n_items]
    graft_dst: np.ndarray            # int32 [n_items]
    fresh_seq: np.ndarray            # int32 [n_fresh]
    fresh_pos: np.ndarray            # int32 [n_fresh]
    fresh_row: np.ndarray            # int32 [n_fresh] row index of the token within its seq's fresh span
    n_decode: int

    @property
    def n_pages(self) -> int:
        if self.page_size == 0:
            return 0
        per_seq = -(-self.max_tokens // self.page_size)
        return self.n_seqs * per_seq

    def context_tokens(self, seq: int) -> int:
        m = self.graft_seq == seq
        return int(self.lib_lengths[self.graft_seg[m]].sum())

    @property
    def grafted_tokens(self) -> int:
        return int(self.lib_lengths[self.graft_seg].sum())

    def seq_len_after_prefill(self, seq: int) -> int:
        end = 0
        m = self.graft_seq == seq
        if m.any():
            end = int((self.graft_dst[m] + self.lib_lengths[self.graft_seg[m]]).max())
        f = self.fresh_seq == seq
        if f.any():
            end = max(end, int(self.fresh_pos[f].max()) + 1)
        return end

    def fresh_of_seq(self, seq: int):
        m = self.fresh_seq == seq
        return self.fresh_pos[m], self.fresh_row[m]


def _round_up(x: int, m: int) -> int:
    return -(-x // m) * m


def _finish(name, shape, seed, lengths, kv_scale, q_scale, outlier_rate, page_size,
            graft, fresh, n_decode, n_seqs) -> Workload:
    lengths = np.asarray(lengths, dtype=np.int32)
    gs = np.array([g[0] for g in graft], dtype=np.int32)
    gg = np.array([g[1] for g in graft], dtype=np.int32)
    gd = np.array([g[2] for g in graft], dtype=np.int32)
    fs = np.array([f[0] for f in fresh], dtype=np.int32)
    fp = np.array([f[1] for f in fresh], dtype=np.int32)
    fr = np.array([f[2] for f in fresh], dtype=np.int32)
    ends = []
    for s in range(n_seqs):
        e = 0
        m = gs == s
        if m.any():
            e = int((gd[m] + lengths[gg[m]]).max())
        f = fs == s
        if f.any():
            e = max(e, int(fp[f].max()) + 1)
        ends.append(e + n_decode)
    max_tokens = _round_up(max(ends), 64)
    return Workload(name=name, shape=shape, seed=seed, lib_lengths=lengths,
                    lib_src_pos0=np.zeros_like(lengths), kv_scale=kv_scale, q_scale=q_scale,
                    outlier_rate=outlier_rate, n_seqs=n_seqs, page_size=page_size,
                    max_tokens=max_tokens, graft_seq=gs, graft_seg=gg, graft_dst=gd,
                    fresh_seq=fs, fresh_pos=fp, fresh_row=fr, n_decode=n_decode)


def _consecutive_task(seq, seg_ids, lengths, start):
    out, pos = [], start
    for s in seg_ids:
        out.append((seq, int(s), pos))
        pos += int(lengths[s])
    return out, pos


def workload(name: str, seed: int = 1, *, n_layers: Optional[int] = None,
             n_decode: Optional[int] = None, n_lib: Optional[int] = None,
             task: Optional[int] = None) -> Workload:
    """Build one of the named workloads.

    ``tiny``     1 layer, 4/2 heads, D 64, theta 1e4, fp32; 8 segments of 96/128/160
                 tokens plus a 64-token prefix; 3 grafted; 16 patch tokens; 8 decode steps.
    ``7b``       32 layers, 32/8 heads, D 128, theta 1e6, bf16; 256 segments U[200,800]
                 plus a 1024-token system prompt; 6 grafted; 64 patch; 256 decode.
    ``long16k``  as 7b; 256 segments U[400,1200], 2048 prefix, 20 grafted with gaps of
                 U{0..32} fresh tokens before each; 256 patch; 128 decode.
    ``batched``  as 7b; 512 segments U[500,1000], 32 tasks of 8 Zipf(1.1) segments,
                 16-token pages; 32 patch per task; 128 decode.
    ``34b``      48 layers, 64/8 heads, D 128, bf16; 1024 segments U[200,1600]; 4 tasks of
                 24 segments; 512 patch; 64 decode; 1% outlier pairs x8.
    ``n_layers``/``n_decode``/``n_lib`` shrink a workload for tests (same plan law).
    ``task`` redraws which segments are grafted (and the gaps) from a second
    stream while keeping the library of ``seed``: a stream of distinct tasks
    over one resident library.
    """
    rng = np.random.default_rng(seed)

    class _Split:
        """Library draws from the seed's stream; task draws from (seed, task) when given."""

        def __init__(self):
            self.t = np.random.default_rng([seed, task]) if task is not None else rng

        def __getattr__(self, k):
            return getattr(self.t, k)

    trng = _Split()
    if name == "tiny":
        shape = Shape(n_layers or 1, 4, 2, 64, 1e4, "f32")
        nl = n_lib or 8
        lengths = list(rng.choice([96, 128, 160], size=nl))
        lengths.append(64)                       # system-prompt segment
        prefix = nl
        chosen = trng.choice(nl, size=3, replace=False)
        graft, pos = _consecutive_task(0, [prefix] + list(chosen), lengths, 0)
        fresh = [(0, pos + j, j) for j in range(16)]
        return _finish(name, shape, seed, lengths, 1.0, 1.0, 0.0, 0, graft, fresh,
                       8 if n_decode is None else n_decode, 1)
    if name in ("7b", "long16k"):
        shape = Shape(n_layers or 32, 32, 8, 128, 1e6, "bf16")
        nl = n_lib or 256
        if name == "7b":
            lengths = list(rng.integers(200, 800, size=nl, endpoint=True))
            lengths.append(1024)
            chosen = trng.choice(nl, size=6, replace=False)
            graft, pos = _consecutive_task(0, [nl] + list(chosen), lengths, 0)
            fresh = [(0, pos + j, j) for j in range(64)]
            nd = 256
        else:
            lengths = list(rng.integers(400, 1200, size=nl, endpoint=True))
            lengths.append(2048)
            chosen = trng.choice(nl, size=min(20, nl), replace=False)
            graft = [(0, nl, 0)]
            pos, row = 2048, 0
            fresh = []
            for s in chosen:
                gap = int(trng.integers(0, 32, endpoint=True))
                for j in range(gap):
                    fresh.append((0, pos + j, row))
                    row += 1
                pos += gap
                graft.append((0, int(s), pos))
                pos += int(lengths[s])
            for j in range(256):
                fresh.append((0, pos + j, row))
                row += 1
            nd = 128
        return _finish(name, shape, seed, lengths, 0.5, 1.0, 0.0, 0, graft, fresh,
                       nd if n_decode is None else n_decode, 1)
    if name == "batched":
        shape = Shape(n_layers or 32, 32, 8, 128, 1e6, "bf16")
        nl = n_lib or 512
        lengths = list(rng.integers(500, 1000, size=nl, endpoint=True))
        ranks = np.arange(1, nl + 1, dtype=np.float64)
        p = ranks ** -1.1
        p /= p.sum()
        perm = rng.permutation(nl)
        n_tasks = 32
        graft, fresh = [], []
        for t in range(n_tasks):
            chosen = perm[trng.choice(nl, size=8, replace=False, p=p)]
            items, pos = _consecutive_task(t, list(chosen), lengths, 0)
            graft += items
            fresh += [(t, pos + j, j) for j in range(32)]
        return _finish(name, shape, seed, lengths, 0.5, 1.0, 0.0, 16, graft, fresh,
                       128 if n_decode is None else n_decode, n_tasks)
    if name == "34b":
        shape = Shape(n_layers or 48, 64, 8, 128, 1e6, "bf16")
        nl = n_lib or 1024
        lengths = list(rng.integers(200, 1600, size=nl, endpoint=True))
        graft, fresh = [], []
        for t in range(4):
            chosen = trng.choice(nl, size=min(24, nl), replace=False)
            items, pos = _consecutive_task(t, list(chosen), lengths, 0)
            graft += items
            fresh += [(t, pos + j, j) for j in range(512)]
        return _finish(name, shape, seed, lengths, 1.0, 1.0, 0.01, 0, graft, fresh,
                       64 if n_decode is None else n_decode, 4)
    raise ValueError(f"unknown workload {name!r}")


WORKLOADS: List[str] = ["tiny", "7b", "long16k", "batched", "34b"]


def custom(shape: Shape, seed: int, lengths, seq_segments, n_fresh: int, n_decode: int, *,
           page_size: int = 0, kv_scale: float = 0.5, name: str = "custom") -> Workload:
    """A hand-made workload for edge cases: sequence i grafts the segments
    ``seq_segments[i]`` back to back from position 0, then ``n_fresh`` fresh
    tokens follow, then ``n_decode`` decode steps."""
    graft, fresh = [], []
    for seq, segs in enumerate(seq_segments):
        items, pos = _consecutive_task(seq, list(segs), lengths, 0)
        graft += items
        fresh += [(seq, pos + j, j) for j in range(n_fresh)]
    return _finish(name, shape, seed, list(lengths), kv_scale, 1.0, 0.0, page_size, graft, fresh, n_decode,
                   len(seq_segments))


# ----------------------------------------------------------------------------
# Convenience: host values of the tensors a workload feeds the path
# ----------------------------------------------------------------------------

def lib_segment(w: Workload, seg: int, layer: int, which: str) -> np.ndarray:
    """Library K or V of one segment at one layer: [len][Hkv][D] (storage dtype)."""
    sh = w.shape
    n = int(w.lib_lengths[seg])
    return tensor_values(w.seed, "lib_" + which, layer, seg, np.arange(n), sh.n_kv_heads,
                         sh.head_dim, w.kv_scale, sh.dtype, w.outlier_rate)


def fresh_tokens(w: Workload, seq: int, layer: int, which: str, rows) -> np.ndarray:
    """Fresh (patch/gap) q, k or v rows of one sequence at one layer."""
    sh = w.shape
    heads = sh.n_q_heads if which == "q" else sh.n_kv_heads
    scale = w.q_scale if which == "q" else w.kv_scale
    return tensor_values(w.seed, "fresh_" + which, layer, seq, rows, heads, sh.head_dim,
                         scale, sh.dtype, w.outlier_rate)


def decode_tokens(w: Workload, seq: int, layer: int, which: str, steps) -> np.ndarray:
    sh = w.shape
    heads = sh.n_q_heads if which == "q" else sh.n_kv_heads
    scale = w.q_scale if which == "q" else w.kv_scale
    return tensor_values(w.seed, "dec_" + which, layer, seq, steps, heads, sh.head_dim,
                         scale, sh.dtype, w.outlier_rate)
