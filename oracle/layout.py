"""Placement of grafted segments and fresh tokens in the composite cache (oracle).

The paper composes retrieved function modules as contiguous, order-preserving
token runs (App. B.1, module-level cache reuse; App. C.7: each module keeps
its internal token order) and appends the patch span behind the reused prefix
(Sec. 4.2, Eq. 6).  This module writes out, as plain bookkeeping, where each
token lands, which positions are written, and which requests the boundary
rejects.  Everything here is integer work and must agree with the library bit
for bit.

State of a cache: ``n_seqs`` sequences, each with ``max_tokens`` positions per
layer.  A position is *written* in a layer once a graft (all layers) or an
append (one layer) has stored it.  Contiguous caches put position ``p`` in slot
``p``.  Paged caches use pages of ``page_size`` positions: logical page
``p // page_size`` maps to a physical page of a pool shared by all sequences
(one page table per sequence, shared by all layers), slot ``p % page_size``.

Page assignment (a reading: the paper has no paged cache; any injective map is
valid, this one is fixed so layouts compare bit for bit): within one call,
the logical pages that are touched and not yet mapped are mapped in ascending
``(sequence, logical page)`` order, each to the lowest-numbered free physical
page.  ``reset`` returns a sequence's pages to the free pool; ``truncate``
(cache-patching keeps a prefix) returns the pages past the kept prefix.

Validation (checked in this order; the first failing class is reported):

``EINVAL``   malformed call (negative counts, duplicate sequences in a decode).
``ERANGE``   sequence, segment, layer or position out of range, or a span
             running past ``max_tokens``.
``ESTATE``   decode on a sequence with nothing written in that layer.
``EOVERLAP`` a graft span that meets another span of the call or a position
             written in any layer; a fresh position given twice or already
             written in that layer.
``EHOLE``    attention would read an unwritten position: after the call, some
             position below the largest query position of a sequence (or below
             a decode position) is unwritten in that layer.
``ENOMEM``   the page pool cannot map the new logical pages.

A rejected call changes nothing.

Pins (tests/test_oracle_layout.py): hand-worked placements and page tables on
tiny plans, one test per error class, brute-force enumeration of written sets,
and properties on random plans (spans disjoint, order preserved, deltas).
"""
from __future__ import annotations

import heapq
from typing import Dict, List, Sequence, Tuple

import numpy as np

OK, EINVAL, ERANGE, EOVERLAP, EHOLE, ENOMEM, ESTATE, EHIP = range(8)
STATUS_NAMES = ["OK", "EINVAL", "ERANGE", "EOVERLAP", "EHOLE", "ENOMEM", "ESTATE", "EHIP"]


class FcgError(Exception):
    def __init__(self, code: int, msg: str = ""):
        super().__init__(f"{STATUS_NAMES[code]}: {msg}")
        self.code = code


class Layout:
    def __init__(self, n_layers: int, n_seqs: int, max_tokens: int, page_size: int,
                 n_pages: int, seg_len: Sequence[int], seg_src_pos0: Sequence[int],
                 alias_v: bool = False):
        """``alias_v`` (paged only): a logical page that one grafted segment
        covers entirely takes its values from the library in place; ``v_alias``
        holds the library token of the page's first position (the library
        stores segments back to back, segment g from ``sum(seg_len[:g])``),
        -1 where the page holds its own values."""
        self.n_layers = int(n_layers)
        self.n_seqs = int(n_seqs)
        self.max_tokens = int(max_tokens)
        self.page_size = int(page_size)
        self.n_pages = int(n_pages)
        self.seg_len = [int(x) for x in seg_len]
        self.seg_src_pos0 = [int(x) for x in seg_src_pos0]
        self.written = np.zeros((self.n_seqs, self.n_layers, self.max_tokens), dtype=bool)
        if self.page_size:
            n_lp = -(-self.max_tokens // self.page_size)
            self.page_table = np.full((self.n_seqs, n_lp), -1, dtype=np.int32)
            self._free = list(range(self.n_pages))
            heapq.heapify(self._free)
        else:
            self.page_table = np.zeros((self.n_seqs, 0), dtype=np.int32)
            self._free = []
        self.alias_v = bool(alias_v) and self.page_size > 0
        self.v_alias = np.full(self.page_table.shape, -1, dtype=np.int32)
        self.seg_tok0 = np.concatenate([[0], np.cumsum(self.seg_len)]).astype(np.int64)[:len(self.seg_len)]

    # -- queries ---------------------------------------------------------------
    def seq_len(self, seq: int, layer: int) -> int:
        w = np.flatnonzero(self.written[seq, layer])
        return int(w[-1]) + 1 if w.size else 0

    def slot(self, seq: int, pos: int) -> Tuple[int, int]:
        """(physical page, slot) in paged mode; (-1, pos) in contiguous mode."""
        if not self.page_size:
            return -1, pos
        return int(self.page_table[seq, pos // self.page_size]), pos % self.page_size

    # -- page mapping ----------------------------------------------------------
    def _pages_needed(self, touched: Dict[int, set]) -> List[Tuple[int, int]]:
        need = []
        for seq in sorted(touched):
            for lp in sorted({p // self.page_size for p in touched[seq]}):
                if self.page_table[seq, lp] < 0:
                    need.append((seq, lp))
        return need

    def _map(self, need: List[Tuple[int, int]]) -> None:
        for seq, lp in need:
            self.page_table[seq, lp] = heapq.heappop(self._free)

    def _check_pages(self, touched: Dict[int, set]) -> List[Tuple[int, int]]:
        if not self.page_size:
            return []
        need = self._pages_needed(touched)
        if len(need) > len(self._free):
            raise FcgError(ENOMEM, f"{len(need)} pages needed, {len(self._free)} free")
        return need

    # -- operations ------------------------------------------------------------
    def graft(self, seqs, segs, dsts) -> List[Tuple[int, int, int, int]]:
        """Place segment ``segs[i]`` of the library at ``dsts[i]`` of ``seqs[i]``.

        Returns per item ``(seq, seg, dst, delta)`` with
        ``delta = dst - src_pos0(seg)``, the turn its keys receive.
        """
        seqs, segs, dsts = (list(map(int, a)) for a in (seqs, segs, dsts))
        if not (len(seqs) == len(segs) == len(dsts)):
            raise FcgError(EINVAL, "array lengths differ")
        for s, g, d in zip(seqs, segs, dsts):
            if not (0 <= s < self.n_seqs):
                raise FcgError(ERANGE, f"seq {s}")
            if not (0 <= g < len(self.seg_len)):
                raise FcgError(ERANGE, f"segment {g}")
            if d < 0 or d + self.seg_len[g] > self.max_tokens:
                raise FcgError(ERANGE, f"span [{d}, {d + self.seg_len[g]})")
        touched: Dict[int, set] = {}
        for s, g, d in zip(seqs, segs, dsts):
            span = set(range(d, d + self.seg_len[g]))
            have = touched.setdefault(s, set())
            if have & span:
                raise FcgError(EOVERLAP, f"spans of seq {s} overlap")
            have |= span
        for s, span in touched.items():
            idx = np.fromiter(span, dtype=np.int64)
            if self.written[s][:, idx].any():
                raise FcgError(EOVERLAP, f"seq {s} span meets written positions")
        need = self._check_pages(touched)
        self._map(need)
        for s, g, d in zip(seqs, segs, dsts):
            self.written[s, :, d:d + self.seg_len[g]] = True
            if self.alias_v:
                P = self.page_size
                for lp in range(d // P, (d + self.seg_len[g]) // P):
                    if lp * P >= d:    # the page lies inside the segment's span
                        self.v_alias[s, lp] = self.seg_tok0[g] + lp * P - d
        return [(s, g, d, d - self.seg_src_pos0[g]) for s, g, d in zip(seqs, segs, dsts)]

    def append(self, layer: int, seqs, positions) -> None:
        """Fresh tokens (patch prefill) written at ``positions`` in ``layer``."""
        seqs, positions = list(map(int, seqs)), list(map(int, positions))
        if len(seqs) != len(positions):
            raise FcgError(EINVAL, "array lengths differ")
        if not (0 <= layer < self.n_layers):
            raise FcgError(ERANGE, f"layer {layer}")
        for s, p in zip(seqs, positions):
            if not (0 <= s < self.n_seqs):
                raise FcgError(ERANGE, f"seq {s}")
            if not (0 <= p < self.max_tokens):
                raise FcgError(ERANGE, f"position {p}")
        touched: Dict[int, set] = {}
        for s, p in zip(seqs, positions):
            have = touched.setdefault(s, set())
            if p in have or self.written[s, layer, p]:
                raise FcgError(EOVERLAP, f"seq {s} position {p}")
            have.add(p)
        for s, ps in touched.items():
            top = max(ps)
            w = self.written[s, layer, :top + 1].copy()
            w[list(ps)] = True
            if not w.all():
                raise FcgError(EHOLE, f"seq {s} has unwritten positions below {top}")
        need = self._check_pages(touched)
        self._map(need)
        for s, p in zip(seqs, positions):
            self.written[s, layer, p] = True

    def decode(self, layer: int, seqs) -> List[int]:
        """One decode token per sequence, appended at its current length."""
        seqs = list(map(int, seqs))
        if len(set(seqs)) != len(seqs):
            raise FcgError(EINVAL, "duplicate sequence")
        if not (0 <= layer < self.n_layers):
            raise FcgError(ERANGE, f"layer {layer}")
        for s in seqs:
            if not (0 <= s < self.n_seqs):
                raise FcgError(ERANGE, f"seq {s}")
        pos = [self.seq_len(s, layer) for s in seqs]
        for s, p in zip(seqs, pos):
            if p >= self.max_tokens:
                raise FcgError(ERANGE, f"seq {s} is full")
        for s, p in zip(seqs, pos):
            if p == 0:
                raise FcgError(ESTATE, f"seq {s} is empty in layer {layer}")
        for s, p in zip(seqs, pos):
            if not self.written[s, layer, :p].all():
                raise FcgError(EHOLE, f"seq {s} has a hole below {p}")
        touched = {s: {p} for s, p in zip(seqs, pos)}
        need = self._check_pages(touched)
        self._map(need)
        for s, p in zip(seqs, pos):
            self.written[s, layer, p] = True
        return pos

    def reset(self, seq: int) -> None:
        if not (0 <= seq < self.n_seqs):
            raise FcgError(ERANGE, f"seq {seq}")
        self.written[seq] = False
        self.v_alias[seq] = -1
        if self.page_size:
            for lp in np.flatnonzero(self.page_table[seq] >= 0):
                heapq.heappush(self._free, int(self.page_table[seq, lp]))
            self.page_table[seq] = -1

    def truncate(self, seq: int, pos: int) -> None:
        """Keep only the prefix [0, pos) of a sequence, in every layer.

        For cache-patching the cached states before the faulty span stay and
        only what follows is generated again (Sec. 4.2, Eq. 6; the patch step
        of Alg. 1): the positions from the error span on are forgotten, and
        the pages that hold no kept position return to the pool.
        """
        if not (0 <= seq < self.n_seqs):
            raise FcgError(ERANGE, f"seq {seq}")
        if not (0 <= pos <= self.max_tokens):
            raise FcgError(ERANGE, f"position {pos}")
        self.written[seq, :, pos:] = False
        if self.page_size:
            first = -(-pos // self.page_size)        # first logical page with no kept position
            # a page split by the cut keeps its first rows but takes new
            # tokens after them: it holds its own values from now on
            self.v_alias[seq, pos // self.page_size:] = -1
            for lp in range(first, self.page_table.shape[1]):
                if self.page_table[seq, lp] >= 0:
                    heapq.heappush(self._free, int(self.page_table[seq, lp]))
                    self.page_table[seq, lp] = -1
