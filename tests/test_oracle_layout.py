"""Pins of the oracle's placement and validation rules (oracle/layout.py)."""
import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

from oracle.layout import (EHOLE, EINVAL, ENOMEM, EOVERLAP, ERANGE, ESTATE, FcgError, Layout)


def _lay(**kw):
    args = dict(n_layers=2, n_seqs=2, max_tokens=16, page_size=0, n_pages=0,
                seg_len=[3, 5, 2], seg_src_pos0=[0, 0, 4])
    args.update(kw)
    return Layout(**args)


def test_contiguous_placement_by_hand():
    L = _lay()
    res = L.graft([0, 0], [1, 0], [0, 5])
    # seg 1 (5 tokens, source at 0) at 0 -> delta 0; seg 0 (3 tokens) at 5 -> delta 5
    assert res == [(0, 1, 0, 0), (0, 0, 5, 5)]
    assert L.written[0].tolist() == [[True] * 8 + [False] * 8] * 2
    assert not L.written[1].any()
    assert L.seq_len(0, 0) == 8 and L.seq_len(0, 1) == 8
    # seg 2 was captured at source position 4: grafted at 10 it turns by 6
    assert L.graft([1], [2], [10]) == [(1, 2, 10, 6)]
    # fresh tokens at 8, 9 of layer 1 only; decode then appends at the length
    L.append(1, [0, 0], [9, 8])
    assert L.seq_len(0, 1) == 10 and L.seq_len(0, 0) == 8
    assert L.decode(1, [0]) == [10]
    assert L.decode(0, [0]) == [8]
    assert L.slot(0, 7) == (-1, 7)


def test_paged_assignment_by_hand():
    L = _lay(page_size=4, n_pages=6, max_tokens=16)
    # one call: seq 1 gets seg 1 at 2 (positions 2..6, logical pages 0, 1); seq 0 gets seg 0 at 0 (page 0)
    L.graft([1, 0], [1, 0], [2, 0])
    # mapped in ascending (seq, logical page): (0,0)->0, (1,0)->1, (1,1)->2
    assert L.page_table.tolist() == [[0, -1, -1, -1], [1, 2, -1, -1]]
    # seq 0, layer 0: positions 3 (page 0, mapped) and 4 (logical page 1, new) -> physical 3
    L.append(0, [0, 0], [3, 4])
    assert L.page_table[0].tolist() == [0, 3, -1, -1]
    assert L.slot(0, 4) == (3, 0) and L.slot(1, 6) == (2, 2)
    # decode on seq 0 layer 0 appends at 5 (logical page 1, mapped: nothing new)
    assert L.decode(0, [0]) == [5]
    # seq 1 has positions 0, 1 unwritten: decoding it would read a hole
    with pytest.raises(FcgError) as e:
        L.decode(0, [1])
    assert e.value.code == EHOLE
    # releasing seq 1 frees 1 and 2; the next new page takes the lowest free one
    L.reset(1)
    assert L.page_table[1].tolist() == [-1] * 4
    L.graft([1], [2], [8])                      # positions 8, 9 -> logical page 2
    assert L.page_table[1].tolist() == [-1, -1, 1, -1]
    L.graft([0], [2], [12])                     # logical page 3 of seq 0 -> physical 2
    assert L.page_table[0].tolist() == [0, 3, -1, 2]


@pytest.mark.parametrize("call,code", [
    (lambda L: L.graft([0], [0], [0, 1]), EINVAL),
    (lambda L: L.decode(0, [0, 0]), EINVAL),
    (lambda L: L.graft([2], [0], [0]), ERANGE),
    (lambda L: L.graft([0], [3], [0]), ERANGE),
    (lambda L: L.graft([0], [1], [-1]), ERANGE),
    (lambda L: L.graft([0], [1], [12]), ERANGE),          # 12 + 5 > 16
    (lambda L: L.append(2, [0], [0]), ERANGE),
    (lambda L: L.append(0, [0], [16]), ERANGE),
    (lambda L: L.decode(0, [1]), ESTATE),
    (lambda L: L.graft([0, 0], [0, 1], [0, 2]), EOVERLAP),
    (lambda L: L.append(0, [0, 0], [0, 0]), EOVERLAP),
    (lambda L: L.append(0, [0], [1]), EHOLE),             # position 0 unwritten
])
def test_error_classes_on_empty_cache(call, code):
    L = _lay()
    before = (L.written.copy(), L.page_table.copy())
    with pytest.raises(FcgError) as e:
        call(L)
    assert e.value.code == code
    np.testing.assert_array_equal(L.written, before[0])
    np.testing.assert_array_equal(L.page_table, before[1])


def test_error_classes_after_graft():
    L = _lay()
    L.graft([0], [1], [0])                                # 0..4 in both layers
    with pytest.raises(FcgError) as e:
        L.graft([0], [0], [4])                            # meets written position 4
    assert e.value.code == EOVERLAP
    with pytest.raises(FcgError) as e:
        L.append(1, [0], [3])
    assert e.value.code == EOVERLAP
    with pytest.raises(FcgError) as e:
        L.append(0, [0], [6])                             # 5 unwritten
    assert e.value.code == EHOLE
    L.graft([0], [2], [7])                                # 7, 8 written; 5, 6 are a hole
    with pytest.raises(FcgError) as e:
        L.decode(0, [0])
    assert e.value.code == EHOLE
    L.append(0, [0, 0], [5, 6])
    assert L.decode(0, [0]) == [9]


def test_page_pool_exhaustion_changes_nothing():
    L = _lay(page_size=4, n_pages=2)
    L.graft([0], [1], [0])                                # pages 0, 1 (positions 0..4)
    before = L.page_table.copy()
    with pytest.raises(FcgError) as e:
        L.graft([1], [0], [0])
    assert e.value.code == ENOMEM
    np.testing.assert_array_equal(L.page_table, before)
    assert not L.written[1].any()
    L.reset(0)
    L.graft([1], [0], [0])
    assert L.page_table[1, 0] == 0


@settings(max_examples=60, deadline=None)
@given(st.data())
def test_random_plans_against_enumeration(data):
    n_seg = data.draw(st.integers(1, 6))
    seg_len = data.draw(st.lists(st.integers(1, 9), min_size=n_seg, max_size=n_seg))
    src = data.draw(st.lists(st.integers(0, 50), min_size=n_seg, max_size=n_seg))
    page = data.draw(st.sampled_from([0, 4, 16]))
    L = Layout(3, 2, 64, page, 64, seg_len, src)
    occupied = {0: set(), 1: set()}
    pages_used = 0
    for _ in range(data.draw(st.integers(1, 5))):
        seq = data.draw(st.integers(0, 1))
        seg = data.draw(st.integers(0, n_seg - 1))
        dst = data.draw(st.integers(0, 64 - seg_len[seg]))
        span = set(range(dst, dst + seg_len[seg]))
        ok = not (span & occupied[seq])
        try:
            res = L.graft([seq], [seg], [dst])
            assert ok
            assert res == [(seq, seg, dst, dst - src[seg])]
            occupied[seq] |= span
        except FcgError as e:
            assert not ok and e.code == EOVERLAP
    for seq in (0, 1):
        for layer in range(3):
            assert set(np.flatnonzero(L.written[seq, layer]).tolist()) == occupied[seq]
    if page:
        mapped = L.page_table[L.page_table >= 0]
        assert len(set(mapped.tolist())) == len(mapped)            # injective
        # exactly the touched logical pages are mapped, and they use pages 0..k-1
        want = sum(len({p // page for p in occupied[s]}) for s in (0, 1))
        assert len(mapped) == want and sorted(mapped.tolist()) == list(range(want))


def test_truncate_by_hand():
    # page size 4; seq 0 grafted at 0..4 (pages 0, 1), seq 1 at 8..12 (logical pages 2, 3)
    L = _lay(page_size=4, n_pages=8)
    L.graft([0, 1], [1, 1], [0, 8])
    assert L.page_table[0].tolist()[:2] == [0, 1] and L.page_table[1].tolist()[2:4] == [2, 3]
    # keep [0, 3) of seq 0: positions 3, 4 are forgotten in every layer; page 1
    # (positions 4..7) holds nothing kept and is freed, page 0 stays
    L.truncate(0, 3)
    assert not L.written[0, :, 3:].any() and L.written[0, :, :3].all()
    assert L.page_table[0].tolist()[:2] == [0, -1]
    assert L.seq_len(0, 0) == 3
    # the freed page is the lowest free one and is taken first
    L.graft([0], [0], [4])
    assert L.page_table[0, 1] == 1
    # decode after a truncation appends at the cut
    L.truncate(0, 3)
    assert L.decode(1, [0]) == [3]
    assert L.written[0, 1, 3] and not L.written[0, 0, 3]
    # keeping everything changes nothing; keeping nothing frees every page of the sequence
    before = L.written.copy()
    L.truncate(1, L.max_tokens)
    np.testing.assert_array_equal(L.written, before)
    L.truncate(1, 0)
    assert not L.written[1].any() and (L.page_table[1] < 0).all()
    for bad in ((-1, 0), (2, 0), (0, -1), (0, L.max_tokens + 1)):
        with pytest.raises(FcgError) as e:
            L.truncate(*bad)
        assert e.value.code == ERANGE


@settings(max_examples=60, deadline=None)
@given(st.data())
def test_truncate_against_enumeration(data):
    """Grafts and truncations on a random plan, checked against explicit
    position sets: after truncate(s, p) the written set of s is what it was,
    cut at p, in every layer, and a logical page stays mapped iff it was
    mapped and holds a position below p."""
    seg_len = data.draw(st.lists(st.integers(1, 9), min_size=1, max_size=4))
    src = [0] * len(seg_len)
    page = data.draw(st.sampled_from([0, 4, 16]))
    L = Layout(2, 2, 64, page, 64, seg_len, src)
    occupied = {0: set(), 1: set()}
    mapped = {0: set(), 1: set()}
    for _ in range(data.draw(st.integers(1, 8))):
        seq = data.draw(st.integers(0, 1))
        if data.draw(st.booleans()):
            seg = data.draw(st.integers(0, len(seg_len) - 1))
            dst = data.draw(st.integers(0, 64 - seg_len[seg]))
            span = set(range(dst, dst + seg_len[seg]))
            try:
                L.graft([seq], [seg], [dst])
                assert not (span & occupied[seq])
                occupied[seq] |= span
                if page:
                    mapped[seq] |= {p // page for p in span}
            except FcgError as e:
                assert span & occupied[seq] and e.code == EOVERLAP
        else:
            cut = data.draw(st.integers(0, 64))
            L.truncate(seq, cut)
            occupied[seq] = {p for p in occupied[seq] if p < cut}
            if page:
                mapped[seq] = {lp for lp in mapped[seq] if lp * page < cut}
        for s in (0, 1):
            for layer in range(2):
                assert set(np.flatnonzero(L.written[s, layer]).tolist()) == occupied[s]
            if page:
                assert set(np.flatnonzero(L.page_table[s] >= 0).tolist()) == mapped[s]
    if page:
        pages = L.page_table[L.page_table >= 0].tolist()
        assert len(set(pages)) == len(pages)                       # injective


def test_value_aliases_by_hand():
    # segments of 40 and 20 tokens stored back to back in the library (tokens 0.., 40..)
    L = Layout(2, 2, 96, 16, 32, [40, 20], [0, 0], alias_v=True)
    L.graft([0, 0, 1], [0, 1, 0], [8, 48, 16])
    # seq 0: segment 0 at 8..47 covers logical page 1 (16..31) and 2 (32..47) entirely;
    # segment 1 at 48..67 covers page 3 (48..63) and part of page 4
    assert L.v_alias[0].tolist() == [-1, 8, 24, 40, -1, -1]
    # seq 1: segment 0 at 16..55 covers pages 1 and 2; page 3 (48..63) only in part
    assert L.v_alias[1].tolist() == [-1, 0, 16, -1, -1, -1]
    # a cut inside an aliased page takes the page back: it will hold new tokens
    L.truncate(0, 36)
    assert L.v_alias[0].tolist() == [-1, 8, -1, -1, -1, -1]
    # a cut on a page boundary keeps the pages before it as they were
    L.truncate(1, 32)
    assert L.v_alias[1].tolist() == [-1, 0, -1, -1, -1, -1]
    L.reset(1)
    assert (L.v_alias[1] == -1).all()
    # without the flag nothing is aliased
    M = Layout(2, 1, 96, 16, 32, [40, 20], [0, 0])
    M.graft([0], [0], [8])
    assert (M.v_alias == -1).all()


@settings(max_examples=60, deadline=None)
@given(st.data())
def test_value_aliases_against_enumeration(data):
    """A logical page aliases the library exactly when one grafted segment
    covers all 16 of its positions and no cut has split or dropped it; the
    alias then names the library token at the page's first position."""
    seg_len = data.draw(st.lists(st.integers(1, 40), min_size=1, max_size=4))
    tok0 = np.concatenate([[0], np.cumsum(seg_len)])
    L = Layout(1, 1, 128, 16, 64, seg_len, [0] * len(seg_len), alias_v=True)
    want = {}
    for _ in range(data.draw(st.integers(1, 6))):
        if data.draw(st.booleans()):
            g = data.draw(st.integers(0, len(seg_len) - 1))
            d = data.draw(st.integers(0, 128 - seg_len[g]))
            try:
                L.graft([0], [g], [d])
            except FcgError:
                continue
            for lp in range(8):
                if lp * 16 >= d and lp * 16 + 16 <= d + seg_len[g]:
                    want[lp] = int(tok0[g]) + lp * 16 - d
        else:
            cut = data.draw(st.integers(0, 128))
            L.truncate(0, cut)
            want = {lp: a for lp, a in want.items() if lp * 16 + 16 <= cut}
        assert L.v_alias[0].tolist() == [want.get(lp, -1) for lp in range(8)]
