"""The library's host planner (layout-only caches) against the oracle's placement rules, bit for bit."""
import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

from oracle.layout import FcgError as OracleError, Layout
from paper_2606_13097_amd import fcg, synth


def _pair(n_layers, n_seqs, max_tokens, page, n_pages, seg_len, src, alias=False):
    desc = fcg.model_desc(n_layers, 4, 2, 64, 1e4, "f32")
    alias = alias and page > 0
    flags = fcg.FCG_LAYOUT_ONLY | (fcg.FCG_ALIAS_V if alias else 0)
    cache = fcg.Cache(desc, n_seqs, max_tokens, page, n_pages, flags=flags)
    ora = Layout(n_layers, n_seqs, max_tokens, page, n_pages, seg_len, src, alias_v=alias)
    return desc, cache, ora


def _lib(desc, seg_len, src):
    lib = fcg.Library(desc, max(1, sum(seg_len)), max(1, len(seg_len)), flags=fcg.FCG_LAYOUT_ONLY)
    for n, p0 in zip(seg_len, src):
        fcg.fcg_lib_add_segment(lib, n, p0)
    return lib


def _compare(cache, ora, n_seqs, n_layers):
    for s in range(n_seqs):
        for l in range(n_layers):
            pt, n, wr = fcg.fcg_cache_export_layout(cache, s, l)
            np.testing.assert_array_equal(wr.astype(bool), ora.written[s, l])
            assert n == ora.seq_len(s, l)
            if cache.page_size:
                np.testing.assert_array_equal(pt, ora.page_table[s])
                np.testing.assert_array_equal(fcg.fcg_cache_export_v_alias(cache, s), ora.v_alias[s])


def _run_both(fn_c, fn_o):
    try:
        res_o = fn_o()
        code_o = 0
    except OracleError as e:
        res_o, code_o = None, e.code
    try:
        res_c = fn_c()
        code_c = 0
    except fcg.FcgError as e:
        res_c, code_c = None, e.status
    assert code_c == code_o, (code_c, code_o, fcg.fcg_last_error())
    return res_c, res_o


@settings(max_examples=80, deadline=None)
@given(st.data())
def test_append_decode_reset_match_oracle(data):
    n_layers = data.draw(st.integers(1, 3))
    n_seqs = data.draw(st.integers(1, 3))
    page = data.draw(st.sampled_from([0, 16]))
    max_tokens = data.draw(st.integers(1, 80))
    n_pages = data.draw(st.integers(1, 12))
    _, cache, ora = _pair(n_layers, n_seqs, max_tokens, page, n_pages, [], [])
    for _ in range(data.draw(st.integers(1, 12))):
        op = data.draw(st.sampled_from(["append", "append", "decode", "reset", "truncate"]))
        layer = data.draw(st.integers(-1, n_layers))
        if op == "append":
            n = data.draw(st.integers(0, 6))
            seqs = data.draw(st.lists(st.integers(-1, n_seqs), min_size=n, max_size=n))
            base = data.draw(st.integers(0, max_tokens))
            pos = data.draw(st.lists(st.integers(max(0, base - 8) - 1, base + 3), min_size=n, max_size=n))
            _run_both(lambda: fcg.fcg_patch_prefill(cache, layer, seqs, pos, None, None, None, None),
                      lambda: ora.append(layer, seqs, pos))
        elif op == "decode":
            seqs = data.draw(st.lists(st.integers(-1, n_seqs), min_size=0, max_size=3))
            rc, ro = _run_both(lambda: fcg.fcg_decode(cache, layer, seqs, None, None, None, None),
                               lambda: ora.decode(layer, seqs))
            if ro is not None:
                assert list(rc) == list(ro)
        elif op == "reset":
            s = data.draw(st.integers(-1, n_seqs))
            _run_both(lambda: fcg.fcg_cache_reset(cache, s), lambda: ora.reset(s))
        else:
            s = data.draw(st.integers(-1, n_seqs))
            p = data.draw(st.integers(-1, max_tokens + 1))
            _run_both(lambda: fcg.fcg_cache_truncate(cache, s, p), lambda: ora.truncate(s, p))
    _compare(cache, ora, n_seqs, n_layers)


def test_prefill_then_decode_by_hand():
    _, cache, ora = _pair(2, 2, 40, 16, 4, [], [])
    fcg.fcg_patch_prefill(cache, 0, [1, 1, 1], [0, 2, 1], None, None, None, None)
    ora.append(0, [1, 1, 1], [0, 2, 1])
    assert list(fcg.fcg_decode(cache, 0, [1], None, None, None, None)) == [3]
    ora.decode(0, [1])
    _compare(cache, ora, 2, 2)
    pt, n, _ = fcg.fcg_cache_export_layout(cache, 1, 0)
    assert n == 4 and pt[0] == 0 and list(pt[1:]) == [-1, -1]
    with pytest.raises(fcg.FcgError) as e:
        fcg.fcg_decode(cache, 1, [1], None, None, None, None)
    assert e.value.status == fcg.FCG_ESTATE
    with pytest.raises(fcg.FcgError) as e:
        fcg.fcg_patch_prefill(cache, 0, [0], [20], None, None, None, None)
    assert e.value.status == fcg.FCG_EHOLE


@settings(max_examples=80, deadline=None)
@given(st.data())
def test_graft_plans_match_oracle(data):
    n_seg = data.draw(st.integers(1, 6))
    seg_len = data.draw(st.lists(st.integers(1, 40), min_size=n_seg, max_size=n_seg))
    src = data.draw(st.lists(st.integers(0, 100), min_size=n_seg, max_size=n_seg))
    n_layers, n_seqs = data.draw(st.integers(1, 3)), data.draw(st.integers(1, 3))
    page = data.draw(st.sampled_from([0, 16]))
    max_tokens = data.draw(st.integers(8, 160))
    n_pages = data.draw(st.integers(1, 16))
    desc, cache, ora = _pair(n_layers, n_seqs, max_tokens, page, n_pages, seg_len, src, alias=data.draw(st.booleans()))
    lib = _lib(desc, seg_len, src)
    for _ in range(data.draw(st.integers(1, 6))):
        n = data.draw(st.integers(0, 4))
        seqs = data.draw(st.lists(st.integers(-1, n_seqs), min_size=n, max_size=n))
        segs = data.draw(st.lists(st.integers(-1, n_seg), min_size=n, max_size=n))
        dsts = data.draw(st.lists(st.integers(-2, max_tokens), min_size=n, max_size=n))
        _run_both(lambda: fcg.fcg_graft(cache, lib, seqs, segs, dsts), lambda: ora.graft(seqs, segs, dsts))
        if data.draw(st.booleans()):
            layer = data.draw(st.integers(0, n_layers - 1))
            seqs = data.draw(st.lists(st.integers(0, n_seqs - 1), min_size=1, max_size=2))
            rc, ro = _run_both(lambda: fcg.fcg_decode(cache, layer, seqs, None, None, None, None),
                               lambda: ora.decode(layer, seqs))
        if data.draw(st.booleans()):
            s = data.draw(st.integers(0, n_seqs - 1))
            _run_both(lambda: fcg.fcg_cache_reset(cache, s), lambda: ora.reset(s))
        if data.draw(st.booleans()):
            s = data.draw(st.integers(0, n_seqs - 1))
            p = data.draw(st.integers(0, max_tokens))
            _run_both(lambda: fcg.fcg_cache_truncate(cache, s, p), lambda: ora.truncate(s, p))
    _compare(cache, ora, n_seqs, n_layers)


@pytest.mark.parametrize("name", synth.WORKLOADS)
def test_workload_plans_match_oracle(name):
    """Each workload's graft + patch + decode plan, planned by the library and by the oracle."""
    w = synth.workload(name, seed=2, n_layers=2, n_decode=20)
    sh = w.shape
    n_pages = w.n_pages
    desc, cache, ora = _pair(2, w.n_seqs, w.max_tokens, w.page_size, n_pages, list(w.lib_lengths),
                             list(w.lib_src_pos0))
    lib = _lib(desc, list(w.lib_lengths), list(w.lib_src_pos0))
    rc, ro = _run_both(lambda: fcg.fcg_graft(cache, lib, w.graft_seq, w.graft_seg, w.graft_dst),
                       lambda: ora.graft(w.graft_seq, w.graft_seg, w.graft_dst))
    for layer in range(2):
        _run_both(lambda: fcg.fcg_patch_prefill(cache, layer, w.fresh_seq, w.fresh_pos, None, None, None, None),
                  lambda: ora.append(layer, w.fresh_seq, w.fresh_pos))
        for step in range(w.n_decode):
            seqs = list(range(w.n_seqs))
            rc, ro = _run_both(lambda: fcg.fcg_decode(cache, layer, seqs, None, None, None, None),
                               lambda: ora.decode(layer, seqs))
            assert list(rc) == list(ro)
    _compare(cache, ora, w.n_seqs, 2)
    for s in range(w.n_seqs):
        assert ora.seq_len(s, 0) == w.seq_len_after_prefill(s) + w.n_decode
