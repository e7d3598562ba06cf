"""Locality score and residency (Sec. 4.1, Eq. 3; App. B.1, Eq. 8-10): the oracle
pinned by hand-worked values, bounds and limiting weights; the library's native
scorer against the oracle, exactly."""
import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

from oracle.locality import Locality
from paper_2606_13097_amd import fcg


def _hand_example():
    L = Locality(4, window=20, alpha=0.4, beta=0.3, gamma=0.3)
    for t in ([0, 1, 2], [1, 2], [3]):
        L.record(t)
    for f, p in enumerate([10.0, 20.0, 5.0, 40.0]):
        L.set_ppl(f, p)
    return L


def test_components_by_hand():
    L = _hand_example()
    # calls: 0 once, 1 twice, 2 twice, 3 once
    np.testing.assert_array_equal(L.l_freq(), [0.5, 1.0, 1.0, 0.5])
    # 0 is followed by 1 once (of one call); 1 by 2 twice (of two); 2 and 3 end their traces
    np.testing.assert_array_equal(L.l_asso_sum(), [1.0, 1.0, 0.0, 0.0])
    np.testing.assert_array_equal(L.l_sema(), [0.25, 0.5, 0.125, 1.0])
    np.testing.assert_array_equal(L.l_curr(), [0, 0, 0, 1])
    # 0.4*0.5 + 0.3*1 + 0.3*0.25 ; 0.4 + 0.3 + 0.15 ; 0.4 + 0 + 0.0375 ; current -> 1
    np.testing.assert_allclose(L.scores(), [0.575, 0.85, 0.4375, 1.0], rtol=0, atol=1e-15)
    # residency in descending score (3, 1, 0, 2) with costs 5, 4, 3, 2: budget 10 keeps
    # 3 and 1 (9) and fits neither 0 (12) nor 2 (11); budget 12 also fits 0; budget 11
    # skips 0 (12) but fits 2 (11)
    np.testing.assert_array_equal(L.residency(10, [3, 4, 2, 5]), [0, 1, 0, 1])
    np.testing.assert_array_equal(L.residency(12, [3, 4, 2, 5]), [1, 1, 0, 1])
    np.testing.assert_array_equal(L.residency(11, [3, 4, 2, 5]), [0, 1, 1, 1])


def test_perplexity_threshold_and_pinned_entries_by_hand():
    L = _hand_example()          # scores [0.575, 0.85, 0.4375, 1.0], perplexities [10, 20, 5, 40]
    cost = [3, 4, 2, 5]
    # tau = 15: entries 1 and 3 (perplexity >= 15) are placed first, in score order
    # (3, 1), then 0 and 2 (in score order 0, 2) in what remains.  Budget 11: 3 and 1
    # (9), 0 does not fit (12), 2 does (11) -- the plain order gives the same here
    np.testing.assert_array_equal(L.residency(11, cost, tau=15.0), [0, 1, 1, 1])
    # tau = 25: only entry 3 is at or above it; then 1, 0, 2 in score order.  Budget 7:
    # 3 (5) then 1 does not fit (9), 0 does not (8), 2 does (7)
    np.testing.assert_array_equal(L.residency(7, cost, tau=25.0), [0, 0, 1, 1])
    # the same budget without the threshold also keeps 3 then 2
    np.testing.assert_array_equal(L.residency(7, cost), [0, 0, 1, 1])
    # a threshold that reorders: tau = 8 puts 1, 0, 3 (>= 8) before 2; budget 9 keeps 3 (5)
    # and 1 (9) either way, budget 8: 3 (5), 1 does not fit, 0 fits (8), then 2 does not
    np.testing.assert_array_equal(L.residency(8, cost, tau=8.0), [1, 0, 0, 1])
    # without it, 2 (cost 2) comes after 0 (cost 3) in score order as well: same result
    np.testing.assert_array_equal(L.residency(8, cost), [1, 0, 0, 1])
    # tau = 30 with budget 9: only 3 is at or above; then 1 (9); the rest do not fit
    np.testing.assert_array_equal(L.residency(9, cost, tau=30.0), [0, 1, 0, 1])
    # pinned entries stay whatever their score, their cost counted first: pin 2 (cost 2),
    # budget 9: then 3 (7), 1 does not fit (11), 0 does not (10)
    np.testing.assert_array_equal(L.residency(9, cost, pinned=[0, 0, 1, 0]), [0, 0, 1, 1])
    # a pinned set over the budget keeps only the pins
    np.testing.assert_array_equal(L.residency(1, cost, pinned=[1, 1, 0, 0]), [1, 1, 0, 0])


def test_threshold_demotes_low_perplexity_entries():
    """With the budget for one entry, the threshold decides between a high score with a low
    perplexity and a lower score with a high one."""
    L = Locality(2)
    L.record([0, 0, 1])       # 0 is called twice: the higher frequency
    L.record([0])             # 0 is current: score 1
    L.set_ppl(0, 4.0)
    L.set_ppl(1, 30.0)
    assert L.scores()[0] > L.scores()[1]
    np.testing.assert_array_equal(L.residency(1, [1, 1]), [1, 0])
    np.testing.assert_array_equal(L.residency(1, [1, 1], tau=15.0), [0, 1])


def test_window_forgets_old_traces():
    L = Locality(3, window=2)
    L.record([0, 0, 0])
    L.record([1])
    L.record([2, 1])       # the first trace leaves the window
    np.testing.assert_array_equal(L.counts(), [0, 2, 1])
    np.testing.assert_array_equal(L.cooccur()[2], [0, 1, 0])


def test_limits_of_the_weights():
    rng = np.random.default_rng(4)
    traces = [list(rng.integers(0, 6, size=rng.integers(1, 8))) for _ in range(12)]
    for a, b, g, comp in ((1, 0, 0, "l_freq"), (0, 1, 0, "l_asso_sum"), (0, 0, 1, "l_sema")):
        L = Locality(6, 20, a, b, g)
        for t in traces:
            L.record(t)
        for f in range(6):
            L.set_ppl(f, float(f + 1))
        want = getattr(L, comp)()
        cur = L.l_curr()
        np.testing.assert_allclose(L.scores(), np.where(cur > 0, 1.0, want), rtol=0, atol=1e-15)


@settings(max_examples=60, deadline=None)
@given(st.data())
def test_bounds_and_library_parity(data):
    n = data.draw(st.integers(1, 7))
    window = data.draw(st.integers(1, 5))
    w = data.draw(st.sampled_from([(0.4, 0.3, 0.3), (1.0, 0.0, 0.0), (0.2, 0.5, 0.3), (0.0, 0.0, 1.0)]))
    ora = Locality(n, window, *w)
    lib = fcg.Locality(n, window, *w)
    for _ in range(data.draw(st.integers(0, 8))):
        t = data.draw(st.lists(st.integers(0, n - 1), min_size=0, max_size=6))
        ora.record(t)
        fcg.fcg_locality_record(lib, t)
    for f in range(n):
        if data.draw(st.booleans()):
            p = data.draw(st.floats(0, 100, allow_nan=False))
            ora.set_ppl(f, p)
            fcg.fcg_locality_set_ppl(lib, f, p)
    s = ora.scores()
    for comp in (ora.l_freq(), ora.l_asso_sum(), ora.l_sema(), s):
        assert ((comp >= 0) & (comp <= 1)).all()
    np.testing.assert_array_equal(fcg.fcg_locality_scores(lib), s)
    cost = data.draw(st.lists(st.integers(0, 9), min_size=n, max_size=n))
    budget = data.draw(st.integers(0, 30))
    np.testing.assert_array_equal(fcg.fcg_locality_residency(lib, budget, cost), ora.residency(budget, cost))


def test_library_errors():
    with pytest.raises(fcg.FcgError) as e:
        fcg.Locality(3, 20, 0.5, 0.5, 0.5)
    assert e.value.status == fcg.FCG_EINVAL
    lib = fcg.Locality(3)
    with pytest.raises(fcg.FcgError) as e:
        fcg.fcg_locality_record(lib, [0, 3])
    assert e.value.status == fcg.FCG_ERANGE
    with pytest.raises(fcg.FcgError) as e:
        fcg.fcg_locality_set_ppl(lib, 0, -1.0)
    assert e.value.status == fcg.FCG_EINVAL
    with pytest.raises(fcg.FcgError) as e:
        fcg.fcg_locality_residency(lib, -1, [1, 1, 1])
    assert e.value.status == fcg.FCG_EINVAL


def _layout_library(lengths, host_tokens):
    desc = fcg.model_desc(2, 4, 2, 64, 1e4, "f32")
    lib = fcg.Library(desc, int(sum(lengths)), len(lengths), flags=fcg.FCG_LAYOUT_ONLY)
    for n in lengths:
        fcg.fcg_lib_add_segment(lib, int(n), 0)
    fcg.fcg_lib_host_reserve(lib, host_tokens)
    return lib, 2 * 2 * 2 * 64 * 4          # K+V bytes of a token over both layers


@pytest.mark.parametrize("tau", [0.0, 15.0])
def test_library_update_step_follows_the_oracle(tau):
    """fcg_lib_update_residency on a layout-only library (no device memory): after each
    task's trace the resident set equals the oracle's residency of the same scores under
    the same byte budget, and the moves are the differences between consecutive sets."""
    rng = np.random.default_rng(7)
    lengths = rng.integers(20, 200, size=12)
    lib, b_tok = _layout_library(lengths, int(lengths.sum()))
    ora = Locality(12)
    loc = fcg.Locality(12)
    for f in range(12):
        p = float(rng.uniform(2.0, 30.0))
        ora.set_ppl(f, p)
        fcg.fcg_locality_set_ppl(loc, f, p)
    cost = lengths.astype(np.int64) * b_tok
    budget = int(cost.sum() * 0.4)
    state = np.ones(12, dtype=np.uint8)
    moved = [0, 0]
    for t in range(10):
        trace = list(rng.choice(12, size=int(rng.integers(2, 6)), replace=False))
        ora.record(trace)
        fcg.fcg_locality_record(loc, trace)
        n_off, n_re = fcg.fcg_lib_update_residency(lib, loc, budget, tau)
        want = ora.residency(budget, cost, tau=tau)
        got = np.array([fcg.fcg_lib_segment_state(lib, f)[0] for f in range(12)], dtype=np.uint8)
        np.testing.assert_array_equal(got, want)
        assert n_off == int(((state == 1) & (want == 0)).sum()) and n_re == int(((state == 0) & (want == 1)).sum())
        moved[0] += n_off
        moved[1] += n_re
        state = want
    assert moved[0] > 0 and moved[1] > 0
    loc.close()
    lib.close()


def test_library_update_step_errors():
    lib, _ = _layout_library([10, 20], 30)
    loc = fcg.Locality(3)
    with pytest.raises(fcg.FcgError) as e:
        fcg.fcg_lib_update_residency(lib, loc, 100)
    assert e.value.status == fcg.FCG_EINVAL
    loc.close()
    loc = fcg.Locality(2)
    with pytest.raises(fcg.FcgError) as e:
        fcg.fcg_lib_update_residency(lib, loc, 100, -1.0)
    assert e.value.status == fcg.FCG_EINVAL
    # a negative budget takes the default: on a library without device memory, its slabs
    assert fcg.fcg_lib_update_residency(lib, loc, -1) == (0, 0)
    assert fcg.fcg_lib_update_residency(lib, loc, 0) == (2, 0)
    loc.close()
    lib.close()
