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
