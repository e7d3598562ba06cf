"""Host tier of the segment library (offload / reload, Sec. 4.1 and App. C.5): the
device token allocator against a first-fit model, state errors, and the pins that
value-aliasing caches hold.  Layout-only libraries: no device memory is touched."""
import pytest
from hypothesis import given, settings, strategies as st

from paper_2606_13097_amd import fcg

DESC = fcg.model_desc(1, 4, 2, 64, 1e4, "bf16")


def _lib(cap=64, host=1000, n=16):
    lib = fcg.Library(DESC, cap, n, flags=fcg.FCG_LAYOUT_ONLY)
    if host:
        fcg.fcg_lib_host_reserve(lib, host)
    return lib


class FirstFit:
    """Model of the device token space: freed ranges (coalesced) below a high-water mark."""

    def __init__(self, cap):
        self.cap, self.used, self.free = cap, 0, []

    def alloc(self, n):
        for i, (a, m) in enumerate(self.free):
            if m >= n:
                self.free[i:i + 1] = [(a + n, m - n)] if m > n else []
                return a
        if self.used + n > self.cap:
            return -1
        self.used += n
        return self.used - n

    def release(self, a, n):
        rs = sorted(self.free + [(a, n)])
        merged = []
        for s, m in rs:
            if merged and merged[-1][0] + merged[-1][1] == s:
                merged[-1] = (merged[-1][0], merged[-1][1] + m)
            else:
                merged.append((s, m))
        if merged and merged[-1][0] + merged[-1][1] == self.used:
            self.used = merged.pop()[0]
        self.free = merged


def test_offload_reload_by_hand():
    lib = _lib()
    for n in (10, 20, 5):
        fcg.fcg_lib_add_segment(lib, n, 0)                      # at 0, 10, 30
    fcg.fcg_lib_offload(lib, 1)                                 # frees [10, 30)
    assert fcg.fcg_lib_segment_state(lib, 1) == (False, True)
    assert fcg.fcg_lib_segment_info(lib, 1)[0] == -1
    assert fcg.fcg_lib_add_segment(lib, 15, 0) == 3
    assert fcg.fcg_lib_segment_info(lib, 3)[0] == 10            # first fit; [25, 30) stays free
    fcg.fcg_lib_reload(lib, 1)
    assert fcg.fcg_lib_segment_info(lib, 1)[0] == 35            # 20 tokens fit only past the high-water mark
    fcg.fcg_lib_offload(lib, 1)                                 # the top range returns to the mark
    fcg.fcg_lib_offload(lib, 2)                                 # [30, 35) joins [25, 30) -> back to the mark at 25
    fcg.fcg_lib_reload(lib, 1)
    assert fcg.fcg_lib_segment_info(lib, 1)[0] == 25
    assert fcg.fcg_lib_segment_state(lib, 2) == (False, True)


def test_state_errors():
    lib = _lib(cap=40, host=25)
    for n in (10, 20):
        fcg.fcg_lib_add_segment(lib, n, 0)
    for call, code in ((lambda: fcg.fcg_lib_reload(lib, 0), fcg.FCG_ESTATE),
                       (lambda: fcg.fcg_lib_offload(lib, 2), fcg.FCG_ERANGE),
                       (lambda: fcg.fcg_lib_host_reserve(lib, 10), fcg.FCG_ESTATE)):
        with pytest.raises(fcg.FcgError) as e:
            call()
        assert e.value.status == code
    fcg.fcg_lib_offload(lib, 1)                                 # 20 of 25 host tokens
    with pytest.raises(fcg.FcgError) as e:
        fcg.fcg_lib_offload(lib, 0)                             # 10 more do not fit
    assert e.value.status == fcg.FCG_ENOMEM
    with pytest.raises(fcg.FcgError) as e:
        fcg.fcg_lib_offload(lib, 1)
    assert e.value.status == fcg.FCG_ESTATE
    fcg.fcg_lib_add_segment(lib, 30, 0)                         # takes [10, 40): nothing left for segment 1
    with pytest.raises(fcg.FcgError) as e:
        fcg.fcg_lib_reload(lib, 1)
    assert e.value.status == fcg.FCG_ENOMEM
    # a cache cannot graft an offloaded segment
    cache = fcg.Cache(DESC, 1, 64, flags=fcg.FCG_LAYOUT_ONLY)
    with pytest.raises(fcg.FcgError) as e:
        fcg.fcg_graft(cache, lib, [0], [1], [0])
    assert e.value.status == fcg.FCG_ESTATE
    no_host = _lib(host=0)
    fcg.fcg_lib_add_segment(no_host, 4, 0)
    with pytest.raises(fcg.FcgError) as e:
        fcg.fcg_lib_offload(no_host, 0)
    assert e.value.status == fcg.FCG_ESTATE


def test_alias_caches_pin_segments():
    lib = _lib()
    fcg.fcg_lib_add_segment(lib, 32, 0)
    fcg.fcg_lib_add_segment(lib, 8, 0)
    cache = fcg.Cache(DESC, 2, 64, page_size=16, n_pages=8, flags=fcg.FCG_LAYOUT_ONLY | fcg.FCG_ALIAS_V)
    fcg.fcg_graft(cache, lib, [0, 1], [0, 0], [0, 16])
    for _ in range(2):
        with pytest.raises(fcg.FcgError) as e:
            fcg.fcg_lib_offload(lib, 0)
        assert e.value.status == fcg.FCG_ESTATE and "in place" in fcg.fcg_last_error()
        fcg.fcg_cache_reset(cache, 0)                           # sequence 1 still pins it
    fcg.fcg_cache_reset(cache, 1)
    fcg.fcg_lib_offload(lib, 0)
    fcg.fcg_lib_offload(lib, 1)                                 # never grafted with aliases
    fcg.fcg_lib_reload(lib, 0)
    fcg.fcg_graft(cache, lib, [0], [0], [0])
    cache.close()                                               # destroying the cache unpins
    fcg.fcg_lib_offload(lib, 0)


@settings(max_examples=80, deadline=None)
@given(st.data())
def test_allocator_against_first_fit_model(data):
    cap = data.draw(st.integers(16, 96))
    lib = _lib(cap=cap, host=10_000, n=64)
    model = FirstFit(cap)
    where = {}       # segment -> device offset or -1
    sizes = {}
    for _ in range(data.draw(st.integers(1, 25))):
        op = data.draw(st.sampled_from(["add", "add", "offload", "reload"]))
        if op == "add":
            n = data.draw(st.integers(1, 24))
            at = model.alloc(n)
            try:
                g = fcg.fcg_lib_add_segment(lib, n, 0)
                assert at >= 0
                where[g], sizes[g] = at, n
            except fcg.FcgError as e:
                assert at < 0 and e.status == fcg.FCG_ENOMEM
        elif where:
            g = data.draw(st.sampled_from(sorted(where)))
            if op == "offload" and where[g] >= 0:
                fcg.fcg_lib_offload(lib, g)
                model.release(where[g], sizes[g])
                where[g] = -1
            elif op == "reload" and where[g] < 0:
                at = model.alloc(sizes[g])
                try:
                    fcg.fcg_lib_reload(lib, g)
                    assert at >= 0
                    where[g] = at
                except fcg.FcgError as e:
                    assert at < 0 and e.status == fcg.FCG_ENOMEM
        for g, at in where.items():
            assert fcg.fcg_lib_segment_info(lib, g)[0] == at
    live = sorted((at, at + sizes[g]) for g, at in where.items() if at >= 0)
    assert all(b <= c for (_, b), (c, _) in zip(live, live[1:]))   # disjoint
    assert all(0 <= a and b <= cap for a, b in live)
