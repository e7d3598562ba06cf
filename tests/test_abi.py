"""The C-ABI library loads on the CPU and exports every symbol include/fcg.h declares."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "fcg.h")


def _declared():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^(?:fcg_status|const char\*)\s+(fcg_\w+)\s*\(", text, re.M)))


def test_header_declares_the_entry_points():
    names = _declared()
    for n in ("fcg_graft", "fcg_patch_prefill", "fcg_decode", "fcg_lib_create", "fcg_cache_create"):
        assert n in names


def test_library_exports_every_declared_symbol():
    from paper_2606_13097_amd import fcg
    lib = ctypes.CDLL(fcg.LIB_PATH)
    missing = [n for n in _declared() if not hasattr(lib, n)]
    assert not missing
    assert sorted(fcg.EXPORTS) == _declared()


def test_status_strings_and_errors_without_gpu():
    from paper_2606_13097_amd import fcg
    for i, name in enumerate(fcg.STATUS):
        assert fcg.fcg_status_string(i) == name
    bad = fcg.model_desc(1, 4, 3, 64, 1e4, "f32")            # 4 % 3 != 0
    with pytest.raises(fcg.FcgError) as e:
        fcg.Cache(bad, 1, 16, flags=fcg.FCG_LAYOUT_ONLY)
    assert e.value.status == fcg.FCG_EINVAL and "multiple" in fcg.fcg_last_error()
    for hd in (32, 96, 256):
        with pytest.raises(fcg.FcgError):
            fcg.Cache(fcg.model_desc(1, 4, 2, hd, 1e4, "bf16"), 1, 16, flags=fcg.FCG_LAYOUT_ONLY)
    with pytest.raises(fcg.FcgError) as e:
        fcg.Cache(fcg.model_desc(1, 4, 2, 64, 1e4, "bf16"), 1, 16, page_size=8, n_pages=4,
                  flags=fcg.FCG_LAYOUT_ONLY)
    assert e.value.status == fcg.FCG_EINVAL
    # value aliasing needs a paged cache, and binds a cache to one library
    desc = fcg.model_desc(1, 4, 2, 64, 1e4, "bf16")
    with pytest.raises(fcg.FcgError) as e:
        fcg.Cache(desc, 1, 16, flags=fcg.FCG_LAYOUT_ONLY | fcg.FCG_ALIAS_V)
    assert e.value.status == fcg.FCG_EINVAL
    c = fcg.Cache(desc, 2, 64, page_size=16, n_pages=8, flags=fcg.FCG_LAYOUT_ONLY | fcg.FCG_ALIAS_V)
    libs = [fcg.Library(desc, 64, 2, flags=fcg.FCG_LAYOUT_ONLY) for _ in range(2)]
    for lib in libs:
        fcg.fcg_lib_add_segment(lib, 32, 0)
    fcg.fcg_graft(c, libs[0], [0], [0], [16])
    assert fcg.fcg_cache_export_v_alias(c, 0).tolist() == [-1, 0, 16, -1]
    with pytest.raises(fcg.FcgError) as e:
        fcg.fcg_graft(c, libs[1], [1], [0], [0])
    assert e.value.status == fcg.FCG_EINVAL and "one library" in fcg.fcg_last_error()
    with pytest.raises(fcg.FcgError) as e:
        fcg.fcg_cache_export_v_alias(c, 2)
    assert e.value.status == fcg.FCG_ERANGE


def test_timing_api_without_device_work():
    from paper_2606_13097_amd import fcg
    c = fcg.Cache(fcg.model_desc(1, 4, 2, 64, 1e4, "f32"), 1, 32, flags=fcg.FCG_LAYOUT_ONLY)
    fcg.fcg_cache_timing(c, True)
    fcg.fcg_patch_prefill(c, 0, [0, 0], [0, 1], None, None, None, None)
    for kind in range(5):
        assert fcg.fcg_cache_timing_read(c, kind) == (0, 0.0)
    with pytest.raises(fcg.FcgError) as e:
        fcg.fcg_cache_timing_read(c, 5)
    assert e.value.status == fcg.FCG_ERANGE
