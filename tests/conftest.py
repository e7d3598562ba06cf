import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) and the built HIP library")
    config.addinivalue_line("markers", "slow: long CPU test (full-size sampled parity)")


def pytest_terminal_summary(terminalreporter, exitstatus, config):
    """Observed parity errors of the GPU tests, per test: the margins, not only pass/fail."""
    gu = sys.modules.get("gpuutil")
    stats = getattr(gu, "STATS", None) if gu else None
    if not stats:
        return
    tr = terminalreporter
    tr.section("observed parity errors (bf16 bar: |got-ref| <= 2e-2 + %.4g |ref|, Frobenius <= 1e-2)" % gu.C_ATTN)
    by_test = {}
    for st in stats:
        by_test.setdefault(st["test"], []).append(st)
    for test, rows in by_test.items():
        parts = []
        a = [r for r in rows if r["kind"] == "attn-bf16"]
        if a:
            parts.append("attn bf16 x%d: max-abs %.3e, worst bar use %.3f, max Frobenius %.3e, needed c %.3g, "
                         "max|ref| %.3g" % (len(a), max(r["max_abs"] for r in a), max(r["bar_use"] for r in a),
                                            max(r["fro"] for r in a), max(r["need_c"] for r in a),
                                            max(r["max_ref"] for r in a)))
        f = [r for r in rows if r["kind"] == "attn-f32"]
        if f:
            parts.append("attn fp32 x%d: normwise %.3e" % (len(f), max(r["normwise"] for r in f)))
        k = [r for r in rows if r["kind"] == "keys-bf16"]
        if k:
            parts.append("keys bf16: %d of %d off the oracle's rounding, %d outside the bar" % (
                sum(r["off_rounding"] for r in k), sum(r["n"] for r in k), sum(r["outside_bar"] for r in k)))
        kf = [r for r in rows if r["kind"] == "keys-f32"]
        if kf:
            parts.append("keys fp32: normwise %.3e" % max(r["normwise"] for r in kf))
        tr.write_line(f"{test}: " + "; ".join(parts))
