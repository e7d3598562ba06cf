"""Turn rocprofv3 CSV output into the short summaries kept under ``profiles/``.

    python -m paper_2606_13097_amd.profiling stats KERNEL_STATS_CSV --title T --command C \
        [--trace KERNEL_TRACE_CSV --launches graft_kernel [--launches ...] --note N]
    python -m paper_2606_13097_amd.profiling traffic --kernel graft_kernel --source csrc/k_graft.hip \
        --fetch F.csv --write W.csv --copy-fetch CF.csv --copy-write CW.csv --copy-bytes 1073741824 \
        --skip 1 --command C
    python -m paper_2606_13097_amd.profiling mfma --kernel attn_prefill_mfma_kernel \
        --source csrc/k_attn_mfma.hip --ops OPS.csv --gemm-ops GEMM.csv --gemm-flops 1.37e11 --command C

``stats`` with ``--trace`` also lists every launch of the named kernels in dispatch order
(from a kernel trace of the same run, or an excerpt of it with the same columns), so that
per-phase averages can be read against the bench's own figures.  ``traffic`` averages the kernel's FETCH_SIZE and WRITE_SIZE (KiB per dispatch) over its
dispatches after the first ``--skip`` ones, and calibrates each counter by what it reads
for a plain device copy of ``--copy-bytes`` bytes.  ``mfma`` does the same for the bf16
matrix-op counter SQ_INSTS_VALU_MFMA_MOPS_BF16, calibrated by a bf16 GEMM of known FLOPs
(``--gemm-flops``; its largest dispatch).  Each JSON records the SHA-256 of the kernel's
source files: ``bench.py`` reports the figures only while they are unchanged.
"""
from __future__ import annotations

import argparse
import csv
import hashlib
import json
import os
import sys

PKG = os.path.dirname(os.path.abspath(__file__))


def source_sha256(rel: str) -> str:
    """SHA-256 over the kernel's source files (``a.hip+b.hpp``: their bytes in that order)."""
    h = hashlib.sha256()
    for part in rel.split("+"):
        with open(os.path.join(PKG, part), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def _short(name: str) -> str:
    n = name.replace("void ", "")
    depth, out = 0, []
    for ch in n:  # cut the argument list, keep template arguments
        if ch == "(" and depth == 0:
            break
        depth += ch == "<"
        depth -= ch == ">"
        out.append(ch)
    return "".join(out).strip() or name[:40]


def stats_markdown(path: str, title: str, command: str) -> str:
    rows = list(csv.DictReader(open(path)))
    lines = [f"# {title}", "", "Command:", "", f"    {command}", "",
             "| kernel | calls | avg (us) | min (us) | max (us) | total (ms) |", "|---|---|---|---|---|---|"]
    for r in rows:
        lines.append(f"| {_short(r['Name'])} | {r['Calls']} | {float(r['AverageNs']) / 1e3:.2f} | "
                     f"{float(r['MinNs']) / 1e3:.2f} | {float(r['MaxNs']) / 1e3:.2f} | "
                     f"{float(r['TotalDurationNs']) / 1e6:.2f} |")
    return "\n".join(lines) + "\n"


def launches_markdown(trace: str, kernels, note: str = "") -> str:
    """Every launch of each named kernel, in dispatch order: duration in microseconds."""
    rows = list(csv.DictReader(open(trace)))
    rows.sort(key=lambda r: int(r["Start_Timestamp"]))
    out = []
    for k in kernels:
        d = [(int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3 for r in rows if k in r["Kernel_Name"]]
        if not d:
            continue
        out += ["", f"{k}: {len(d)} launches in dispatch order (us):", "",
                "    " + ", ".join(f"{x:.1f}" for x in d)]
    if out and note:
        out += ["", note]
    return "\n".join(out) + ("\n" if out else "")


def _per_dispatch(path: str, kernel: str, counter: str):
    vals = []
    for r in csv.DictReader(open(path)):
        if kernel in r["Kernel_Name"] and r["Counter_Name"] == counter:
            vals.append((int(r["Dispatch_Id"]), float(r["Counter_Value"])))
    return [v for _, v in sorted(vals)]


def traffic(args) -> dict:
    end = args.skip + args.take if args.take else None
    f = _per_dispatch(args.fetch, args.kernel, "FETCH_SIZE")[args.skip:end]
    w = _per_dispatch(args.write, args.kernel, "WRITE_SIZE")[args.skip:end]
    cf = max(v for v in _per_dispatch(args.copy_fetch, args.copy_kernel, "FETCH_SIZE"))
    cw = max(v for v in _per_dispatch(args.copy_write, args.copy_kernel, "WRITE_SIZE"))
    ff = args.copy_bytes / (cf * 1024.0)
    wf = args.copy_bytes / (cw * 1024.0)
    fetch_b = sum(f) / len(f) * 1024.0 * ff
    write_b = sum(w) / len(w) * 1024.0 * wf
    return {"kernel": args.kernel, "source": args.source, "source_sha256": source_sha256(args.source),
            "dispatches": len(f), "fetch_kib_avg": sum(f) / len(f), "write_kib_avg": sum(w) / len(w),
            "fetch_factor": ff, "write_factor": wf, "traffic_bytes_per_launch": fetch_b + write_b,
            "command": args.command}


def _sum_per_dispatch(path: str, kernel: str, counter: str):
    """Counter values summed per dispatch (a raw counter may come in several rows)."""
    acc = {}
    for r in csv.DictReader(open(path)):
        if kernel in r["Kernel_Name"] and r["Counter_Name"] == counter:
            d = int(r["Dispatch_Id"])
            acc[d] = acc.get(d, 0.0) + float(r["Counter_Value"])
    return [acc[d] for d in sorted(acc)]


MOPS = "SQ_INSTS_VALU_MFMA_MOPS_BF16"


def mfma(args) -> dict:
    end = args.skip + args.take if args.take else None
    m = _sum_per_dispatch(args.ops, args.kernel, MOPS)[args.skip:end]
    g = max(_sum_per_dispatch(args.gemm_ops, "", MOPS))
    per_op = args.gemm_flops / g
    return {"kernel": args.kernel, "source": args.source, "source_sha256": source_sha256(args.source),
            "counter": MOPS, "dispatches": len(m), "ops_avg": sum(m) / len(m), "flops_per_op": per_op,
            "gemm_flops": args.gemm_flops, "gemm_ops": g,
            "counter_flops_per_launch": sum(m) / len(m) * per_op, "command": args.command}


def main(argv=None):
    ap = argparse.ArgumentParser()
    sub = ap.add_subparsers(dest="cmd", required=True)
    s = sub.add_parser("stats")
    s.add_argument("csv")
    s.add_argument("--title", required=True)
    s.add_argument("--command", required=True)
    s.add_argument("--trace", default=None, help="kernel trace CSV of the same run")
    s.add_argument("--launches", action="append", default=[], help="kernel whose launches to list")
    s.add_argument("--note", default="")
    t = sub.add_parser("traffic")
    for k in ("kernel", "source", "fetch", "write", "copy_fetch", "copy_write", "command"):
        t.add_argument("--" + k.replace("_", "-"), dest=k, required=True)
    t.add_argument("--copy-kernel", default="copyBuffer")
    t.add_argument("--copy-bytes", type=float, default=float(1 << 30))
    t.add_argument("--skip", type=int, default=0, help="dispatches to leave out first (warm-up)")
    t.add_argument("--take", type=int, default=0, help="dispatches to average after those (0: all)")
    m = sub.add_parser("mfma")
    for k in ("kernel", "source", "ops", "gemm_ops", "command"):
        m.add_argument("--" + k.replace("_", "-"), dest=k, required=True)
    m.add_argument("--gemm-flops", type=float, required=True)
    m.add_argument("--skip", type=int, default=0)
    m.add_argument("--take", type=int, default=0)
    a = ap.parse_args(argv)
    if a.cmd == "stats":
        sys.stdout.write(stats_markdown(a.csv, a.title, a.command))
        if a.trace and a.launches:
            sys.stdout.write(launches_markdown(a.trace, a.launches, a.note))
    else:
        json.dump(traffic(a) if a.cmd == "traffic" else mfma(a), sys.stdout, indent=1)
        sys.stdout.write("\n")


if __name__ == "__main__":
    main()
