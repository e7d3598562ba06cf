"""Build the gfx950 shared libraries of the package in-tree with hipcc.

    python -m paper_2606_13097_amd.build        # or __graft_entry__.build()

Produces ``paper_2606_13097_amd/libfcg.so`` (the grafting hot path, C ABI in
``include/fcg.h``), ``paper_2606_13097_amd/synth/libfcg_synth.so`` (the
device twin of the seeded input generator) and
``paper_2606_13097_amd/measure/libfcg_measure.so`` (a matrix-core rate probe
for the bench).  Every call recompiles.
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import shutil
import subprocess
import sys
import tempfile

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")

ARCH = os.environ.get("FCG_OFFLOAD_ARCH", "gfx950")
HIPCC = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"

COMMON = [
    f"--offload-arch={ARCH}", "-O3", "-fPIC", "-std=c++17", "-x", "hip",
    # code objects loadable by the HIP runtime that PyTorch ships (ROCm 7.0)
    "-mcode-object-version=5",
    # no packed-fp32 instructions: plain float code only
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function", "-Wno-unused-variable",
    "-I", INCLUDE, "-I", CSRC,
]

LIBS = {
    os.path.join(PKG, "libfcg.so"): [
        os.path.join(CSRC, f) for f in
        ("api.cpp", "planner.cpp", "locality.cpp", "k_graft.hip", "k_append.hip", "k_attn_rows.hip", "k_attn_mfma.hip",
         "k_decode.hip", "k_decode_mfma.hip", "noalloc.hip")
    ],
    os.path.join(PKG, "synth", "libfcg_synth.so"): [os.path.join(PKG, "synth", "synth.hip")],
    os.path.join(PKG, "measure", "libfcg_measure.so"): [os.path.join(PKG, "measure", "peak.hip")],
}


def _run(cmd):
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    out = "\n".join(l for l in r.stdout.splitlines() if "packed-fp32-ops" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"build step failed ({r.returncode}): {' '.join(cmd)}\n{out}")
    return out


def build(verbose: bool = False) -> list:
    built = []
    with tempfile.TemporaryDirectory(prefix="fcg_build_") as tmp:
        jobs = []
        for so, srcs in LIBS.items():
            objs = []
            for s in srcs:
                o = os.path.join(tmp, os.path.basename(so) + "." + os.path.basename(s) + ".o")
                objs.append(o)
                jobs.append([HIPCC, *COMMON, "-c", s, "-o", o])
            built.append((so, objs))
        workers = min(8, os.cpu_count() or 4)
        with cf.ThreadPoolExecutor(workers) as ex:
            for out in ex.map(_run, jobs):
                if verbose and out.strip():
                    print(out)
        for so, objs in built:
            tmp_so = so + ".tmp"
            _run([HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp_so])
            os.replace(tmp_so, so)
    return [so for so, _ in built]


if __name__ == "__main__":
    for p in build(verbose="-v" in sys.argv):
        print("built", p)
