"""Checks on the gfx950 code objects inside the built ``libfcg.so`` (no GPU needed).

Every device function must be inlined into its kernel: a function called out of
line needs a call frame and register save/restore on every launch.  The decode
kernel's split merge once ended up out of line (the compiler's choice when more
kernel instances called it) and every decode launch took ~2 us longer.  In the
code objects an out-of-line device function shows as a FUNC symbol without the
kernel descriptor (``<name>.kd``) that every kernel has.
"""
import os
import shutil
import subprocess
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIB = os.path.join(ROOT, "paper_2606_13097_amd", "libfcg.so")
LLVM = "/opt/rocm/llvm/bin"
TOOLS = [os.path.join(LLVM, t) for t in ("llvm-objcopy", "clang-offload-bundler", "llvm-readelf")]
TARGET = "hipv4-amdgcn-amd-amdhsa--gfx950"
MAGIC = b"__CLANG_OFFLOAD_BUNDLE__"


def _code_objects(tmp):
    fat = os.path.join(tmp, "fatbin")
    subprocess.run([TOOLS[0], f"--dump-section=.hip_fatbin={fat}", LIB, os.path.join(tmp, "stripped")], check=True,
                   capture_output=True)
    data = open(fat, "rb").read()
    starts = []
    i = data.find(MAGIC)
    while i >= 0:
        starts.append(i)
        i = data.find(MAGIC, i + 1)
    objs = []
    for n, s in enumerate(starts):  # one offload bundle per source file with device code
        e = starts[n + 1] if n + 1 < len(starts) else len(data)
        b = os.path.join(tmp, f"b{n}")
        open(b, "wb").write(data[s:e])
        co = os.path.join(tmp, f"c{n}.co")
        subprocess.run([TOOLS[1], "--unbundle", "--type=o", f"--targets={TARGET}", f"--input={b}", f"--output={co}"],
                       check=True, capture_output=True)
        objs.append(co)
    return objs


def _symbols(co):
    out = subprocess.run([TOOLS[2], "-s", "--wide", co], check=True, capture_output=True, text=True).stdout
    funcs, kds = set(), set()
    for line in out.splitlines():
        f = line.split()
        if len(f) >= 8 and f[3] == "FUNC":
            funcs.add(f[7])
        if len(f) >= 8 and f[3] == "OBJECT" and f[7].endswith(".kd"):
            kds.add(f[7][:-3])
    return funcs, kds


@pytest.mark.skipif(not os.path.exists(LIB), reason="libfcg.so is not built")
@pytest.mark.skipif(not all(os.path.exists(t) for t in TOOLS), reason="ROCm LLVM tools not found")
def test_every_device_function_is_inlined_into_its_kernel():
    tmp = tempfile.mkdtemp(prefix="fcg_codegen_")
    try:
        objs = _code_objects(tmp)
        assert len(objs) >= 6, "one gfx950 code object per source file with kernels"
        kernels, outlined = 0, []
        for co in objs:
            funcs, kds = _symbols(co)
            kernels += len(kds)
            outlined += sorted(f for f in funcs if f not in kds)
        assert kernels > 0
        assert not outlined, f"device functions called out of line: {outlined[:5]}"
    finally:
        shutil.rmtree(tmp, ignore_errors=True)
