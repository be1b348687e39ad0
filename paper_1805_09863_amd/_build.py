"""Build libkbest.so (HIP for gfx950) in-tree.

Usage: ``python -m paper_1805_09863_amd._build`` or ``build()``.  Every call
recompiles all sources; objects go to ``_build/`` at the repository root
and the shared library to ``paper_1805_09863_amd/libkbest.so``.  The device
assembly of the sources with hand-written memory instructions is checked
for hazards (isa_check.py); a hazard fails the build before anything is
linked.
"""
from __future__ import annotations

import concurrent.futures as cf
import glob
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
OBJDIR = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libkbest.so")
ARCH = "gfx950"

# -packed-fp32-ops: keep the compiler from emitting packed fp32 VALU ops.
HIPFLAGS = ["--offload-arch=" + ARCH, "-O3", "-std=c++17", "-fPIC", "-Wall",
            "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
            "-I", INCLUDE]


def _hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


def _compile(hipcc: str, src: str) -> str:
    obj = os.path.join(OBJDIR, os.path.basename(src) + ".o")
    cmd = [hipcc] + HIPFLAGS + ["-c", src, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"compile failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    return obj


# Sources whose inline-assembly memory instructions take scalar operands or
# rely on an M0 set by an earlier statement: their device assembly is checked
# for the wait states and M0 uses that the compiler does not handle there.
ISA_CHECKED = ("k1_wide.hip",)


def _device_asm(hipcc: str, src: str) -> str:
    out = os.path.join(OBJDIR, os.path.basename(src) + "." + ARCH + ".s")
    cmd = [hipcc] + HIPFLAGS + ["--cuda-device-only", "-S", src, "-o", out]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"compile failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    return out


def check_isa(asm_path: str) -> None:
    from paper_1805_09863_amd import isa_check
    with open(asm_path) as f:
        bad = isa_check.check(f.read())
    if bad:
        raise RuntimeError(f"{asm_path}: {len(bad)} inline-assembly hazard(s):\n  " + "\n  ".join(bad[:20]))


def build(verbose: bool = False, jobs: int | None = None) -> str:
    hipcc = _hipcc()
    os.makedirs(OBJDIR, exist_ok=True)
    srcs = sorted(glob.glob(os.path.join(CSRC, "*.hip")))
    checked = [s for s in srcs if os.path.basename(s) in ISA_CHECKED]
    jobs = jobs or min(len(srcs), max(1, min(8, os.cpu_count() or 1)))
    with cf.ThreadPoolExecutor(max_workers=jobs) as ex:
        asm = [ex.submit(_device_asm, hipcc, s) for s in checked]   # the long ones first
        objs = list(ex.map(lambda s: _compile(hipcc, s), srcs))
        for a in asm:
            check_isa(a.result())
    tmp = LIB + ".tmp"
    cmd = [hipcc, "--offload-arch=" + ARCH, "-shared", "-fPIC", "-o", tmp] + objs
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, LIB)
    if verbose:
        print(f"built {LIB} from {len(srcs)} sources", file=sys.stderr)
    return LIB


if __name__ == "__main__":
    build(verbose=True)
