"""Build liblosa.so (the C-ABI library) in-tree with hipcc for gfx950.

    python -m paper_2608_12032_amd.build

Compiles every source under csrc/ to an object in parallel, then links the
shared library next to this file.  Always rebuilds.
"""
from __future__ import annotations

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
OUT = os.path.join(PKG, "liblosa.so")
OBJDIR = os.path.join(PKG, "_build")
ARCH = "gfx950"

SOURCES = ["calib.hip", "select.hip", "sparse_fwd.hip", "f32_path.hip", "recall.hip",
           "noalloc.hip", "abi.cpp"]

COMMON = [
    "-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
    # keep the compiler from emitting packed fp32 arithmetic
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # MFMA results in arch VGPRs: the softmax works on the score accumulators
    # directly instead of copying them out of AGPRs
    "-mllvm", "-amdgpu-mfma-vgpr-form",
    "-I", INCLUDE, "-I", CSRC,
    "-Wno-unused-command-line-argument",
]


def _hipcc() -> str:
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    cand = os.path.join(rocm, "bin", "hipcc")
    return cand if os.path.exists(cand) else "hipcc"


def _run(cmd):
    p = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    # the host compiler pass does not know the packed-fp32 feature: harmless
    out = "\n".join(line for line in p.stdout.splitlines()
                    if "packed-fp32-ops" not in line and line.strip())
    if p.returncode != 0:
        raise RuntimeError(f"command failed ({p.returncode}): {' '.join(cmd)}\n{out}")
    return out


def _check_stubs(lib: str) -> None:
    """Fail if a kernel's host launch stub is missing from the library.

    The host compiler pass can drop a kernel template instantiation without a
    diagnostic; the library then links but cannot be loaded."""
    p = subprocess.run(["nm", "-D", "--undefined-only", lib], stdout=subprocess.PIPE,
                       stderr=subprocess.STDOUT, text=True)
    if p.returncode != 0:
        return  # no nm: the load test catches the same problem
    missing = [ln.split()[-1] for ln in p.stdout.splitlines() if "__device_stub__" in ln]
    if missing:
        raise RuntimeError("kernel launch stubs missing from the host build: " + ", ".join(missing))


def build(verbose: bool = False, jobs: int | None = None) -> str:
    os.makedirs(OBJDIR, exist_ok=True)
    hipcc = _hipcc()
    objs = []
    cmds = []
    for src in SOURCES:
        obj = os.path.join(OBJDIR, os.path.splitext(src)[0] + ".o")
        objs.append(obj)
        cmds.append([hipcc, *COMMON, "-c", os.path.join(CSRC, src), "-o", obj])
    jobs = jobs or min(len(cmds), max(1, os.cpu_count() or 1))
    with ThreadPoolExecutor(jobs) as ex:
        outs = list(ex.map(_run, cmds))
    if verbose:
        for c, o in zip(cmds, outs):
            print(" ".join(c))
            if o:
                print(o)
    tmp = OUT + ".tmp"
    _run([hipcc, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs])
    _check_stubs(tmp)
    os.replace(tmp, OUT)
    return OUT


if __name__ == "__main__":
    path = build(verbose="-v" in sys.argv)
    print(path)
