"""Host-side sanitizer check of the C ABI's validation code.

    python -m paper_2608_12032_amd.hostsan

Builds a copy of the library whose host code (abi.cpp: argument checks,
workspace sizing, error strings) carries AddressSanitizer and
UndefinedBehaviorSanitizer, linked with the kernel objects of the last
regular build (the GPU code is not instrumented), then runs the CPU tests of
the ABI against that copy in a child process with the ASan runtime preloaded.
Needs no GPU: the CPU tests reach only the validation paths.  Exits with the
tests' status; any sanitizer report aborts them.
"""
from __future__ import annotations

import glob
import os
import subprocess
import sys

from . import build as B

SAN_DIR = os.path.join(B.OBJDIR, "hostsan")
SAN_LIB = os.path.join(SAN_DIR, "liblosa.so")
# -Xarch_host before each -fsanitize= keeps the device code uninstrumented
SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
       "-Xarch_host", "-fno-omit-frame-pointer", "-Xarch_host", "-fno-sanitize-recover=all"]


def _asan_runtime() -> str:
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    found = sorted(glob.glob(os.path.join(rocm, "lib/llvm/lib/clang/*/lib/linux/"
                                                "libclang_rt.asan-x86_64.so")))
    if not found:
        raise RuntimeError("no clang ASan runtime (libclang_rt.asan-x86_64.so) under " + rocm)
    return found[-1]


def build_sanitized() -> str:
    kernels = [os.path.join(B.OBJDIR, os.path.splitext(s)[0] + ".o")
               for s in B.SOURCES if s != "abi.cpp"]
    missing = [o for o in kernels if not os.path.exists(o)]
    if missing:
        raise RuntimeError("kernel objects missing; run `python -m paper_2608_12032_amd.build` "
                           "first: " + ", ".join(missing))
    os.makedirs(SAN_DIR, exist_ok=True)
    hipcc = B._hipcc()
    abi_obj = os.path.join(SAN_DIR, "abi.o")
    B._run([hipcc, *B.COMMON, *SAN, "-c", os.path.join(B.CSRC, "abi.cpp"), "-o", abi_obj])
    B._run([hipcc, f"--offload-arch={B.ARCH}", "-shared", "-fPIC", *SAN, "-o", SAN_LIB,
            *kernels, abi_obj])
    return SAN_LIB


def main() -> int:
    lib = build_sanitized()
    env = dict(os.environ)
    env["LD_PRELOAD"] = _asan_runtime()
    env["ASAN_OPTIONS"] = "detect_leaks=0:halt_on_error=1"
    env["UBSAN_OPTIONS"] = "print_stacktrace=1:halt_on_error=1"
    env["LOSA_LIBRARY"] = lib
    tests = os.path.join(B.ROOT, "tests", "test_abi_cpu.py")
    p = subprocess.run([sys.executable, "-m", "pytest", "-q", "-m", "not gpu", "-p",
                        "no:cacheprovider", tests], env=env, cwd=B.ROOT)
    return p.returncode


if __name__ == "__main__":
    sys.exit(main())
