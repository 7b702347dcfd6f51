"""Host-side AddressSanitizer + UndefinedBehaviorSanitizer build of libdora (CPU
checks only).

    python -m paper_2604_26256_amd.sanitize OUT_DIR

Builds OUT_DIR/libdora.so from the same sources as build.py, with the host
half of every translation unit (the C-ABI front end, argument validation,
the host pool, the planners, and the host side of each .hip file)
instrumented; device code is compiled as usual.  The result needs the clang
ASan runtime loaded first in the process (LD_PRELOAD), and is selected by the
binding through DORA_LIBRARY.  It is meant for the CPU test suite, which
calls only host code; it is never used on a GPU.
"""
from __future__ import annotations

import os
import subprocess
import sys

from paper_2604_26256_amd import build as B

# Every sanitizer flag is given to the host compilation only.
HOST_SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
            "-Xarch_host", "-fno-omit-frame-pointer", "-Xarch_host", "-fno-sanitize-recover=all",
            "-Xarch_host", "-g"]


def asan_runtime() -> str:
    """Path of the clang ASan runtime matching hipcc's compiler."""
    clang = os.path.join(os.path.dirname(os.path.realpath(B._hipcc())), "..", "llvm", "bin",
                         "clang")
    if not os.path.exists(clang):
        clang = "/opt/rocm/llvm/bin/clang"
    out = subprocess.run([clang, "-print-file-name=libclang_rt.asan-x86_64.so"],
                         stdout=subprocess.PIPE, text=True, check=True).stdout.strip()
    if not os.path.exists(out):
        raise RuntimeError("clang ASan runtime not found")
    return out


def build(out_dir: str) -> str:
    hipcc = B._hipcc()
    objdir = os.path.join(out_dir, "_obj")
    os.makedirs(objdir, exist_ok=True)
    common = [c for c in B.COMMON if c != "-O3"] + ["-O1"]
    objs = []
    for src in B.HIP_SOURCES:
        obj = os.path.join(objdir, src + ".o")
        B._run([hipcc, "-x", "hip", *B.DEVICE, *common, *HOST_SAN, "-c",
                os.path.join(B.CSRC, src), "-o", obj])
        objs.append(obj)
    for src in B.CXX_SOURCES:
        obj = os.path.join(objdir, src + ".o")
        B._run([hipcc, *common, *HOST_SAN, "-c", os.path.join(B.CSRC, src), "-o", obj])
        objs.append(obj)
    lib = os.path.join(out_dir, "libdora.so")
    B._run([hipcc, f"--offload-arch={B.ARCH}", "-shared", "-fPIC", *objs, *HOST_SAN,
            "-Xarch_host", "-shared-libsan", "-o", lib])
    return lib


if __name__ == "__main__":
    print(build(sys.argv[1] if len(sys.argv) > 1 else os.path.join(B.PKG, "_san")))
