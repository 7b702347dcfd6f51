"""AddressSanitizer + UndefinedBehaviorSanitizer build of the oracle (test
infrastructure, CPU only): the same dora_oracle.c, compiled with the clang of
the ROCm toolchain (its ASan runtime is the one the sanitized libdora uses,
so both can share one process) and LLVM's OpenMP runtime.  Selected by
oracle/__init__.py through DORA_ORACLE_LIBRARY.  Only tests/ use it."""
from __future__ import annotations

import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
CLANG = "/opt/rocm/llvm/bin/clang"
OMP_DIR = "/opt/rocm/llvm/lib"


def build(out_dir: str) -> str:
    os.makedirs(out_dir, exist_ok=True)
    lib = os.path.join(out_dir, "liboracle.so")
    cmd = [CLANG, "-O1", "-g", "-std=c11", "-ffp-contract=off", "-fopenmp", "-fPIC", "-shared",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           "-fno-omit-frame-pointer", "-shared-libsan", f"-L{OMP_DIR}", f"-Wl,-rpath,{OMP_DIR}",
           os.path.join(HERE, "dora_oracle.c"), "-o", lib, "-lm"]
    subprocess.run(cmd, check=True)
    return lib
