"""The public headers are C: a C99 program (tests/abi_c_client.c) compiles
against include/dora.h and include/dora_measure.h with gcc in strict mode,
links with libdora.so, and drives the host-side entry points with no GPU."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2604_26256_amd")


def test_headers_compile_as_c_and_the_abi_runs_from_c(tmp_path):
    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None:
        pytest.skip("no C compiler")
    lib = os.environ.get("DORA_LIBRARY") or os.path.join(PKG, "libdora.so")
    if not os.path.exists(lib):
        pytest.fail("libdora.so is not built (run __graft_entry__.build())")
    exe = str(tmp_path / "abi_c_client")
    subprocess.run([cc, "-std=c99", "-Wall", "-Wextra", "-Werror", "-pedantic",
                    "-I", os.path.join(ROOT, "include"),
                    os.path.join(ROOT, "tests", "abi_c_client.c"), lib,
                    "-Wl,-rpath," + os.path.dirname(lib),
                    # a sanitizer build of the library resolves its runtime's
                    # symbols at load time (the runtime is preloaded)
                    "-Wl,--allow-shlib-undefined", "-o", exe], check=True)
    r = subprocess.run([exe], stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True,
                       timeout=120)
    assert r.returncode == 0 and r.stdout.strip().endswith("ok"), r.stdout
