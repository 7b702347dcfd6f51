"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only).

Builds libdora with every translation unit's host half instrumented (the
C-ABI validation, the host pool, the planners, the launch wrappers) and the
oracle with the same clang, then runs the rest of the CPU suite against those
builds in a child process with the ASan runtime preloaded.  Any ASan or UBSan
report fails the child (halt on the first error), and so this test.
"""
import glob
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.timeout(900)
def test_cpu_suite_under_asan_and_ubsan(tmp_path):
    sys.path.insert(0, ROOT)
    try:
        from oracle import sanitize_build as oracle_san
        from paper_2604_26256_amd import sanitize as lib_san
    except ImportError as e:  # the sanitizer builders are not shipped everywhere
        pytest.skip(f"sanitizer build scripts unavailable: {e}")
    try:
        runtime = lib_san.asan_runtime()
    except (RuntimeError, OSError, subprocess.CalledProcessError) as e:
        pytest.skip(f"no clang ASan runtime: {e}")
    out = str(tmp_path)
    lib = lib_san.build(out)
    olib = oracle_san.build(out)
    logs = os.path.join(out, "san")
    env = dict(os.environ)
    env.update({
        "LD_PRELOAD": runtime,
        "ASAN_OPTIONS": f"detect_leaks=0:verify_asan_link_order=0:log_path={logs}",
        "UBSAN_OPTIONS": f"print_stacktrace=1:halt_on_error=1:log_path={logs}",
        "DORA_LIBRARY": lib,
        "DORA_ORACLE_LIBRARY": olib,
    })
    probe = subprocess.run(
        [sys.executable, "-c", "import oracle; from paper_2604_26256_amd import dora; "
         "oracle._load(); print(dora.LIB_PATH); print(oracle._LIB_PATH)"],
        cwd=ROOT, env=env, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True,
        timeout=300)
    assert probe.returncode == 0, probe.stdout[-2000:]
    assert probe.stdout.split()[-2:] == [lib, olib], probe.stdout  # the builds under test
    r = subprocess.run(
        [sys.executable, "-m", "pytest", os.path.join(ROOT, "tests"), "-q", "-x",
         "-m", "not gpu", "-p", "no:cacheprovider",
         "--deselect", "tests/test_host_sanitizers.py::test_cpu_suite_under_asan_and_ubsan"],
        cwd=ROOT, env=env, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True,
        timeout=800)
    reports = sorted(glob.glob(logs + "*"))
    text = "".join(open(f).read() for f in reports)
    assert not reports, f"sanitizer reports:\n{text[:4000]}"
    assert r.returncode == 0, r.stdout[-4000:]
    assert " passed" in r.stdout
