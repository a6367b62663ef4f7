"""The host compilation code (csrc/host.cpp: reverse Cuthill-McKee, bandwidth,
dense and 1-bit block packing, receiver-major lists, supernode slices) built
with -fsanitize=address,undefined and driven over edge-case inputs in a
child process with the sanitizer runtime preloaded.  Any out-of-bounds
access, use after free or undefined behaviour aborts the child; its results
are also checked against the oracle (tests/host_sanitized_cases.py)."""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _runtime(name):
    cxx = os.environ.get("CXX_SAN", "g++")
    if shutil.which(cxx) is None:
        return None
    r = subprocess.run([cxx, f"-print-file-name={name}"], capture_output=True, text=True)
    path = r.stdout.strip()
    return path if os.path.isabs(path) and os.path.exists(path) else None


def test_host_code_under_address_and_undefined_behaviour_sanitizers():
    asan = _runtime("libasan.so")
    if asan is None:
        pytest.skip("no g++ with the address sanitizer runtime")
    from paper_1906_11786_amd.build import build_host_sanitized
    lib = build_host_sanitized()
    env = dict(os.environ)
    env["LD_PRELOAD"] = asan
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=1:halt_on_error=1"
    env["UBSAN_OPTIONS"] = "halt_on_error=1:print_stacktrace=1"
    env["OMP_NUM_THREADS"] = "1"
    r = subprocess.run([sys.executable, os.path.join(ROOT, "tests", "host_sanitized_cases.py"), lib],
                       capture_output=True, text=True, env=env, timeout=600)
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-4000:]
    assert "ALL OK" in r.stdout, out[-4000:]
    assert "runtime error" not in out and "AddressSanitizer" not in out, out[-4000:]
