"""The host-side ABI checks of test_abi_cpu.py, run again against a build whose
host code (argument validation, configuration checks, arena planning) is
compiled with AddressSanitizer.  A heap or stack overflow, use after free or
double free in those paths aborts the child process with a report.  No GPU
is needed: none of these calls reaches the HIP runtime."""

import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_abi_host_code_under_asan():
    from paper_2309_01226_amd import build as B
    rt = B.asan_runtime()
    if rt is None:
        pytest.skip("the compiler ships no shared AddressSanitizer runtime")
    lib = B.build_asan(verbose=False)
    env = dict(os.environ)
    env.update(SAT_LIBRARY=lib, LD_PRELOAD=rt,
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=1:halt_on_error=1")
    r = subprocess.run([sys.executable, "-m", "pytest", os.path.join(ROOT, "tests", "test_abi_cpu.py"),
                        "-q", "-p", "no:cacheprovider"],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    out = r.stdout + r.stderr
    assert "AddressSanitizer" not in out, out[-4000:]
    assert r.returncode == 0, out[-4000:]
    assert " passed" in out, out[-2000:]


def test_asan_build_is_instrumented_and_selected():
    """The child really loads the instrumented library: SAT_LIBRARY points the
    binding at it, and its host code calls the sanitizer's checks."""
    from paper_2309_01226_amd import build as B
    if B.asan_runtime() is None:
        pytest.skip("the compiler ships no shared AddressSanitizer runtime")
    lib = B.build_asan(verbose=False)
    syms = subprocess.run(["nm", "-D", lib], capture_output=True, text=True).stdout
    assert "__asan_report" in syms
    env = dict(os.environ, SAT_LIBRARY=lib)
    r = subprocess.run([sys.executable, "-c", "from paper_2309_01226_amd import _lib; print(_lib.LIB_PATH)"],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=120)
    assert r.returncode == 0 and r.stdout.strip() == lib, r.stdout + r.stderr
