"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU).

Builds the library with both sanitizers on its host compilation (segment
formation, packing, span validation, size and workspace arithmetic, argument
checks of every entry point) and runs the host ABI tests, random span lists
included, against that build in a child process with the ASan runtime
preloaded.  Any out-of-bounds access, use after free or undefined behaviour
in the host code aborts the child."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_host_abi_tests_pass_under_asan_and_ubsan():
    from paper_2607_11185_amd import build as B
    try:
        lib = B.build(sanitize=True, jobs=5)
        rt = B.asan_runtime()
    except (RuntimeError, OSError, subprocess.CalledProcessError) as e:
        pytest.skip(f"sanitizer build unavailable: {e}")
    assert os.path.exists(rt), rt
    syms = subprocess.run(["nm", "-D", "--undefined-only", lib], capture_output=True, text=True,
                          check=True).stdout
    assert "__asan_report_load" in syms and "__ubsan_handle_" in syms, "not instrumented"
    env = dict(os.environ, SEG_LIB_PATH=lib, LD_PRELOAD=rt,
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-p", "no:cacheprovider",
                        "-m", "not gpu", os.path.join(ROOT, "tests", "test_abi_host.py")],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=900)
    tail = (r.stdout + r.stderr)[-3000:]
    assert r.returncode == 0, tail
    assert "passed" in r.stdout and "failed" not in r.stdout, tail
