"""The CPU oracle under AddressSanitizer and UndefinedBehaviorSanitizer: the oracle's own tests
run in a child Python process against a sanitizer build of oracle/octoref.c (host code only; no
GPU is involved), and must pass with no sanitizer report."""
import glob
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.skipif(bool(os.environ.get("OCTOREF_LIB")), reason="already the sanitizer run")
def test_oracle_tests_clean_under_asan_and_ubsan():
    from oracle import build
    try:
        asan = subprocess.run(["gcc", "-print-file-name=libasan.so"], capture_output=True,
                              text=True, check=True).stdout.strip()
    except (OSError, subprocess.CalledProcessError):
        pytest.skip("gcc is not available")
    if not os.path.isabs(asan) or not os.path.exists(asan):
        pytest.skip("the gcc AddressSanitizer runtime is not installed")
    lib = build.build(sanitize=True)
    env = dict(os.environ)
    env.update({
        "OCTOREF_LIB": lib,
        "LD_PRELOAD": asan,
        # the Python interpreter itself is not instrumented and keeps objects alive at exit
        "ASAN_OPTIONS": "detect_leaks=0:abort_on_error=0:halt_on_error=1",
        "UBSAN_OPTIONS": "halt_on_error=1:print_stacktrace=1",
    })
    files = sorted(f for f in glob.glob(os.path.join(ROOT, "tests", "test_oracle_*.py"))
                   if not f.endswith("test_oracle_sanitizers.py"))
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-m", "not gpu",
                        "-p", "no:cacheprovider", *files], cwd=ROOT, env=env,
                       capture_output=True, text=True, timeout=1500)
    out = r.stdout + r.stderr
    assert "AddressSanitizer" not in out and "runtime error:" not in out, out[-4000:]
    assert r.returncode == 0, out[-4000:]
    assert " passed" in out
