"""The host side of the library (argument validation, overlap checks, error state, the
Hadamard constructions) under AddressSanitizer and UndefinedBehaviorSanitizer: the
sanitizer build of the library runs every test of tests/test_abi.py in a child process
that loads the shared ASan runtime first.  No GPU is used."""

import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.skipif(shutil.which("hipcc") is None and not os.path.exists("/opt/rocm/bin/hipcc"),
                    reason="hipcc is needed to build the sanitizer library")
def test_abi_suite_under_asan_and_ubsan():
    from paper_2405_16406_amd import build

    lib = build.build_sanitized()
    env = dict(os.environ)
    pre = env.get("LD_PRELOAD", "")
    env["LD_PRELOAD"] = build.asan_runtime() + (":" + pre if pre else "")
    env["ASAN_OPTIONS"] = "detect_leaks=0:halt_on_error=1:abort_on_error=0"
    env["UBSAN_OPTIONS"] = "halt_on_error=1:print_stacktrace=1"
    env["SQ_TEST_LIBRARY"] = lib
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_abi.py")],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=900)
    out = r.stdout[-4000:] + r.stderr[-4000:]
    assert r.returncode == 0, out
    assert "passed" in r.stdout and "AddressSanitizer" not in out and "runtime error" not in out, out
