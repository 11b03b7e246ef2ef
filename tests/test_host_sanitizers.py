"""The C-ABI layer's host code under AddressSanitizer and
UndefinedBehaviorSanitizer: abi.hip (argument validation, shape, overflow
and overlap checks, error messages) is rebuilt with both sanitizers on its
host code (paper_2009_00804_amd.build.build_sanitized) and the ABI host
tests run against that library in a child process with the ASan runtime
preloaded.  Any sanitizer report fails the test.  No GPU is used: every
call in those tests returns from validation."""
import os
import shutil
import subprocess
import sys

import pytest

from paper_2009_00804_amd import build as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.skipif(shutil.which("hipcc") is None and not os.path.exists("/opt/rocm/bin/hipcc"),
                    reason="ROCm toolchain absent")
def test_abi_host_checks_clean_under_asan_and_ubsan():
    lib = B.build_sanitized()
    env = dict(os.environ)
    env["LD_PRELOAD"] = B.asan_runtime()
    env["ASAN_OPTIONS"] = "detect_leaks=0:halt_on_error=1"
    env["UBSAN_OPTIONS"] = "halt_on_error=1:print_stacktrace=1"
    code = ("import sys, pytest\n"
            "import paper_2009_00804_amd.saga as S\n"
            f"S.LIB_PATH = {lib!r}\n"
            "sys.exit(pytest.main(['-q', '-s', '-p', 'no:cacheprovider', '-m', 'not gpu',\n"
            "                      'tests/test_abi_host.py']))\n")
    r = subprocess.run([sys.executable, "-c", code], cwd=ROOT, env=env, capture_output=True, text=True,
                       timeout=600)
    out = r.stdout + r.stderr
    assert "AddressSanitizer" not in out and "runtime error:" not in out, out[-6000:]
    assert r.returncode == 0, out[-6000:]
    assert " passed" in out
