"""The C-ABI checks of test_abi.py against a build whose host code runs under
AddressSanitizer and UndefinedBehaviorSanitizer (argument validation, workspace
arithmetic, error strings; no GPU needed).  A sanitizer report aborts the child
interpreter, so the test fails on any out-of-bounds access, use after free,
signed overflow or misaligned access in the host code these checks reach."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.timeout(900)
def test_abi_checks_under_host_sanitizers(tmp_path):
    from paper_2106_12566_amd import build_hostsan
    try:
        rt = build_hostsan.runtime()
    except RuntimeError as e:
        pytest.skip(str(e))
    lib = build_hostsan.build_hostsan(str(tmp_path / "libkrpe_hostsan.so"))
    env = dict(os.environ, KRPE_LIBRARY=lib, LD_PRELOAD=rt, ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    res = subprocess.run([sys.executable, "-m", "pytest", "-q", "-p", "no:cacheprovider",
                          os.path.join(ROOT, "tests", "test_abi.py")],
                         cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    out = res.stdout + res.stderr
    assert res.returncode == 0, out[-4000:]
    assert "ERROR: AddressSanitizer" not in out and "runtime error:" not in out, out[-4000:]
