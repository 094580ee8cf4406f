"""Build the library with AddressSanitizer and UndefinedBehaviorSanitizer on its host code.

    python -m paper_2106_12566_amd.build_hostsan OUT.so

Only the host side of each source is instrumented (every sanitizer flag goes
to the host compilation); the device code is the same gfx950 code as in the
product build.  Load the result into an uninstrumented interpreter with the
sanitizer runtime preloaded:

    LD_PRELOAD=$(python -m paper_2106_12566_amd.build_hostsan --runtime) \\
    ASAN_OPTIONS=detect_leaks=0 KRPE_LIBRARY=OUT.so python -m pytest tests/test_abi.py

(the interpreter's own allocations are not tracked, hence detect_leaks=0).
"""
from __future__ import annotations

import glob
import os
import subprocess
import sys

from paper_2106_12566_amd import build

HOST_SANITIZERS = "-Xarch_host -fsanitize=address -Xarch_host -fsanitize=undefined -Xarch_host -fno-sanitize-recover=undefined -Xarch_host -fno-omit-frame-pointer"


def runtime() -> str:
    """Path of the clang AddressSanitizer runtime that hipcc links against."""
    for root in ("/opt/rocm/llvm/lib/clang", "/opt/rocm/lib/llvm/lib/clang"):
        hits = sorted(glob.glob(os.path.join(root, "*", "lib", "linux", "libclang_rt.asan-x86_64.so")))
        if hits:
            return hits[-1]
    raise RuntimeError("libclang_rt.asan-x86_64.so not found under the ROCm LLVM tree")


def build_hostsan(out: str) -> str:
    cmd = build.command(out)
    cmd[cmd.index("-O3")] = "-O1"
    cmd[1:1] = ["-g", *HOST_SANITIZERS.split()]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed ({res.returncode}):\n{res.stdout}\n{res.stderr}")
    return out


if __name__ == "__main__":
    if sys.argv[1:] == ["--runtime"]:
        print(runtime())
    elif len(sys.argv) == 2:
        print(build_hostsan(os.path.abspath(sys.argv[1])))
    else:
        sys.exit(__doc__)
