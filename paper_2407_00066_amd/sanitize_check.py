"""The CPU test suite against sanitizer builds of the host code.

    python -m paper_2407_00066_amd.sanitize_check [pytest args]

Builds libcts.so (host code under AddressSanitizer and
UndefinedBehaviorSanitizer; the device code as always) and the C oracle
(both sanitizers) into a scratch directory with ROCm's clang, then runs
`pytest -m "not gpu"` on them in a child process with the shared sanitizer
runtime preloaded (CTS_LIB and CTS_ORACLE_LIB point the loaders at the
sanitizer builds).  Any sanitizer report ends the run with a nonzero status.
No GPU is used: the CPU tests reach the library's argument checks, plans
and workspace layouts, never a kernel launch.
"""
from __future__ import annotations

import glob
import os
import subprocess
import sys
import tempfile

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)


def runtime() -> str:
    libs = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    if not libs:
        raise RuntimeError("the clang AddressSanitizer runtime is not installed")
    return libs[-1]


def main(argv) -> int:
    sys.path.insert(0, ROOT)
    from oracle import oracle
    from paper_2407_00066_amd import build
    out = tempfile.mkdtemp(prefix="cts_san_")
    lib = build.build(out=os.path.join(out, "libcts.so"), sanitize=True)
    olib = oracle.build(out=os.path.join(out, "libcts_oracle.so"), sanitize=True)
    env = dict(os.environ)
    env.update({
        "CTS_LIB": lib, "CTS_ORACLE_LIB": olib, "LD_PRELOAD": runtime(),
        # Python and torch are not instrumented: their allocations are not leaks of ours
        "ASAN_OPTIONS": "detect_leaks=0:abort_on_error=1:halt_on_error=1",
        "UBSAN_OPTIONS": "halt_on_error=1:print_stacktrace=1",
    })
    cmd = [sys.executable, "-m", "pytest", os.path.join(ROOT, "tests"), "-q", "-m", "not gpu", "-p", "no:cacheprovider"]
    return subprocess.run(cmd + list(argv), env=env, cwd=ROOT).returncode


if __name__ == "__main__":
    sys.exit(main(sys.argv[1:]))
