"""Run the CPU tests against AddressSanitizer + UndefinedBehaviorSanitizer builds
of the library's host code and of the C oracle.

    python tests/run_sanitized.py [--no-build] [extra pytest arguments]

Builds both into _build_san/ (hipcc with the sanitizers on the host side only,
the device code as usual; clang for the oracle, so that one sanitizer runtime
serves both), then runs ``pytest -m "not gpu"`` in a child process with the
clang sanitizer runtime preloaded and tests/conftest.py pointing the loaders at
the sanitized libraries.  A sanitizer report aborts the child, which fails the
run.  Nothing here touches a GPU: the CPU tests call only the host entry points
(planning, workspace sizes and layouts, schedules, argument checks, exported
symbols) and the oracle.
"""

from __future__ import annotations

import glob
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

from oracle import build_oracle  # noqa: E402
from paper_2607_06881_amd import build  # noqa: E402


def asan_runtime() -> str:
    libs = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    if not libs:
        raise SystemExit("no clang AddressSanitizer runtime found under /opt/rocm/llvm")
    return libs[-1]


def main(argv: list[str]) -> int:
    if "--no-build" not in argv:
        build.build_sanitized(verbose=True)
        build_oracle.build_sanitized(verbose=True)
    extra = [a for a in argv if a != "--no-build"]
    env = dict(os.environ)
    env.update({
        "LD_PRELOAD": asan_runtime(),
        "MDGEMM_SANITIZED": "1",
        # Python itself keeps objects alive at exit: leak reports would be its own
        "ASAN_OPTIONS": "detect_leaks=0:abort_on_error=1:halt_on_error=1",
        "UBSAN_OPTIONS": "print_stacktrace=1:halt_on_error=1",
    })
    cmd = [sys.executable, "-m", "pytest", os.path.join(ROOT, "tests"), "-m", "not gpu", "-q", "-x",
           "-p", "no:cacheprovider", *extra]
    print(" ".join(cmd), flush=True)
    return subprocess.call(cmd, env=env, cwd=ROOT)


if __name__ == "__main__":
    sys.exit(main(sys.argv[1:]))
