"""Compile the C oracle (``mdoracle.c``) into ``oracle/_build/libmdoracle.so``.

Test infrastructure: the library is loaded only by the tests, the smoke check
and the benchmark's CPU-baseline leg.  ``-ffp-contract=off`` keeps every sum
and product separately rounded, which the error-free transformations need.
"""

from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "mdoracle.c")
OUT_DIR = os.path.join(HERE, "_build")
OUT = os.path.join(OUT_DIR, "libmdoracle.so")

CFLAGS = ["-std=c11", "-O2", "-march=x86-64-v2", "-mfma", "-fno-fast-math", "-ffp-contract=off",
          "-fopenmp", "-fPIC", "-shared", "-Wall", "-Wextra", "-Wno-unused-parameter"]


def build(verbose: bool = False) -> str:
    os.makedirs(OUT_DIR, exist_ok=True)
    tmp = OUT + ".tmp"
    cmd = ["gcc", *CFLAGS, "-o", tmp, SRC, "-lm"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, OUT)
    return OUT


# The oracle under AddressSanitizer + UndefinedBehaviorSanitizer, built by clang
# so that it shares one sanitizer runtime with the library's sanitized build;
# without OpenMP (its loops then run on one thread).
SAN_OUT = os.path.join(os.path.dirname(HERE), "_build_san", "libmdoracle.so")
CLANG = "/opt/rocm/llvm/bin/clang"


def build_sanitized(verbose: bool = False) -> str:
    os.makedirs(os.path.dirname(SAN_OUT), exist_ok=True)
    flags = [f for f in CFLAGS if f not in ("-O2", "-fopenmp")] + [
        "-O1", "-g", "-Wno-unknown-pragmas", "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
        "-fno-omit-frame-pointer", "-shared-libasan"]
    cmd = [CLANG, *flags, "-o", SAN_OUT, SRC, "-lm"]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    return SAN_OUT


if __name__ == "__main__":
    print(build_sanitized(verbose=True) if "--sanitize" in sys.argv[1:] else build(verbose=True))
    sys.exit(0)
