"""Compile ``libmdgemm.so`` (the HIP kernels and the C ABI) for gfx950.

Flags:
* ``--offload-arch=gfx950``: MI355X (CDNA4) code only.
* ``-mllvm -amdgpu-mfma-vgpr-form=1``: keep MFMA accumulators in ordinary
  VGPRs; otherwise the compiler copies loop-carried accumulators between
  AGPRs and VGPRs around every MFMA block, which costs about a third of the
  FP64 matrix-core throughput.
* ``-Xclang -target-feature -Xclang -packed-fp32-ops``: no packed-FP32
  instructions are generated (none of these kernels needs them).

Every kernel of the library is built here from its sources; it links no
vendor BLAS.
"""

from __future__ import annotations

import glob
import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
SOURCES = sorted(glob.glob(os.path.join(HERE, "csrc", "*.hip")))
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(HERE, "libmdgemm.so")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = [
    "--offload-arch=gfx950",
    "-O3",
    "-std=c++17",
    "-fPIC",
    "-shared",
    "-Wall",
    "-Wno-unused-result",
    "-mllvm",
    "-amdgpu-mfma-vgpr-form=1",
    "-Xclang",
    "-target-feature",
    "-Xclang",
    "-packed-fp32-ops",
]


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    proc = subprocess.run(cmd, capture_output=True, text=True)
    noise = "unknown target feature"  # the host pass does not know -packed-fp32-ops
    msgs = [ln for ln in (proc.stdout + proc.stderr).splitlines() if noise not in ln and "packed-fp32-ops" not in ln]
    if proc.returncode != 0:
        raise RuntimeError("hipcc failed:\n" + "\n".join(msgs))
    if verbose and msgs:
        print("\n".join(msgs))


def build(verbose: bool = False) -> str:
    """Compile every source to an object in parallel, then link the library."""
    objdir = os.path.join(HERE, "_build")
    os.makedirs(objdir, exist_ok=True)
    compile_flags = [f for f in FLAGS if f != "-shared"]
    objs = [os.path.join(objdir, os.path.basename(src) + ".o") for src in SOURCES]
    cmds = [[HIPCC, *compile_flags, "-I", INCLUDE, "-I", os.path.join(HERE, "csrc"), "-c", "-o", obj, src]
            for src, obj in zip(SOURCES, objs)]
    with ThreadPoolExecutor(max_workers=min(len(cmds), os.cpu_count() or 1)) as pool:
        for fut in [pool.submit(_run, cmd, verbose) for cmd in cmds]:
            fut.result()
    tmp = LIB + ".tmp"
    _run([HIPCC, "--offload-arch=gfx950", "-fPIC", "-shared", "-o", tmp, *objs], verbose)
    os.replace(tmp, LIB)
    return LIB


# AddressSanitizer and UndefinedBehaviorSanitizer on the host code only (the
# device code is built as usual, unsanitized); run under the clang runtime
# preloaded (tests/run_sanitized.py does this for the CPU tests).
SAN_DIR = os.path.join(ROOT, "_build_san")
SAN_LIB = os.path.join(SAN_DIR, "libmdgemm.so")
SAN_FLAGS = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined", "-Xarch_host",
             "-fno-omit-frame-pointer", "-Xarch_host", "-fno-sanitize-recover=undefined", "-g"]


def build_sanitized(verbose: bool = False) -> str:
    """The library with its host code under ASan + UBSan, in _build_san/."""
    objdir = os.path.join(SAN_DIR, "obj")
    os.makedirs(objdir, exist_ok=True)
    compile_flags = [f for f in FLAGS if f not in ("-shared", "-O3")] + ["-O1", *SAN_FLAGS]
    objs = [os.path.join(objdir, os.path.basename(src) + ".o") for src in SOURCES]
    cmds = [[HIPCC, *compile_flags, "-I", INCLUDE, "-I", os.path.join(HERE, "csrc"), "-c", "-o", obj, src]
            for src, obj in zip(SOURCES, objs)]
    with ThreadPoolExecutor(max_workers=min(len(cmds), os.cpu_count() or 1)) as pool:
        for fut in [pool.submit(_run, cmd, verbose) for cmd in cmds]:
            fut.result()
    _run([HIPCC, "--offload-arch=gfx950", "-fPIC", "-shared", "-Xarch_host", "-fsanitize=address", "-Xarch_host",
          "-fsanitize=undefined", "-shared-libasan", "-o", SAN_LIB, *objs], verbose)
    return SAN_LIB


if __name__ == "__main__":
    if "--sanitize" in sys.argv[1:]:
        print(build_sanitized(verbose=True))
    else:
        print(build(verbose=True))
    sys.exit(0)
