"""Builds libmist.so (HIP, gfx950) in-tree with hipcc."""

from __future__ import annotations

import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libmist.so")
SOURCES = [os.path.join(CSRC, "mist_host.cpp"), os.path.join(CSRC, "mist_plan.cpp"),
           os.path.join(CSRC, "mist_kernels.hip"), os.path.join(CSRC, "mist_exact.hip")]
HEADERS = [os.path.join(CSRC, "mist_internal.h"), os.path.join(INCLUDE, "mist.h")]

ARCH = "gfx950"
FLAGS = [
    "-O3", "-std=c++17", "-fPIC", "-shared",
    f"--offload-arch={ARCH}",
    # The cost model is a fixed sequence of IEEE binary64 operations: no contraction of
    # a*b+c into fma unless written, no fast-math.
    "-ffp-contract=off", "-fno-fast-math",
    # No packed FP32 instructions in device code.
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wextra", "-Wno-unused-parameter",
]


def build(out: str = LIB, extra: list[str] | None = None, verbose: bool = False) -> str:
    """Compiles the library; always rebuilds."""
    tmp = out + ".tmp%d" % os.getpid()
    cmd = ["hipcc", *FLAGS, *(extra or []), "-I", INCLUDE, "-I", CSRC, *SOURCES, "-o", tmp]
    if verbose:
        print(" ".join(cmd), file=sys.stderr)
    subprocess.run(cmd, check=True)
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    print(build(verbose=True))
