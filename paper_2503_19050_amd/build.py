"""Builds libmist.so (HIP, gfx950) in-tree with hipcc."""

from __future__ import annotations

import concurrent.futures
import os
import subprocess
import sys
import tempfile

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libmist.so")
SOURCES = [os.path.join(CSRC, "mist_host.cpp"), os.path.join(CSRC, "mist_plan.cpp"),
           os.path.join(CSRC, "mist_calib.cpp"), os.path.join(CSRC, "mist_kernels.hip"),
           os.path.join(CSRC, "mist_exact.hip"), os.path.join(CSRC, "mist_corun.hip"),
           os.path.join(CSRC, "mist_probe.hip"), os.path.join(CSRC, "mist_noalloc.hip")]
LIBS = ["-lrocblas"]  # the calibration's GEMMs
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


def build(out: str = LIB, extra: list[str] | None = None, verbose: bool = False,
          sources: list[str] | None = None, include: list[str] | None = None) -> str:
    """Compiles the library (every source in its own hipcc process, in parallel) and links it;
    always rebuilds."""
    tmp = out + ".tmp%d" % os.getpid()
    srcs = sources or SOURCES
    inc = [a for d in (include or [CSRC]) + [INCLUDE] for a in ("-I", d)]
    with tempfile.TemporaryDirectory(prefix="mist_build_") as objdir:
        def compile_one(i_src):
            i, src = i_src
            obj = os.path.join(objdir, "%d_%s.o" % (i, os.path.basename(src)))
            cmd = ["hipcc", *FLAGS, *(extra or []), *inc, "-c", src, "-o", obj]
            cmd.remove("-shared")
            if verbose:
                print(" ".join(cmd), file=sys.stderr)
            subprocess.run(cmd, check=True)
            return obj
        with concurrent.futures.ThreadPoolExecutor(max_workers=len(srcs)) as ex:
            objs = list(ex.map(compile_one, enumerate(srcs)))
        cmd = ["hipcc", *FLAGS, *(extra or []), *objs, *LIBS, "-o", tmp]
        if verbose:
            print(" ".join(cmd), file=sys.stderr)
        subprocess.run(cmd, check=True)
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    print(build(verbose=True))
