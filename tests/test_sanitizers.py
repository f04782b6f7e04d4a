"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only).

The oracle (g++) and the library's host side (the descriptor checks and enumeration of space
creation, the inter-stage planner, the calibration's window, fit and Algorithm 1; built with
hipcc, sanitizers on the host pass only) are rebuilt with both sanitizers, errors fatal, and
the CPU suites that exercise them run against those builds in a subprocess that preloads the
matching sanitizer runtime.
"""
import glob
import os
import subprocess
import sys
import tempfile

import pytest

from oracle import oracle as O

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
ENV = {"ASAN_OPTIONS": "detect_leaks=0:abort_on_error=1", "UBSAN_OPTIONS": "halt_on_error=1"}


def _run(code, preload, extra_env=None):
    env = dict(os.environ, LD_PRELOAD=preload, **ENV, **(extra_env or {}))
    r = subprocess.run([sys.executable, "-c", code], cwd=ROOT, env=env, capture_output=True, text=True, timeout=900)
    return r.returncode, (r.stdout + r.stderr)[-3000:]


def test_oracle_under_sanitizers():
    runtime = subprocess.run(["g++", "-print-file-name=libasan.so"], capture_output=True, text=True).stdout.strip()
    if not os.path.isabs(runtime):
        pytest.skip("no libasan for g++")
    with tempfile.TemporaryDirectory() as tmp:
        lib = os.path.join(tmp, "liboracle_san.so")
        flags = [f for f in O.CXXFLAGS if f != "-O2"]
        subprocess.run(["g++", "-O1", "-g", *flags, "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
                        O.SRC, "-o", lib], check=True, capture_output=True)
        code = ("import sys, pytest; sys.exit(pytest.main(['-x', '-q', '-p', 'no:cacheprovider', "
                "'tests/test_oracle_pins.py', 'tests/test_oracle_terms.py', 'tests/test_oracle_reduce.py', "
                "'tests/test_oracle_alpha.py', 'tests/test_oracle_pareto.py', 'tests/test_oracle_calib.py', "
                "'tests/test_oracle_flops.py']))")
        rc, out = _run(code, runtime, {"MIST_ORACLE_LIB": lib})
        assert rc == 0, out


def test_library_host_code_under_sanitizers():
    runtimes = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    if not runtimes:
        pytest.skip("no clang AddressSanitizer runtime")
    sys.path.insert(0, ROOT)
    from paper_2503_19050_amd import build as B
    with tempfile.TemporaryDirectory() as tmp:
        lib = os.path.join(tmp, "libmist_san.so")
        B.build(out=lib, extra=["-g", "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                                "-Xarch_host", "-fno-sanitize-recover=all"])
        code = ("import sys; sys.path.insert(0, %r)\n"
                "from paper_2503_19050_amd import mist\n"
                "mist.load(%r)\n"
                "import pytest\n"
                "sys.exit(pytest.main(['-x', '-q', '-p', 'no:cacheprovider', '-m', 'not gpu', "
                "'tests/test_abi.py', 'tests/test_plan.py', 'tests/test_calib.py']))") % (ROOT, lib)
        rc, out = _run(code, runtimes[-1])
        assert rc == 0, out
