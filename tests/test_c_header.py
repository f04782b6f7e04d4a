"""The boundary is plain C: include/mist.h compiles as C99 with every warning an error, and a C
program that takes the address of every entry point the header declares links against the
built libmist.so and runs the host-side checks without a GPU (null and invalid descriptors are
rejected with MIST_E_INVALID and a message, destroying a null space is a no-op)."""
import os
import re
import shutil
import subprocess

import pytest

from paper_2503_19050_amd import mist

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
INCLUDE = os.path.join(ROOT, "include")
HEADER = os.path.join(INCLUDE, "mist.h")

pytestmark = pytest.mark.skipif(shutil.which("gcc") is None, reason="no gcc")


def _declared():
    with open(HEADER) as f:
        return sorted(set(re.findall(r"\b(mist_[a-z0-9_]+)\s*\(", f.read())))


def test_header_is_c99():
    subprocess.run(["gcc", "-std=c99", "-Wall", "-Wextra", "-pedantic", "-Werror", "-fsyntax-only", "-x", "c",
                    HEADER], check=True)


PROGRAM = r"""
#include <stdio.h>
#include <string.h>
#include "mist.h"

typedef void (*any_fn)(void);
static any_fn volatile entry_points[] = {%s};

int main(void) {
  mist_model_desc m;
  mist_hw_desc hw;
  mist_space_desc s;
  mist_space* S = NULL;
  const char* msg;
  size_t i;
  for (i = 0; i < sizeof entry_points / sizeof entry_points[0]; ++i)
    if (!entry_points[i]) return 10;
  if (mist_space_create(NULL, NULL, 0, NULL, NULL, &S) != MIST_E_INVALID || S) return 1;
  msg = mist_last_error();
  if (!msg || !*msg) return 2;
  memset(&m, 0, sizeof m);
  memset(&hw, 0, sizeof hw);
  memset(&s, 0, sizeof s);
  if (mist_space_create(&m, &hw, 1, &s, NULL, &S) != MIST_E_INVALID || S) return 3;
  msg = mist_last_error();
  if (!msg || !*msg) return 4;
  if (mist_space_destroy(NULL) != MIST_OK) return 5;
  printf("ok %%u entry points: %%s\n", (unsigned)(sizeof entry_points / sizeof entry_points[0]), msg);
  return 0;
}
"""


def test_c_program_links_and_validates(tmp_path):
    lib = mist.LIB_PATH
    if not os.path.exists(lib):
        pytest.skip("libmist.so is not built")
    names = _declared()
    src = tmp_path / "abi.c"
    src.write_text(PROGRAM % ", ".join("(any_fn)%s" % n for n in names))
    exe = tmp_path / "abi"
    libdir = os.path.dirname(lib)
    subprocess.run(["gcc", "-std=c99", "-Wall", "-Wextra", "-pedantic", "-Werror", "-I", INCLUDE, str(src),
                    "-o", str(exe), "-L", libdir, "-lmist", "-Wl,-rpath," + libdir], check=True)
    env = dict(os.environ, HIP_VISIBLE_DEVICES="")
    r = subprocess.run([str(exe)], capture_output=True, text=True, env=env, timeout=120)
    assert r.returncode == 0, (r.returncode, r.stdout, r.stderr)
    assert r.stdout.startswith("ok %d entry points" % len(names)), r.stdout
