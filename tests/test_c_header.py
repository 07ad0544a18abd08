"""The boundary from plain C: include/wise.h compiles as strict C99 and C++17,
and a C program linked against libwise.so gets the documented answers from
calls that never reach the device (size queries, version, status strings,
and argument errors returned before any launch)."""

import os
import shutil
import subprocess

import pytest

from paper_2609_27373_amd import wise

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
INC = os.path.join(ROOT, "include")

C_SRC = r"""
#include <stdio.h>
#include <string.h>
#include "wise.h"

int main(void) {
  wise_shape s;
  memset(&s, 0, sizeof s);
  s.batch = 1; s.heads = 2; s.seq_len = 512; s.head_dim = 64; s.block = 64;
  if (wise_abi_version() != WISE_ABI_VERSION) return 1;
  if (wise_support_capacity(&s) != 2 * 8 * 9 / 2) return 2;
  if (wise_select_workspace_bytes(&s) == 0) return 3;
  if (wise_mask_words(&s) != 1) return 4;
  if (wise_dense_attn_accum(NULL, 0, 0, 0, 0, 0, 0, 0, 0, 0) != WISE_ERR_NULL) return 5;
  if (wise_sparse_attn(&s, 0, 0, 0, 0, 0, 0, 0, 0, 0) != WISE_ERR_NULL) return 6;
  s.head_dim = 80;
  if (wise_select_support(&s, 0, 0.9f, 3u, 0, 0, 0, 0, 0, 0) != WISE_ERR_UNSUPPORTED) return 7;
  if (wise_support_capacity(&s) != -1) return 8;
  if (strncmp(wise_status_string(WISE_ERR_RANGE), "WISE_ERR_RANGE", 14) != 0) return 9;
  printf("ok\n");
  return 0;
}
"""


@pytest.fixture(scope="module")
def built():
    if not os.path.exists(wise.LIB_PATH):
        from paper_2609_27373_amd import build
        build.build()
    return wise.LIB_PATH


@pytest.mark.skipif(shutil.which("gcc") is None, reason="no C compiler")
def test_c_program_against_the_library(built, tmp_path):
    src = tmp_path / "abi.c"
    src.write_text(C_SRC)
    exe = tmp_path / "abi"
    libdir = os.path.dirname(built)
    subprocess.run(["gcc", "-std=c99", "-Wall", "-Wextra", "-Werror", "-pedantic", "-I", INC,
                    str(src), "-o", str(exe), built, f"-Wl,-rpath,{libdir}"],
                   check=True, capture_output=True, text=True)
    res = subprocess.run([str(exe)], capture_output=True, text=True, timeout=60)
    assert res.returncode == 0 and res.stdout.strip() == "ok", (res.returncode, res.stderr)


@pytest.mark.skipif(shutil.which("g++") is None, reason="no C++ compiler")
def test_header_compiles_as_cpp(tmp_path):
    src = tmp_path / "h.cpp"
    src.write_text('#include "wise.h"\nint main() { return wise_abi_version() > 0 ? 0 : 1; }\n')
    subprocess.run(["g++", "-std=c++17", "-Wall", "-Wextra", "-Werror", "-fsyntax-only", "-I", INC,
                    str(src)], check=True, capture_output=True, text=True)
