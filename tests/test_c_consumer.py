"""The boundary is a C ABI: include/memattn.h compiles as strict C99 (and as
C++17), and a plain C program links libmemattn.so and calls its host-side
entry points (workspace sizes, status strings, argument validation, the
last-error text) without a GPU or Python."""
import os
import shutil
import subprocess

import pytest

import paper_2607_05708_amd as pm

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
INCLUDE = os.path.join(ROOT, "include")
GCC = shutil.which("gcc")
GXX = shutil.which("g++")
pytestmark = pytest.mark.skipif(GCC is None or GXX is None, reason="gcc/g++ not available")

C_PROGRAM = r"""
#include <stdio.h>
#include <string.h>
#include "memattn.h"

int main(void) {
  const size_t ws = mem_workspace_bytes(1024, 1048576, 1024, 32, MEM_BF16);
  if (ws == 0) return 1;
  if (mem_workspace_bytes(16, 1024, 256, 0, MEM_F32) != 0) return 2;  /* k = 0 */
  if (mem_scratch_bytes() == 0) return 3;
  if (strlen(mem_status_string(MEM_ERR_INVALID_ARG)) == 0) return 4;
  /* argument errors come back before any device work */
  int32_t idx[8];
  mem_topk_out out = {idx, NULL, NULL, NULL};
  float emb[4];
  mem_bank bank = {emb, 1, 4, MEM_F32, 4};
  const mem_status st = mem_retrieve_topk(&bank, emb, 1, 4, 2, 1.0f, out, NULL, NULL, 0, NULL);
  if (st != MEM_ERR_INVALID_ARG) return 5;  /* k = 2 > 1 candidate */
  if (strlen(mem_last_error()) == 0) return 6;
  bank.d = 0;
  if (mem_build_relations(&bank, 1, 1.0f, 1, out, NULL, 0, NULL) != MEM_ERR_INVALID_ARG) return 7;
  printf("workspace %zu bytes; last error: %s\n", ws, mem_last_error());
  return 0;
}
"""


def test_header_is_c99_and_cxx17():
    for cmd in ([GCC, "-std=c99", "-Wall", "-Wextra", "-Werror", "-pedantic", "-fsyntax-only", "-x", "c",
                 os.path.join(INCLUDE, "memattn.h")],
                [GXX, "-std=c++17", "-Wall", "-Wextra", "-Werror", "-fsyntax-only", "-x", "c++",
                 os.path.join(INCLUDE, "memattn.h")]):
        r = subprocess.run(cmd, capture_output=True, text=True)
        assert r.returncode == 0, r.stderr


def test_c_program_links_and_validates(tmp_path):
    lib = pm.library_path()
    if not os.path.exists(lib):
        pytest.skip("libmemattn.so is not built")
    src = tmp_path / "consumer.c"
    exe = tmp_path / "consumer"
    src.write_text(C_PROGRAM)
    libdir = os.path.dirname(lib)
    r = subprocess.run([GCC, "-std=c99", "-Wall", "-Wextra", "-Werror", "-pedantic", "-I", INCLUDE, str(src),
                        "-L", libdir, "-lmemattn", f"-Wl,-rpath,{libdir}", "-Wl,-rpath-link,/opt/rocm/lib",
                        "-o", str(exe)], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=60)
    assert r.returncode == 0, (r.returncode, r.stdout, r.stderr)
    assert r.stdout.startswith("workspace ")
