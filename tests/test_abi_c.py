"""The C ABI from plain C: include/caddtree.h compiles as C (gcc -std=c11), the program links
against libcaddtree.so, and host-side validation and the host-only cost fit run without a GPU."""

import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2606_01813_amd")

C_SRC = r"""
#include <stdio.h>
#include <string.h>
#include "caddtree.h"

int main(void) {
  /* a plan with a decreasing cost table is rejected before any HIP call */
  double tv[4] = {1.0, 2.0, 1.5, 3.0};
  caddtree_config_t cfg;
  memset(&cfg, 0, sizeof(cfg));
  cfg.L = 4; cfg.V = 1024; cfg.K = 4; cfg.budget_cap = 3;
  cfg.dtype = CADDTREE_F32; cfg.mask = CADDTREE_MASK_U8; cfg.flags = 0;
  cfg.t_draft = 1.0; cfg.t_verify_host = tv;
  caddtree_plan_t plan = 0;
  caddtree_status_t st = caddtree_plan_create(&cfg, &plan);
  printf("create %d %s | %s\n", (int)st, caddtree_status_string(st), caddtree_last_error());
  if (st != CADDTREE_E_COST || plan != 0) return 1;
  /* NULL arguments */
  if (caddtree_build(0, 0, 1, 1024, 0, 0, 0, 0, 0, 0) != CADDTREE_E_INVALID) return 2;
  /* host-only convex fit of a profile */
  double x[5] = {1, 2, 3, 4, 5}, y[5] = {1.0, 1.2, 1.1, 1.9, 3.0}, f[5], table[8];
  st = caddtree_fit_cost(x, y, 5, f, 7, table);
  printf("fit %d:", (int)st);
  for (int i = 0; i < 8; ++i) printf(" %.6f", table[i]);
  printf("\n");
  if (st != CADDTREE_OK) return 3;
  for (int i = 2; i < 8; ++i)
    if (table[i] - 2 * table[i - 1] + table[i - 2] < -1e-12) return 4;
  return 0;
}
"""


@pytest.fixture(scope="module")
def binary(tmp_path_factory):
    gcc = shutil.which("gcc")
    if gcc is None:
        pytest.skip("gcc is not available")
    lib = os.path.join(PKG, "libcaddtree.so")
    if not os.path.exists(lib):
        pytest.fail("libcaddtree.so is not built")
    d = tmp_path_factory.mktemp("cabi")
    src = d / "abi.c"
    src.write_text(C_SRC)
    exe = d / "abi"
    cmd = [gcc, "-std=c11", "-Wall", "-Werror", "-D__HIP_PLATFORM_AMD__", "-I", os.path.join(ROOT, "include"),
           "-I", "/opt/rocm/include", str(src), "-L", PKG, "-lcaddtree", f"-Wl,-rpath,{PKG}", "-o", str(exe)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    return exe


def test_header_compiles_and_links_as_c(binary):
    r = subprocess.run([str(binary)], capture_output=True, text=True, timeout=60)
    assert r.returncode == 0, (r.returncode, r.stdout, r.stderr)
    assert "create 3 cost model rejected" in r.stdout


def test_bench_refuses_more_than_one_gpu():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=600)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
