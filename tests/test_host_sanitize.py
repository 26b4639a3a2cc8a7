"""The host code of the library under AddressSanitizer and UndefinedBehaviorSanitizer (CPU, no GPU).

api.cpp (plan validation, argument checks, workspace sizing) and costfit.cpp (the active-set
least-squares fit) are compiled with g++ -fsanitize=address,undefined and linked, with the
kernels' objects of the normal build, into a test program that drives every host path it can
reach without a GPU: every plan-validation error, NULL and bad arguments of every entry point,
workspace sizing, and cost fits of noisy profiles of many sizes, including degenerate ones.
Any sanitizer report fails the test.
"""

import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2606_01813_amd")
CSRC = os.path.join(PKG, "csrc")

DRIVER = r"""
#include <cmath>
#include <cstdio>
#include <cstring>
#include <random>
#include <vector>
#include "caddtree.h"

static int fails = 0;
#define EXPECT(c) do { if (!(c)) { std::printf("FAILED line %d: %s\n", __LINE__, #c); ++fails; } } while (0)

static caddtree_config_t base(std::vector<double>& tv, int cap) {
  tv.resize((size_t)cap + 1);
  for (int n = 0; n <= cap; ++n) tv[n] = 1.0 + 0.002 * n + 0.00002 * n * n;
  caddtree_config_t c;
  std::memset(&c, 0, sizeof(c));
  c.L = 16; c.V = 151936; c.K = 8; c.budget_cap = cap; c.dtype = CADDTREE_BF16; c.mask = CADDTREE_MASK_U8;
  c.t_draft = 1.0; c.t_verify_host = tv.data();
  return c;
}

static caddtree_status_t create(const caddtree_config_t& c) {
  caddtree_plan_t p = nullptr;
  caddtree_status_t st = caddtree_plan_create(&c, &p);
  if (p) caddtree_plan_destroy(p);
  EXPECT(std::strlen(caddtree_status_string(st)) > 0);
  return st;
}

int main() {
  std::vector<double> tv;
  // plan validation: each bad field is rejected before any HIP call
  { auto c = base(tv, 512); c.L = 0; EXPECT(create(c) == CADDTREE_E_INVALID); }
  { auto c = base(tv, 512); c.L = 33; EXPECT(create(c) == CADDTREE_E_UNSUPPORTED); }
  { auto c = base(tv, 512); c.K = 17; EXPECT(create(c) == CADDTREE_E_UNSUPPORTED); }
  { auto c = base(tv, 512); c.V = 3; c.K = 4; EXPECT(create(c) == CADDTREE_E_INVALID); }
  { auto c = base(tv, 4096); c.budget_cap = 4097; EXPECT(create(c) == CADDTREE_E_UNSUPPORTED); }
  { auto c = base(tv, 512); c.dtype = (caddtree_dtype_t)9; EXPECT(create(c) == CADDTREE_E_INVALID); }
  { auto c = base(tv, 512); c.flags = 8; EXPECT(create(c) == CADDTREE_E_INVALID); }
  { auto c = base(tv, 512); c.t_draft = NAN; EXPECT(create(c) == CADDTREE_E_COST); }
  { auto c = base(tv, 512); tv[100] = tv[99] - 1.0; EXPECT(create(c) == CADDTREE_E_COST); }
  { auto c = base(tv, 512); tv[200] += 0.5; EXPECT(create(c) == CADDTREE_E_COST); }          // a kink: concave
  { auto c = base(tv, 512); tv[7] = INFINITY; EXPECT(create(c) == CADDTREE_E_COST); }
  { auto c = base(tv, 512); c.n_ctx = 65; EXPECT(create(c) == CADDTREE_E_UNSUPPORTED); }
  { auto c = base(tv, 512); c.n_ctx = 3; EXPECT(create(c) == CADDTREE_E_INVALID); }         // grid missing
  {
    std::vector<double> t3(3 * 33);
    for (int j = 0; j < 3; ++j) for (int n = 0; n <= 32; ++n) t3[j * 33 + n] = 1.0 + (0.1 + j) * n;
    int64_t grid[3] = {0, 1000, 1000};
    auto c = base(tv, 32); c.t_verify_host = t3.data(); c.n_ctx = 3; c.ctx_grid_host = grid;
    EXPECT(create(c) == CADDTREE_E_INVALID);                                                  // not increasing
    grid[2] = 2000;
    caddtree_status_t st = create(c);
    EXPECT(st == CADDTREE_OK || st == CADDTREE_E_HIP);                                        // no GPU here
  }
  for (int cap : {0, 1, 31, 512, 4096}) {                     // valid plans pass validation
    auto c = base(tv, cap);
    caddtree_status_t st = create(c);
    EXPECT(st == CADDTREE_OK || st == CADDTREE_E_HIP);
    c.flags = CADDTREE_FIXED_BUDGET;
    st = create(c);
    EXPECT(st == CADDTREE_OK || st == CADDTREE_E_HIP);
  }
  EXPECT(caddtree_plan_create(nullptr, nullptr) == CADDTREE_E_INVALID);
  caddtree_plan_destroy(nullptr);
  EXPECT(caddtree_workspace_bytes(nullptr, 10) == 0);
  // every entry point with a NULL plan
  EXPECT(caddtree_build(nullptr, nullptr, 1, 1024, 0, nullptr, nullptr, nullptr, 0, nullptr) == CADDTREE_E_INVALID);
  EXPECT(caddtree_build_noalloc(nullptr, nullptr, 1, 1024, 0, nullptr, nullptr, nullptr) == CADDTREE_E_INVALID);
  EXPECT(caddtree_reduce_topk(nullptr, nullptr, 1, 1024, nullptr, nullptr, nullptr, nullptr, nullptr) ==
         CADDTREE_E_INVALID);
  EXPECT(caddtree_expand(nullptr, nullptr, nullptr, nullptr, 1, nullptr, nullptr, nullptr, nullptr, nullptr, nullptr,
                         nullptr, nullptr, nullptr) == CADDTREE_E_INVALID);
  EXPECT(caddtree_emit(nullptr, nullptr, nullptr, nullptr, 1, 0, nullptr, nullptr, nullptr) == CADDTREE_E_INVALID);
  EXPECT(caddtree_accept(nullptr, nullptr, nullptr, nullptr, 1, nullptr, nullptr, 8, nullptr, nullptr, nullptr, nullptr,
                         nullptr, nullptr) == CADDTREE_E_INVALID);
  EXPECT(std::strlen(caddtree_last_error()) > 0);
  for (int s = 0; s < 8; ++s) EXPECT(caddtree_status_string((caddtree_status_t)s) != nullptr);

  // the cost fit: error paths
  double x[4] = {1, 2, 2, 3}, y[4] = {1, 2, 3, 4}, f[4], tab[9];
  EXPECT(caddtree_fit_cost(x, y, 4, f, 8, tab) == CADDTREE_E_INVALID);          // x not increasing
  EXPECT(caddtree_fit_cost(nullptr, y, 4, f, 8, tab) == CADDTREE_E_INVALID);
  EXPECT(caddtree_fit_cost(x, y, 0, f, 8, tab) == CADDTREE_E_INVALID);
  x[2] = 2.5; y[1] = NAN;
  EXPECT(caddtree_fit_cost(x, y, 4, f, 8, tab) == CADDTREE_E_INVALID);
  y[1] = 2.0;
  EXPECT(caddtree_fit_cost(x, y, 4, f, 4097, tab) == CADDTREE_E_INVALID);
  // fits of noisy convex profiles of many sizes (and a constant and a single point)
  std::mt19937_64 rng(7);
  std::normal_distribution<double> noise(0.0, 1.0);
  for (int N : {1, 2, 3, 7, 64, 257, 1024, 3000}) {
    for (int rep = 0; rep < 3; ++rep) {
      std::vector<double> xs(N), ys(N), fit(N), table(1025);
      for (int j = 0; j < N; ++j) {
        xs[j] = 1.0 + j * (rep + 1);
        const double t = xs[j];
        ys[j] = rep == 2 ? 5.0 : 2.0 + 0.01 * t + 1e-5 * t * t + (rep == 0 ? 0.05 : 0.5) * noise(rng);
      }
      caddtree_status_t st = caddtree_fit_cost(xs.data(), ys.data(), N, fit.data(), 1024, table.data());
      EXPECT(st == CADDTREE_OK);
      for (int n = 2; n <= 1024; ++n) EXPECT(table[n] - 2 * table[n - 1] + table[n - 2] > -1e-9 * (1 + std::fabs(table[n])));
      for (int n = 1; n <= 1024; ++n) EXPECT(table[n] >= table[n - 1] - 1e-9 * (1 + std::fabs(table[n])));
      EXPECT(caddtree_fit_cost(xs.data(), ys.data(), N, nullptr, 0, nullptr) == CADDTREE_OK);
    }
  }
  std::printf("host checks done, %d failures\n", fails);
  return fails == 0 ? 0 : 1;
}
"""


@pytest.fixture(scope="module")
def sanitized(tmp_path_factory):
    gxx = shutil.which("g++")
    if gxx is None:
        pytest.skip("g++ is not available")
    objs = os.path.join(PKG, "_build")
    from paper_2606_01813_amd import _build
    device_objs = [os.path.join(objs, os.path.splitext(n)[0] + ".o") for n in _build.SOURCES if n.endswith(".hip")]
    missing = [o for o in device_objs if not os.path.exists(o)]
    if missing:
        pytest.fail(f"build the library first (python -m paper_2606_01813_amd._build): {missing}")
    d = tmp_path_factory.mktemp("asan")
    (d / "driver.cpp").write_text(DRIVER)
    inc = ["-D__HIP_PLATFORM_AMD__", "-I", os.path.join(ROOT, "include"), "-I", CSRC, "-I", "/opt/rocm/include"]
    san = ["-fsanitize=address,undefined", "-fno-sanitize-recover=undefined", "-fno-omit-frame-pointer"]
    built = []
    for src in ("api.cpp", "costfit.cpp", str(d / "driver.cpp")):
        path = src if os.path.isabs(src) else os.path.join(CSRC, src)
        obj = str(d / (os.path.basename(src) + ".o"))
        cmd = [gxx, "-std=c++17", "-O1", "-g", "-fPIC", "-Wall"] + san + inc + ["-c", path, "-o", obj]
        r = subprocess.run(cmd, capture_output=True, text=True)
        assert r.returncode == 0, r.stderr
        built.append(obj)
    exe = str(d / "host_asan")
    cmd = [gxx] + san + built + device_objs + ["-L", "/opt/rocm/lib", "-lamdhip64", "-Wl,-rpath,/opt/rocm/lib",
                                               "-o", exe]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    return exe


def test_host_code_is_clean_under_asan_and_ubsan(sanitized):
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:halt_on_error=1:abort_on_error=0",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1", HIP_VISIBLE_DEVICES="")
    r = subprocess.run([sanitized], capture_output=True, text=True, timeout=300, env=env)
    out = r.stdout + r.stderr
    assert "ERROR: AddressSanitizer" not in out and "runtime error" not in out, out[-4000:]
    assert r.returncode == 0, out[-4000:]
    assert "host checks done, 0 failures" in r.stdout
