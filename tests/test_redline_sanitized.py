"""The host-only Redline C++ (selection, budget sweep, split exceedance,
Monte Carlo) built on its own with AddressSanitizer and UndefinedBehavior-
Sanitizer and driven on random and boundary inputs, including every
argument error: no memory error, no undefined behaviour, and the same
selections as the shipped library."""
import os
import shutil
import subprocess

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

DRIVER = r'''
#include <stdio.h>
#include <stdlib.h>
#include <string>
#include "bd.h"
namespace bd { void set_error(const char* msg); }
static std::string g;
void bd::set_error(const char* msg) { g = msg; }
int main(int argc, char** argv) {
  unsigned s = 12345;
  auto rnd = [&]() { s = s * 1103515245u + 12345u; return (s >> 8) & 0xffff; };
  long checksum = 0;
  for (int trial = 0; trial < 60; ++trial) {
    const int n = 1 + rnd() % 300, m = 1 + rnd() % 9, ref = rnd() % m;
    unsigned char* c = (unsigned char*)malloc((size_t)n * m);
    for (int i = 0; i < n * m; ++i) c[i] = (rnd() % 10) < 8;
    for (int i = 0; i < n; ++i) c[ref * n + i] = 1;
    double* cost = (double*)malloc(sizeof(double) * m);
    for (int j = 0; j < m; ++j) cost[j] = 1.0 + (rnd() % 100) / 10.0;
    int* order = (int*)malloc(sizeof(int) * m);
    for (int j = 0; j < m; ++j) order[j] = m - 1 - j;
    int* V = (int*)malloc(sizeof(int) * m);
    double* p = (double*)malloc(sizeof(double) * m);
    unsigned char* valid = (unsigned char*)malloc(m);
    int sel = -1, ties = 0;
    if (rl_risk_select(n, m, ref, c, cost, 0.1, 0.1, V, p, valid, &sel, &ties) != BD_OK) return 2;
    checksum += sel;
    for (int meth = 0; meth < 5; ++meth) {
      unsigned char* mask = (unsigned char*)malloc(n);
      for (int i = 0; i < n; ++i) mask[i] = (i % 3) != 1 || n < 3;
      if (rl_select(n, m, ref, c, mask, cost, 0.05, 0.1, meth, order, V, p, valid, &sel) != BD_OK) return 3;
      checksum += sel;
      free(mask);
    }
    double alphas[4] = {0.2, 0.05, 0.1, 0.3};
    int sels[4], nv[4];
    double hat = 0;
    if (rl_alpha_sweep(n, m, ref, c, cost, alphas, 4, 0.1, 0, order, sels, nv, &hat) != BD_OK) return 4;
    if (n >= 2) {
      const int ns = 7;
      unsigned char* cal = (unsigned char*)malloc((size_t)ns * n);
      for (int k = 0; k < ns; ++k)
        for (int i = 0; i < n; ++i) cal[k * n + i] = ((i + k) % 2) == 0;
      int dep[ns], tv[ns], counts[4];
      double gain = 0;
      if (rl_split_exceedance(n, m, ref, c, cost, 0.1, 0.1, 0, order, ns, cal, dep, tv, counts, &gain) != BD_OK) return 5;
      free(cal);
    }
    double risk[9];
    for (int j = 0; j < m; ++j) risk[j] = (rnd() % 20) / 100.0;
    const int trials = 5, kk = (trial % 2) ? m : 1;
    double* u = (double*)malloc(sizeof(double) * trials * kk * n);
    for (int i = 0; i < trials * kk * n; ++i) u[i] = rnd() / 65536.0;
    int ft = 0, vc[9];
    if (rl_monte_carlo(n, m, risk, 0.1, 0.1, trial % 5, order, trials, kk, u, &ft, vc) != BD_OK) return 6;
    free(u); free(c); free(cost); free(order); free(V); free(p); free(valid);
  }
  // argument errors return BD_EINVAL without touching the outputs
  unsigned char c1[4] = {1, 1, 1, 1};
  double cost1[2] = {1, 2};
  int sel = 0;
  if (rl_risk_select(0, 2, 0, c1, cost1, 0.1, 0.1, 0, 0, 0, &sel, 0) != BD_EINVAL) return 7;
  if (rl_risk_select(2, 2, 2, c1, cost1, 0.1, 0.1, 0, 0, 0, &sel, 0) != BD_EINVAL) return 8;
  if (rl_risk_select(2, 2, 0, c1, cost1, 1.5, 0.1, 0, 0, 0, &sel, 0) != BD_EINVAL) return 9;
  if (rl_select(2, 2, 0, c1, 0, cost1, 0.1, 0.1, 2, 0, 0, 0, 0, &sel) != BD_EINVAL) return 10;
  unsigned char none[2] = {0, 0};
  if (rl_select(2, 2, 0, c1, none, cost1, 0.1, 0.1, 0, 0, 0, 0, 0, &sel) != BD_EINVAL) return 11;
  printf("ok %ld\n", checksum);
  return 0;
}
'''


@pytest.mark.skipif(shutil.which("g++") is None, reason="no g++")
def test_redline_host_code_under_sanitizers(tmp_path):
    src = tmp_path / "driver.cpp"
    src.write_text(DRIVER)
    exe = tmp_path / "driver"
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           "-I", os.path.join(ROOT, "include"), str(src),
           os.path.join(ROOT, "paper_2609_33887_amd", "csrc", "bd_redline.cpp"), "-o", str(exe), "-lpthread"]
    subprocess.run(cmd, check=True, capture_output=True, text=True)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:verify_asan_link_order=0",
               UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([str(exe)], capture_output=True, text=True, env=env, timeout=600)
    assert r.returncode == 0, (r.returncode, r.stdout[-2000:], r.stderr[-4000:])
    assert r.stdout.startswith("ok ")
