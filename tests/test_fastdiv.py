"""Multiply-shift division by invariant integers (the kernels' index
arithmetic): the host/device routine of ``csrc/kernels.hpp`` compiled for the
host with g++ and compared with the integer division it replaces, on edge
cases (powers of two, divisors next to them, dividends at the top of the
32-bit range) and on random pairs."""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(os.path.dirname(HERE), "paper_2401_11471_amd", "csrc")

PROG = r"""
#include <cstdio>
#include <cstdint>
#include <random>
#include <vector>
#include "kernels.hpp"
using namespace lrcnn;
static int bad = 0;
static void check(uint32_t n, uint32_t d) {
  FastDiv f = fast_div(d);
  uint32_t q, r;
  fdiv_qr(n, f, q, r);
  if (q != n / d || r != n % d) {
    if (bad < 10) printf("n=%u d=%u got %u %u\n", n, d, q, r);
    ++bad;
  }
}
int main() {
  std::vector<uint32_t> ds, ns;
  for (uint32_t d = 1; d < 4096; ++d) ds.push_back(d);
  for (int k = 1; k < 31; ++k) {
    uint32_t p = 1u << k;
    ds.push_back(p - 1); ds.push_back(p); ds.push_back(p + 1);
  }
  ds.push_back(0x7fffffffu);
  for (uint32_t n = 0; n < 4096; ++n) ns.push_back(n);
  for (int k = 1; k <= 32; ++k) {
    uint64_t p = 1ull << k;
    ns.push_back((uint32_t)(p - 1)); ns.push_back((uint32_t)(p - 2));
    if (k < 32) ns.push_back((uint32_t)p);
  }
  for (uint32_t d : ds) {
    for (uint32_t n : ns) check(n, d);
    // multiples of d and their neighbours
    for (uint64_t k = 1; k < 64; ++k) {
      uint64_t n = k * d;
      if (n + 1 < (1ull << 32)) { check((uint32_t)n, d); check((uint32_t)(n - 1), d);
                                  check((uint32_t)(n + 1), d); }
    }
  }
  std::mt19937_64 g(7);
  for (int i = 0; i < 4000000; ++i) {
    uint32_t d = (uint32_t)(g() % 0x7fffffffu) + 1;
    if (i & 1) d = (uint32_t)(g() % 100000) + 1;  // divisors of index arithmetic
    check((uint32_t)g(), d);
  }
  printf("bad %d\n", bad);
  return bad != 0;
}
"""


@pytest.mark.skipif(shutil.which("g++") is None, reason="g++ not available")
def test_fast_division_matches_integer_division(tmp_path):
    src = tmp_path / "fd.cpp"
    src.write_text(PROG)
    exe = tmp_path / "fd"
    subprocess.run(["g++", "-O2", "-std=c++17", "-I", CSRC, str(src), "-o", str(exe)],
                   check=True)
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stdout
    assert "bad 0" in r.stdout
