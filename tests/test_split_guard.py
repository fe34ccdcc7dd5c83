"""The split-K buffer guard of the launchers, compiled for the host from
``csrc/kernels.hpp`` with g++ (the same inline routines the launchers call
before every launch).

A split launch writes splits x M x N float32 partial sums. An earlier
microbenchmark forced a split whose partial sums were larger than the
buffer it was given, and the kernel wrote past it (an illegal memory
access on the GPU). Every launcher now refuses such a launch before it is
enqueued (``split_fits``), and the split counts the launchers choose never
need more than the buffer they are given. Checked here:

* ``split_fits`` refuses a split whose partial sums exceed the buffer by
  one element, a null buffer and an M x N that does not index in 32 bits,
  and accepts the exact size;
* over random launch shapes and buffer sizes, the split chosen by the
  convolution and weight-gradient estimates always passes the guard;
* the forced split counts (the layer's fixed forward count) are accepted
  by ``split_valid`` only when no smaller count gives the same chunks, and
  an oversized forced split is refused.
"""
import shutil
import subprocess
from pathlib import Path

import pytest

CSRC = Path(__file__).resolve().parent.parent / "paper_2401_11471_amd" / "csrc"

PROG = r"""
#include <cstdio>
#include <cstdint>
#include <random>
#include "kernels.hpp"
using namespace lrcnn;
static long bad = 0;
#define CHECK(c) do { if (!(c)) { ++bad; if (bad < 20) printf("failed: %s (line %d)\n", #c, __LINE__); } } while (0)
int main() {
  char buf[16];
  const void *p = buf;
  // exact fit, one element short, null, 32-bit index limit
  CHECK(split_fits(1, 1000, 1000, nullptr, 0));
  CHECK(split_fits(2, 128, 256, p, 2ull * 128 * 256 * 4));
  CHECK(!split_fits(2, 128, 256, p, 2ull * 128 * 256 * 4 - 4));
  CHECK(!split_fits(2, 128, 256, nullptr, 1ull << 40));
  CHECK(!split_fits(2, 1ll << 20, 1ll << 12, p, 1ull << 50));
  CHECK(split_fits(2, (1ll << 20) - 1, 1ll << 12, p, 1ull << 50));
  // the fault case: a 128 x 256 tile launch forced to split 2 with a
  // buffer sized for one split
  CHECK(!split_fits(2, 128, 256, p, 128ull * 256 * 4));
  std::mt19937 g(7);
  long n = 0;
  for (int it = 0; it < 200000; ++it) {
    const long long M = 1 + g() % 400000;
    const int N = 1 + g() % 2048;
    const int KT = 1 + g() % 600;
    const size_t cap = (size_t)(g() % (64u << 20));
    const int es = (g() & 1) ? 2 : 4;
    const ConvTiles ct = conv_tiles(M, N, KT, cap, es);
    CHECK(ct.splits >= 1 && split_valid(KT, ct.splits));
    CHECK(split_fits(ct.splits, M, N, p, cap) || (long long)M * N >= (1ll << 32));
    const int Co = 1 + g() % 2048;
    const long long Nw = 1 + g() % 20000, K = 1 + g() % 2000000;
    const WgradTiles wt = wgrad_tiles(Co, Nw, K, cap, es);
    CHECK(split_fits(wt.splits, Co, Nw, p, cap));
    // a forced split: valid counts only, and the guard decides the buffer
    const int s = 1 + g() % 130;
    if (split_valid(KT, s)) {
      const long long kts = (KT + s - 1) / s;
      CHECK(s == 1 || ((KT + kts - 1) / kts == s && s <= KT / 2));
      const size_t need = (size_t)s * (size_t)M * (size_t)N * 4;
      if (s > 1 && (long long)M * N < (1ll << 32)) {
        CHECK(split_fits(s, M, N, p, need));
        CHECK(!split_fits(s, M, N, p, need - 1));
      }
    }
    ++n;
  }
  printf("cases %ld bad %ld\n", n, bad);
  return bad != 0;
}
"""


@pytest.mark.skipif(shutil.which("g++") is None, reason="g++ not available")
def test_split_guard_refuses_oversized_partials(tmp_path):
    src = tmp_path / "sg.cpp"
    src.write_text(PROG)
    exe = tmp_path / "sg"
    subprocess.run(["g++", "-O2", "-std=c++17", "-I", str(CSRC), str(src), "-o", str(exe)],
                   check=True)
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stdout
    assert " bad 0" in r.stdout
