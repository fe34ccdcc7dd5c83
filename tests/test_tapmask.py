"""Tap-window masks of the convolution loaders: the host/device routine of
``csrc/kernels.hpp`` compiled for the host with g++ and compared bit by bit
with a brute-force test of every tap. A row at tap-0 position (by, bx)
reads source (by + ti, bx + tj) in the forward and (by - ti, bx - tj) in
the input gradient. A tap's bit is set exactly when that position lies in
rows [sy0, sy1) and columns [0, Ws). Covered: every kernel shape up to 8x8
(64 taps: the mask's last bit), plus 1 x 63 and 63 x 1. Rows and columns
run far outside the window on both sides, windows can be empty, and
random cases are added."""
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
static long bad = 0, n = 0;
static void check(int by, int bx, int kh, int kw, int sy0, int sy1, int Ws, bool mir) {
  const uint64_t m = tap_window_mask(by, bx, kh, kw, sy0, sy1, Ws, mir);
  uint64_t want = 0;
  for (int ti = 0; ti < kh; ++ti)
    for (int tj = 0; tj < kw; ++tj) {
      const int sy = mir ? by - ti : by + ti, sx = mir ? bx - tj : bx + tj;
      if (sy >= sy0 && sy < sy1 && sx >= 0 && sx < Ws) want |= 1ull << (ti * kw + tj);
    }
  ++n;
  if (m != want) {
    if (bad < 10)
      printf("by=%d bx=%d k=%dx%d rows [%d,%d) Ws=%d mir=%d: %llx want %llx\n", by, bx, kh, kw,
             sy0, sy1, Ws, (int)mir, (unsigned long long)m, (unsigned long long)want);
    ++bad;
  }
}
int main() {
  for (int kh = 1; kh <= 8; ++kh)
    for (int kw = 1; kw <= 8; ++kw)
      for (int mir = 0; mir < 2; ++mir)
        for (int sy0 = 0; sy0 <= 3; ++sy0)
          for (int sy1 = sy0; sy1 <= sy0 + 6; ++sy1)
            for (int Ws = 1; Ws <= 6; ++Ws)
              for (int by = -10; by <= 12; ++by)
                for (int bx = -10; bx <= 12; ++bx) check(by, bx, kh, kw, sy0, sy1, Ws, mir);
  for (int mir = 0; mir < 2; ++mir)
    for (int by = -70; by <= 70; by += 3)
      for (int bx = -70; bx <= 70; bx += 3) {
        check(by, bx, 1, 63, 0, 5, 40, mir);
        check(by, bx, 63, 1, -3, 40, 5, mir);
      }
  std::mt19937 g(11);
  for (int i = 0; i < 2000000; ++i) {
    int kh = 1 + g() % 8, kw = 1 + g() % 8;
    int sy0 = (int)(g() % 200) - 50, sy1 = sy0 + (int)(g() % 120);
    int Ws = 1 + g() % 300;
    int by = (int)(g() % 500) - 100, bx = (int)(g() % 500) - 100;
    check(by, bx, kh, kw, sy0, sy1, Ws, g() & 1);
  }
  printf("cases %ld bad %ld\n", n, bad);
  return bad != 0;
}
"""


@pytest.mark.skipif(shutil.which("g++") is None, reason="g++ not available")
def test_tap_window_mask_matches_brute_force(tmp_path):
    src = tmp_path / "tm.cpp"
    src.write_text(PROG)
    exe = tmp_path / "tm"
    subprocess.run(["g++", "-O2", "-std=c++17", "-I", str(CSRC), str(src), "-o", str(exe)],
                   check=True)
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stdout
    assert " bad 0" in r.stdout
