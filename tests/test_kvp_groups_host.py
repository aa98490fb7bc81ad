"""Host check of the block groups of the balanced dK/dV kernel
(`csrc/kvp_groups.h`), compiled with g++ on its own.

For every axis length and odd window: the groups cover every 4-wide key block
exactly once; a block's run of squares is exactly the squares of its query
box; that box holds every query whose border-clamped window (Sec. 3.2) holds a
key of the block (brute force over the axis); the square list of a group is
strictly increasing; and with 9-wide windows the groups fit the staged 4x4
grid exactly when every single block's box does (so the kernel falls back only
where no grouping could fit: axes of 17 to 20 positions).
"""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2606_31248_amd", "csrc")

HARNESS = r"""
#define __host__
#define __device__
#define __forceinline__ inline
#include <algorithm>
#include <cstdio>
#include <vector>
using std::max;
using std::min;
#include "kvp_groups.h"
using namespace strata::kvp;

static int win_start(int q, int L, int k) {  // border-clamped window of query q
  int s = q - k / 2;
  if (s < 0) s = 0;
  if (s > L - k) s = L - k;
  return s;
}

int main() {
  long checks = 0;
  for (int k = 3; k <= 13; k += 2) {
    for (int L = k; L <= 400; ++L) {
      const int nb = (L + 3) / 4;
      std::vector<int> seen(nb, 0);
      bool single_fits = true;  // every block's own box spans at most four squares
      for (int i = 0; i < n_groups(L); ++i) {
        const AxisGroup r = axis_group(i, L, k);
        if (r.nblk < 1 || r.nblk > 2) { printf("L=%d k=%d group %d: %d blocks\n", L, k, i, r.nblk); return 1; }
        for (int e = 1; e < r.n; ++e)
          if (sq_abs(r, e) <= sq_abs(r, e - 1)) { printf("L=%d k=%d group %d: squares not increasing\n", L, k, i); return 1; }
        for (int t = 0; t < r.nblk; ++t) {
          const int b = t ? r.blk1 : r.blk0, run = t ? r.run1 : r.run0, len = t ? r.len1 : r.len0;
          if (b < 0 || b >= nb) { printf("L=%d k=%d group %d: block %d out of range\n", L, k, i, b); return 1; }
          seen[b]++;
          // the block's query box by brute force: every query whose window holds a key of the block
          int lo = L, hi = -1;
          for (int q = 0; q < L; ++q) {
            const int s = win_start(q, L, k);
            for (int j = 4 * b; j < std::min(4 * b + 4, L); ++j)
              if (j >= s && j < s + k) { lo = std::min(lo, q); hi = std::max(hi, q); }
          }
          single_fits = single_fits && hi / 4 - lo / 4 + 1 <= 4;
          if (run < 0 || run + len > r.n || len != hi / 4 - lo / 4 + 1) {
            printf("L=%d k=%d block %d: run %d+%d of %d, box [%d, %d]\n", L, k, b, run, len, r.n, lo, hi);
            return 1;
          }
          for (int u = 0; u < len; ++u)
            if (sq_abs(r, run + u) != lo / 4 + u) { printf("L=%d k=%d block %d: square %d\n", L, k, b, u); return 1; }
          ++checks;
        }
      }
      for (int b = 0; b < nb; ++b)
        if (seen[b] != 1) { printf("L=%d k=%d: block %d in %d groups\n", L, k, b, seen[b]); return 1; }
      const bool fits = groups_fit(L, k, false) && groups_fit(L, k, true);
      if (k == 9 && fits != single_fits) {
        printf("L=%d: groups fit %d, single blocks fit %d\n", L, (int)fits, (int)single_fits);
        return 1;
      }
      if (k == 9 && !fits && (L < 17 || L > 20)) {
        printf("L=%d: 9-wide windows do not fit the staged grid\n", L);
        return 1;
      }
    }
  }
  printf("ok %ld\n", checks);
  return 0;
}
"""


def test_kvp_block_groups(tmp_path):
    gxx = shutil.which("g++")
    if gxx is None:
        pytest.skip("g++ not available")
    src = tmp_path / "kvp_groups_check.cpp"
    exe = tmp_path / "kvp_groups_check"
    src.write_text(HARNESS)
    subprocess.run([gxx, "-O2", "-std=c++17", "-Wall", "-I", CSRC, str(src), "-o", str(exe)], check=True)
    out = subprocess.run([str(exe)], capture_output=True, text=True, timeout=120)
    assert out.returncode == 0, out.stdout + out.stderr
    assert out.stdout.startswith("ok ")
