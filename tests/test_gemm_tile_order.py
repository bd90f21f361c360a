"""The GEMM grid's tile order (csrc/gemm_sched.h), checked on the CPU.

The header is compiled as host C++ with g++ and every work index of every
grid with 1..200 tile rows, 1..60 tile columns and bands of 0..9 tile rows is
mapped: each tile must be hit exactly once and never outside the grid (a tile
outside it would address memory outside A, B or the output), row-major order
must come back with no bands, and within a band consecutive work indices must
walk down a column before moving to the next one.
"""
import os
import shutil
import subprocess

import pytest

CSRC = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "paper_2607_21291_amd", "csrc")

CHECK = r"""
#define DSF_HD
#include "gemm_sched.h"
#include <cstdio>
#include <vector>
int main() {
  long cases = 0;
  for (int ntm = 1; ntm <= 200; ++ntm)
    for (int ntn = 1; ntn <= 60; ++ntn)
      for (int gm = 0; gm <= 9; ++gm) {
        const int W = ntm * ntn;
        std::vector<char> seen(W, 0);
        for (int i = 0; i < W; ++i) {
          const dsf::GemmTile t = dsf::gemm_tile(i, ntm, ntn, gm);
          if (t.tm < 0 || t.tm >= ntm || t.tn < 0 || t.tn >= ntn) { printf("outside %d %d %d %d\n", ntm, ntn, gm, i); return 1; }
          if (seen[t.tm * ntn + t.tn]++) { printf("twice %d %d %d %d\n", ntm, ntn, gm, i); return 1; }
          if (gm == 0 && (t.tm != i / ntn || t.tn != i % ntn)) { printf("row-major %d %d %d\n", ntm, ntn, i); return 1; }
          if (gm > 0 && i > 0 && (i % (gm * ntn)) != 0) {
            const dsf::GemmTile p = dsf::gemm_tile(i - 1, ntm, ntn, gm);
            const bool down = p.tn == t.tn && t.tm == p.tm + 1;
            const int m0 = i / (gm * ntn) * gm, ge = ntm - m0 < gm ? ntm - m0 : gm;
            const bool next_col = t.tn == p.tn + 1 && t.tm == m0 && p.tm == m0 + ge - 1;
            if (!down && !next_col) { printf("band order %d %d %d %d\n", ntm, ntn, gm, i); return 1; }
          }
        }
        ++cases;
      }
  printf("ok %ld\n", cases);
  return 0;
}
"""


def test_gemm_tile_order_is_a_banded_bijection(tmp_path):
    cxx = shutil.which("g++") or shutil.which("c++")
    if cxx is None:
        pytest.skip("no host C++ compiler")
    src = tmp_path / "check.cpp"
    src.write_text(CHECK)
    exe = tmp_path / "check"
    subprocess.run([cxx, "-O2", "-std=c++17", "-I", CSRC, str(src), "-o", str(exe)], check=True)
    out = subprocess.run([str(exe)], capture_output=True, text=True, timeout=120)
    assert out.returncode == 0, out.stdout + out.stderr
    assert out.stdout.strip() == "ok 120000"
