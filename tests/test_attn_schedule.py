"""The attention grid's work order (csrc/attn_sched.h), checked on the CPU.

The header is compiled as host C++ with g++ and every launch index of every
grid with 1..260 (sequence, head) pairs and 1..80 query blocks is mapped:
the mapping must hit every (pair, block) exactly once and never leave the
grid (an index outside it would address memory outside Q/K/V/out), each
XCD's dispatch sequence must be in non-increasing block order (longest
first), and a pair's blocks may span at most two XCDs whenever an XCD's
range is at least one pair long.
"""
import os
import shutil
import subprocess

import pytest

CSRC = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "paper_2607_21291_amd", "csrc")

CHECK = r"""
#define DSF_HD
#include "attn_sched.h"
#include <cstdio>
#include <vector>
int main() {
  long cases = 0;
  for (int BH = 1; BH <= 260; ++BH)
    for (int nqb = 1; nqb <= 80; ++nqb) {
      const int W = BH * nqb;
      std::vector<int> seen(W, 0), lastq(8, 1 << 30), xmask(BH, 0);
      for (int L = 0; L < W; ++L) {
        const dsf::AttnItem it = dsf::attn_item(L, W, nqb);
        if (it.bh < 0 || it.bh >= BH || it.qblk < 0 || it.qblk >= nqb) { printf("outside BH=%d nqb=%d L=%d\n", BH, nqb, L); return 1; }
        if (seen[it.bh * nqb + it.qblk]++) { printf("twice BH=%d nqb=%d L=%d\n", BH, nqb, L); return 1; }
        const int x = L % 8;
        if (it.qblk > lastq[x]) { printf("order BH=%d nqb=%d L=%d\n", BH, nqb, L); return 1; }
        lastq[x] = it.qblk;
        xmask[it.bh] |= 1 << x;
      }
      for (int b = 0; b < BH; ++b)
        if (W / 8 >= nqb && __builtin_popcount(xmask[b]) > 2) { printf("spread BH=%d nqb=%d\n", BH, nqb); return 1; }
      ++cases;
    }
  printf("ok %ld\n", cases);
  return 0;
}
"""


def test_attention_work_order_is_a_longest_first_bijection(tmp_path):
    cxx = shutil.which("g++") or shutil.which("c++")
    if cxx is None:
        pytest.skip("no host C++ compiler")
    src = tmp_path / "check.cpp"
    src.write_text(CHECK)
    exe = tmp_path / "check"
    subprocess.run([cxx, "-O2", "-std=c++17", "-I", CSRC, str(src), "-o", str(exe)], check=True)
    out = subprocess.run([str(exe)], capture_output=True, text=True, timeout=120)
    assert out.returncode == 0, out.stdout + out.stderr
    assert out.stdout.strip() == "ok 20800"
