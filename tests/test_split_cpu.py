"""The k-range cut of split forward contractions (csrc/nf_split.h), compiled
for the host with g++ and checked over many (K, pieces) pairs: every piece
starts on a whole 16-element stage, the pieces cover [0, K) exactly, no piece
is empty, and the launcher's alignment rule accepts exactly the cuts on whole
stages (the unaligned cut at ceil(K / pieces) that preceded it is rejected
whenever it is off the grid)."""

import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_1902_06714_amd", "csrc")

PROGRAM = r"""
#include <cstdio>
#include "nf_split.h"
int main() {
  long bad = 0, cases = 0;
  for (long K = 1; K <= 5000; ++K) {
    for (long want = 1; want <= 24; ++want) {
      const nf::KSplit s = nf::k_split(K, want);
      ++cases;
      const long sub = s.sub_len, n = s.nsplit;
      bool ok = n >= 1 && n <= (want < 1 ? 1 : want) && sub >= 1;
      if (n > 1) ok = ok && sub % nf::KSPLIT_BK == 0;
      ok = ok && (long)n * sub >= K && (long)(n - 1) * sub < K;     // cover, last piece not empty
      ok = ok && nf::k_pieces_aligned(1, K, n, sub);
      // the earlier cut: ceil(K / want) per piece, accepted only on the grid
      const long naive = (K + want - 1) / want;
      const long nn = (K + naive - 1) / naive;
      const bool grid = nn <= 1 || naive % nf::KSPLIT_BK == 0;
      ok = ok && nf::k_pieces_aligned(1, K, (int)nn, naive) == grid;
      if (!ok) { if (bad < 5) std::printf("bad K=%ld want=%ld n=%ld sub=%ld\n", K, want, n, sub); ++bad; }
    }
  }
  // shards: every shard start must be on the grid as well
  for (long sl = 1; sl <= 200; ++sl) {
    ++cases;
    const bool want_ok = sl % nf::KSPLIT_BK == 0;
    if (nf::k_pieces_aligned(4, sl, 1, sl) != want_ok || !nf::k_pieces_aligned(1, sl, 1, sl)) ++bad;
  }
  std::printf("cases %ld bad %ld\n", cases, bad);
  return bad != 0;
}
"""


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs a host C++ compiler")
def test_k_split_pieces_start_on_whole_stages(tmp_path):
    src = tmp_path / "split.cpp"
    src.write_text(PROGRAM)
    exe = tmp_path / "split"
    subprocess.run(["g++", "-O1", "-std=c++17", "-I", CSRC, str(src), "-o", str(exe)], check=True)
    res = subprocess.run([str(exe)], capture_output=True, text=True)
    assert res.returncode == 0, res.stdout + res.stderr
    assert "bad 0" in res.stdout
