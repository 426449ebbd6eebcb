"""The workgroup -> work-item remaps in csrc/xcd.h must be bijections on
[0, n): a lost item leaves output rows unwritten, a repeated one writes a row
twice.  The kernels only reach the segment order on more than 8 x 128 rows,
beyond what the small GPU cases launch, so both maps are checked here on the
host for every n up to 3000 and the workload sizes; so is the frame-tile
order of query blocks inside a head, for every block count up to 1300 and
frame sizes from 1 to 60 blocks, with one small order written out."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2606_23743_amd", "csrc")

PROGRAM = r"""
#include <cstdio>
#include <vector>
#include "xcd.h"

static bool bijective(int n, int c) {
  std::vector<char> seen(n, 0);
  for (int id = 0; id < n; ++id) {
    const int r = c ? sva::xcd_remap_segments(id, n, c) : sva::xcd_remap(id, n);
    if (r < 0 || r >= n || seen[r]) return false;
    seen[r] = 1;
  }
  return true;
}

int main() {
  const int cs[] = {0, 1, 7, 64, 109, 128, 256};
  const int big[] = {41856, 31648, 10240, 56736, 20 * 512, 2 * 24 * 1182};
  int bad = 0;
  for (int c : cs) {
    for (int n = 1; n <= 3000; ++n) bad += !bijective(n, c);
    for (int n : big) bad += !bijective(n, c);
  }
  // segment order: at slot s of a whole segment, XCD x holds item k*8c + x*c + j
  const int n = 5000, c = 128;
  for (int id = 0; id < 4096; ++id) {
    const int s = id / 8, x = id % 8;
    bad += sva::xcd_remap_segments(id, n, c) != (s / c) * 8 * c + x * c + s % c;
  }
  // frame tiles: a bijection on [0, nB) for every frame size and tile shape
  const int fs[] = {1, 2, 3, 7, 13, 28, 29, 55, 60};
  const int tiles[][2] = {{8, 4}, {1, 1}, {2, 3}, {8, 8}, {5, 7}};
  for (int nb = 1; nb <= 1300; ++nb)
    for (int f : fs)
      for (auto& tl : tiles) {
        std::vector<char> seen(nb, 0);
        for (int l = 0; l < nb; ++l) {
          const int r = sva::frame_tile_order(l, nb, f, tl[0], tl[1]);
          if (r < 0 || r >= nb || seen[r]) { ++bad; break; }
          seen[r] = 1;
        }
      }
  // 10 blocks, 3 per frame, tiles of 2 blocks x 2 frames: super-row {0..5} in
  // the order 0 1 3 4 (two blocks of frames 0 and 1) then 2 5 (the leftover
  // column); the tail holds one whole frame (6 7 8) and block 9
  const int want[10] = {0, 1, 3, 4, 2, 5, 6, 7, 8, 9};
  for (int l = 0; l < 10; ++l) bad += sva::frame_tile_order(l, 10, 3, 2, 2) != want[l];
  std::printf("bad=%d\n", bad);
  return bad != 0;
}
"""


def test_remaps_are_bijections(tmp_path):
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(hipcc):
        pytest.skip("hipcc not available")
    src = tmp_path / "remap.hip"
    src.write_text(PROGRAM)
    exe = tmp_path / "remap"
    subprocess.run([hipcc, "-O2", "-std=c++17", "--offload-arch=gfx950", "-Xclang", "-target-feature",
                    "-Xclang", "-packed-fp32-ops", "-w", "-I", CSRC, str(src), "-o", str(exe)],
                   check=True, capture_output=True)
    res = subprocess.run([str(exe)], capture_output=True, text=True)
    assert res.returncode == 0 and res.stdout.strip() == "bad=0", res.stdout + res.stderr
