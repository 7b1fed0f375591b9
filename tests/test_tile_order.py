"""Host checks of the kernels' tile order (paper_2607_22696_amd/csrc/tile_order.h).

The forward, the backward sweep and the dK/dV gathers take their tiles from the pencil
order; a cell that it skipped or produced twice would leave an output row unwritten or
write it twice.  The header is plain C++, so it is compiled here into a small host program
that enumerates every virtual tile of a geometry and counts how often each (group, frame,
row, column) cell comes out; every cell must come out exactly once, inside the grid, with
XCD-consistent pencils (the XCD of a tile, v % 8, is the same for all tiles of its pencil).
"""
import os
import subprocess

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HDR = os.path.join(ROOT, "paper_2607_22696_amd", "csrc")

PROGRAM = r"""
#include <cstdio>
#include <cstdlib>
#include <vector>
#include "tile_order.h"
using namespace dsa3d;
int main(int argc, char** argv) {
  const int groups = atoi(argv[1]), frames = atoi(argv[2]), rows = atoi(argv[3]),
            cols = atoi(argv[4]), run = atoi(argv[5]), tr = atoi(argv[6]), tc = atoi(argv[7]);
  const long grid = atol(argv[8]);  // workgroups launched (0: one per virtual tile)
  const PencilOrder o = plan_pencils(groups, frames, rows, cols, run, tr, tc);
  const long launched = grid > 0 ? grid : (long)o.vtiles;
  std::vector<int> seen((size_t)groups * frames * rows * cols, 0);
  std::vector<int> xcd_of(o.pencils, -1);
  long bad = 0;
  for (long b = 0; b < launched; ++b) {
    for (int64_t v = b; v < o.vtiles; v += launched) {
      PencilTile t;
      if (!pencil_tile(o, v, t)) continue;
      const long g = ((long)t.group * o.np_r + t.pr) * o.np_c + t.pc;
      if (xcd_of[g] < 0) xcd_of[g] = (int)(b % 8);
      if (xcd_of[g] != (int)(b % 8)) ++bad;
      if (t.frame < 0 || t.frame >= frames || t.group < 0 || t.group >= groups) { ++bad; continue; }
      for (int e = 0; e < run; ++e) {
        int r, c;
        if (!pencil_cell(o, t, e, r, c)) continue;
        if (r < 0 || r >= rows || c < 0 || c >= cols) { ++bad; continue; }
        ++seen[(((size_t)t.group * frames + t.frame) * rows + r) * cols + c];
      }
    }
  }
  long zero = 0, many = 0;
  for (int s : seen) { zero += s == 0; many += s > 1; }
  printf("%ld %ld %ld %d %d %ld\n", bad, zero, many, o.ph, o.pw, (long)o.vtiles);
  return 0;
}
"""


@pytest.fixture(scope="module")
def prog(tmp_path_factory):
    d = tmp_path_factory.mktemp("tile_order")
    src = d / "t.cpp"
    src.write_text(PROGRAM)
    exe = d / "t"
    subprocess.check_call(["g++", "-O2", "-std=c++17", "-I", HDR, str(src), "-o", str(exe)])
    return str(exe)


def run(prog, *args):
    out = subprocess.check_output([prog, *map(str, args)], text=True).split()
    bad, zero, many, ph, pw, vtiles = map(int, out)
    return bad, zero, many, ph, pw, vtiles


# (groups, frames, rows, cols, run, target rows, target cols, workgroups launched)
CASES = [
    (24, 64, 68, 120, 16, 16, 16, 0),     # C5 query tokens, head_dim 128: pencils 17 x 15
    (16, 64, 34, 60, 32, 16, 16, 0),      # C4 query tokens, head_dim 64
    (2, 4, 8, 8, 32, 16, 16, 0),          # tiny grid: one pencil per group, fewer than 8 pencils
    (3, 5, 7, 9, 16, 16, 16, 0),          # ragged everything
    (1, 1, 1, 1, 64, 16, 16, 0),          # one cell
    (6, 3, 17, 33, 8, 16, 16, 0),         # pencils that do not divide the grid
    (24, 32, 34, 30, 2, 8, 4, 0),         # C5 gather voxel blocks (4 x 2 cells, frame pairs)
    (5, 7, 9, 11, 4, 8, 4, 0),
    (24, 64, 68, 120, 16, 16, 16, 8 * 1000),   # a capped grid: workgroups loop over tiles
    (3, 5, 7, 9, 16, 16, 16, 24),
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: "x".join(map(str, c)))
def test_every_cell_exactly_once(prog, case):
    bad, zero, many, ph, pw, vtiles = run(prog, *case)
    assert (bad, zero, many) == (0, 0, 0), (bad, zero, many)
    assert vtiles % 8 == 0


def test_the_1080p_grids_split_into_whole_pencils(prog):
    """68 x 120 tokens -> 4 x 8 pencils of 17 x 15; 34 x 60 -> 2 x 4 of 17 x 15."""
    assert run(prog, 24, 64, 68, 120, 16, 16, 16, 0)[3:5] == (17, 15)
    assert run(prog, 16, 64, 34, 60, 32, 16, 16, 0)[3:5] == (17, 15)
