// Tile order of the 3D-DSA kernels: pencils that walk the frames.
//
// Every kernel works on a grid of cells per (batch, head) group: query tokens for the
// forward and the backward sweep, voxel blocks for the dK/dV gathers.  The cells of one
// frame are cut into pencils of ph x pw cells; a pencil spans all frames of its group and is
// walked frame by frame, each frame's ph x pw rectangle in raster order, `run` cells per
// tile (one workgroup's share).  Pencil g is handed to XCD g % 8: consecutive workgroups
// reach the XCDs round-robin (workgroup b runs on XCD b % 8), so virtual tile v belongs to
// XCD v % 8 and is tile (v / 8) % pencil_tiles of that XCD's pencil number (v / 8) /
// pencil_tiles.  Each XCD's L2 then holds the K/V rows that the queries of one pencil
// reach from a few consecutive frames.  At a spread of +-9.5 voxels (offsets U[-8, 8] on a
// 3x5x5 kernel) most of the rows the in-flight tiles of a pencil of about 12 x 12 tokens
// read are still L2-resident when the next frames reach them (74% of the forward's L2
// requests hit), while runs of consecutive tokens across whole frame rows touch a band of
// rows several times the 4 MB of an XCD's L2 (22% hit).
//
// This header is plain C++ (no HIP types), so that a host test can enumerate the order;
// the kernels include it with DSA3D_TILE_FN defined as __host__ __device__ inline.
#pragma once

#include <stdint.h>

#ifndef DSA3D_TILE_FN
#define DSA3D_TILE_FN inline
#endif

namespace dsa3d {

constexpr int kPencilXcds = 8;

struct PencilOrder {
  int frames, rows, cols;  // cell grid of one (batch, head) group
  int ph, pw;              // pencil size in cells
  int run;                 // cells per tile
  int np_r, np_c;          // pencils along rows and columns
  int runs;                // tiles per pencil frame, ceil(ph * pw / run)
  int64_t pencil_tiles;    // tiles per pencil, frames * runs
  int64_t pencils;         // groups * np_r * np_c
  int64_t vtiles;          // virtual tiles: 8 * ceil(pencils / 8) * pencil_tiles
};

DSA3D_TILE_FN PencilOrder pencils_of(int groups, int frames, int rows, int cols, int run, int nr,
                                     int nc) {
  PencilOrder o;
  o.frames = frames;
  o.rows = rows;
  o.cols = cols;
  o.run = run;
  o.ph = (rows + nr - 1) / nr;
  o.pw = (cols + nc - 1) / nc;
  o.np_r = (rows + o.ph - 1) / o.ph;
  o.np_c = (cols + o.pw - 1) / o.pw;
  o.runs = (o.ph * o.pw + run - 1) / run;
  o.pencil_tiles = (int64_t)frames * o.runs;
  o.pencils = (int64_t)groups * o.np_r * o.np_c;
  o.vtiles = (o.pencils + kPencilXcds - 1) / kPencilXcds * kPencilXcds * o.pencil_tiles;
  return o;
}

// Pencils of about target_r x target_c cells.  The rows (columns) are split into n equal
// parts, rounded up, with n within one of round(rows / target_r) (round(cols / target_c));
// of those nine splits the one that leaves the fewest idle cells (cells of a frame's tiles
// past the grid or past a pencil's rectangle) wins, then the one nearest the target.  On the
// 68 x 120 grid with 16-cell tiles and a 12 x 12 target that gives 10 x 11 pencils, and on
// 34 x 60 with 32-cell tiles 17 x 15 (255 cells in 8 tiles of 32).
DSA3D_TILE_FN PencilOrder plan_pencils(int groups, int frames, int rows, int cols, int run,
                                       int target_r, int target_c) {
  const int nr0 = (2 * rows + target_r) / (2 * target_r);  // round(rows / target_r)
  const int nc0 = (2 * cols + target_c) / (2 * target_c);
  PencilOrder best = pencils_of(groups, frames, rows, cols, run, nr0 < 1 ? 1 : nr0,
                                nc0 < 1 ? 1 : nc0);
  int64_t best_idle = -1, best_dist = 0;
  for (int dr = -1; dr <= 1; ++dr) {
    for (int dc = -1; dc <= 1; ++dc) {
      const int nr = nr0 + dr, nc = nc0 + dc;
      if (nr < 1 || nc < 1 || nr > rows || nc > cols) continue;
      const PencilOrder o = pencils_of(groups, frames, rows, cols, run, nr, nc);
      const int64_t idle = (int64_t)o.np_r * o.np_c * o.runs * run - (int64_t)rows * cols;
      const int64_t dist = (int64_t)(o.ph - target_r) * (o.ph - target_r) +
                           (int64_t)(o.pw - target_c) * (o.pw - target_c);
      if (best_idle < 0 || idle < best_idle || (idle == best_idle && dist < best_dist)) {
        best = o;
        best_idle = idle;
        best_dist = dist;
      }
    }
  }
  return best;
}

// A tile: its group, frame, pencil and first cell inside the pencil's rectangle.
struct PencilTile {
  int group, frame, pr, pc, u0;
};

// Tile of virtual tile v; false for a tile past the last pencil (the XCD has no pencil left).
DSA3D_TILE_FN bool pencil_tile(const PencilOrder& o, int64_t v, PencilTile& t) {
  const int64_t xcd = v % kPencilXcds, slot = v / kPencilXcds;
  const int64_t g = slot / o.pencil_tiles * kPencilXcds + xcd;
  if (g >= o.pencils) return false;
  const int64_t k = slot % o.pencil_tiles;
  const int per_group = o.np_r * o.np_c;
  t.group = (int)(g / per_group);
  const int p = (int)(g % per_group);
  t.pr = p / o.np_c;
  t.pc = p % o.np_c;
  t.frame = (int)(k / o.runs);
  t.u0 = (int)(k % o.runs) * o.run;
  return true;
}

// Cell e of a tile (e < run): its row and column in the grid; false if it lies past the end
// of the pencil's rectangle or outside the grid (ragged pencils at the grid's edges).
DSA3D_TILE_FN bool pencil_cell(const PencilOrder& o, const PencilTile& t, int e, int& row,
                               int& col) {
  const int u = t.u0 + e;
  const int y = u / o.pw, x = u - y * o.pw;
  row = t.pr * o.ph + y;
  col = t.pc * o.pw + x;
  return u < o.ph * o.pw && row < o.rows && col < o.cols;
}

}  // namespace dsa3d
