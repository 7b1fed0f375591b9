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
// reach from a few consecutive frames: at a spread of +-9.5 voxels (offsets U[-8, 8] on a
// 3x5x5 kernel) the rows the in-flight tiles of a 17 x 15 pencil read stay L2-resident
// across many frames, while runs of consecutive tokens across whole frame rows touch a band
// of rows several times the 4 MB of an XCD's L2.
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

// Pencils of about target_r x target_c cells: the rows (columns) are split into
// round(rows / target_r) equal parts, rounded up, so that on grids whose sizes divide
// evenly every pencil is whole (68 x 120 tokens -> 4 x 8 pencils of 17 x 15).
DSA3D_TILE_FN PencilOrder plan_pencils(int groups, int frames, int rows, int cols, int run,
                                       int target_r, int target_c) {
  PencilOrder o;
  o.frames = frames;
  o.rows = rows;
  o.cols = cols;
  o.run = run;
  int nr = (2 * rows + target_r) / (2 * target_r);  // round(rows / target_r)
  int nc = (2 * cols + target_c) / (2 * target_c);
  nr = nr < 1 ? 1 : nr;
  nc = nc < 1 ? 1 : nc;
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
