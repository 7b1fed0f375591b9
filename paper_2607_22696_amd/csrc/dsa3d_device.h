// Device helpers shared by the forward and backward kernels of the 3D-DSA library.
//
// Lane layout: one query row (batch b, token (t,i,j), head m) is served by
// L = row_bytes / 16 lanes, each owning 16 contiguous bytes of the row (8 bf16 or 4 fp32
// channels), so a K/V corner row is one 16-byte load per lane and a wave reads
// G = 64 / L corner rows per load instruction.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "dsa3d_internal.h"

#define DSA3D_TILE_FN __host__ __device__ inline __attribute__((always_inline))
#include "tile_order.h"

namespace dsa3d {
namespace dev {

constexpr int kBlockThreads = 256;
constexpr int kWavesPerBlock = kBlockThreads / 64;
constexpr int kNumXcd = 8;
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// NC = 16-byte chunks of a row per lane (1 or 2).
template <int D, bool BF16, int NC = 1>
struct Layout {
  static constexpr int kElemBytes = BF16 ? 2 : 4;
  static constexpr int kRowBytes = D * kElemBytes;
  static constexpr int kChunks = NC;
  static constexpr int kLanes = kRowBytes / (16 * NC);  // lanes per query row
  static constexpr int kVec = 16 * NC / kElemBytes;      // channels per lane
  static constexpr int kGroups = 64 / kLanes;            // query rows per wave
  static constexpr int kRowsPerBlock = kGroups * kWavesPerBlock;
  static_assert(kLanes >= 2 && kLanes <= 32, "unsupported head_dim");
};

// ---------------------------------------------------------------------------- lane helpers

template <int CTRL>
__device__ inline __attribute__((always_inline)) float dpp_mov(float x) {
  return __builtin_bit_cast(
      float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), CTRL, 0xF, 0xF, false));
}

// Sum over the L consecutive lanes that serve one query; every lane gets the total.
template <int L>
__device__ inline __attribute__((always_inline)) float group_sum(float x) {
  if constexpr (L >= 2) x += dpp_mov<0xB1>(x);   // quad_perm [1,0,3,2]: lane ^ 1
  if constexpr (L >= 4) x += dpp_mov<0x4E>(x);   // quad_perm [2,3,0,1]: lane ^ 2
  if constexpr (L >= 8) x += dpp_mov<0x141>(x);  // row_half_mirror: other quad of the 8
  if constexpr (L >= 16) x += dpp_mov<0x140>(x); // row_mirror: other half of the 16-lane row
  if constexpr (L >= 32) x += __shfl_xor(x, 16);
  return x;
}

__device__ inline __attribute__((always_inline)) float bf16_lo(uint32_t u) { return __uint_as_float(u << 16); }
__device__ inline __attribute__((always_inline)) float bf16_hi(uint32_t u) { return __uint_as_float(u & 0xffff0000u); }

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

__device__ inline __attribute__((always_inline)) float dot2_bf16(uint32_t a, uint32_t b, float c) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a),
                                         __builtin_bit_cast(bf16x2_t, b), c, false);
}

// round-to-nearest-even fp32 -> bf16 (NaN stays NaN)
__device__ inline __attribute__((always_inline)) uint32_t bf16_bits(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (u >> 16) | 0x40u;
  u += 0x7fffu + ((u >> 16) & 1u);
  return u >> 16;
}

// <a, b> over this lane's 16-byte chunk of two rows.
template <bool BF16>
__device__ inline __attribute__((always_inline)) float chunk_dot(const uint4& a, const uint4& b) {
  if constexpr (BF16) {
    float acc = dot2_bf16(a.x, b.x, 0.0f);
    acc = dot2_bf16(a.y, b.y, acc);
    acc = dot2_bf16(a.z, b.z, acc);
    return dot2_bf16(a.w, b.w, acc);
  } else {
    float acc = __uint_as_float(a.x) * __uint_as_float(b.x);
    acc = fmaf(__uint_as_float(a.y), __uint_as_float(b.y), acc);
    acc = fmaf(__uint_as_float(a.z), __uint_as_float(b.z), acc);
    return fmaf(__uint_as_float(a.w), __uint_as_float(b.w), acc);
  }
}

// acc[v] += w * row[v] over this lane's chunk (fp32 accumulators).
template <bool BF16>
__device__ inline __attribute__((always_inline)) void chunk_axpy(float* acc, float w, const uint4& r) {
  const uint32_t u[4] = {r.x, r.y, r.z, r.w};
  if constexpr (BF16) {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      acc[2 * e] = fmaf(w, bf16_lo(u[e]), acc[2 * e]);
      acc[2 * e + 1] = fmaf(w, bf16_hi(u[e]), acc[2 * e + 1]);
    }
  } else {
#pragma unroll
    for (int e = 0; e < 4; ++e) acc[e] = fmaf(w, __uint_as_float(u[e]), acc[e]);
  }
}

template <bool BF16>
__device__ inline __attribute__((always_inline)) void chunk_to_float(const uint4& r, float* f) {
  const uint32_t u[4] = {r.x, r.y, r.z, r.w};
  if constexpr (BF16) {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      f[2 * e] = bf16_lo(u[e]);
      f[2 * e + 1] = bf16_hi(u[e]);
    }
  } else {
#pragma unroll
    for (int e = 0; e < 4; ++e) f[e] = __uint_as_float(u[e]);
  }
}

__device__ inline __attribute__((always_inline)) uint4 load16(const char* base, int64_t byte_off) {
  return *reinterpret_cast<const uint4*>(base + byte_off);
}

// Logical tile of a block: each XCD gets one contiguous range of tiles.
__device__ inline __attribute__((always_inline)) int xcd_tile(int bid, int nblocks) {
  const int xcd = bid % kNumXcd, slot = bid / kNumXcd;
  const int per = nblocks / kNumXcd, rem = nblocks % kNumXcd;
  return xcd * per + min(xcd, rem) + slot;
}

// ---------------------------------------------------------------------------- corner rows
//
// K and V rows are read through structured buffers: one record per token holds the rows of
// all heads of that token (record stride = heads * row_bytes), the resource base sits at
// head m of the first frame of a window of frames, and the record index of a voxel is
// (z - t0) * H * W + y * W + x.  A corner outside the grid (or outside the window) gets an
// index beyond the record count, and the buffer unit returns zeros for it: zero padding
// without branches or masks.  A buffer covers at most 4 GB from its base, so for tensors
// larger than that the window spans the frames around the block's own frame; the rare
// corner inside the grid but outside the window is loaded by a plain global load.

typedef int i32x4_t __attribute__((ext_vector_type(4)));

__device__ i32x4_t dsa3d_struct_buffer_load_v4(__amdgpu_buffer_rsrc_t rsrc, int vindex, int voffset,
                                              int soffset, int aux)
    __asm("llvm.amdgcn.struct.ptr.buffer.load.v4i32");

// Added to an index term to push a record index out of range.  Three of them stay below
// 2^31, and every valid index is below 2^28 (a window spans < 4 GB of records >= 16 B).
constexpr int kPoison = 1 << 29;
// Third descriptor word for untyped 32-bit buffer access on gfx9-class GPUs.
constexpr int kBufferFlags = 0x00020000;

struct RowWindow {
  __amdgpu_buffer_rsrc_t k, v;
  int t0, frames;  // window [t0, t0 + frames); frames == 0: every corner takes the global path
};

// Window of batch item b, head m, centred on frame tc (all arguments wave-uniform).
template <int ROW_BYTES>
__device__ inline __attribute__((always_inline)) RowWindow make_window(const Geometry& g,
                                                                       const void* k, const void* v,
                                                                       int b, int m, int tc) {
  RowWindow w;
  w.frames = g.win_frames;
  w.t0 = 0;
  int64_t base = 0;
  int nrec = 0;  // no window: zero records, so every buffer load returns zeros
  short stride = 16;
  if (w.frames > 0) {
    w.t0 = min(max(tc - (w.frames - 1) / 2, 0), g.T - w.frames);
    base = (((int64_t)b * g.T + w.t0) * g.H * g.W * g.heads + m) * ROW_BYTES;
    nrec = w.frames * g.H * g.W;
    stride = (short)(g.heads * ROW_BYTES);
  }
  w.k = __builtin_amdgcn_make_buffer_rsrc((void*)(static_cast<const char*>(k) + base), stride, nrec,
                                          kBufferFlags);
  w.v = __builtin_amdgcn_make_buffer_rsrc((void*)(static_cast<const char*>(v) + base), stride, nrec,
                                          kBufferFlags);
  return w;
}

__device__ inline __attribute__((always_inline)) uint4 buffer_row(__amdgpu_buffer_rsrc_t r, int vidx,
                                                                  int lane_off) {
  const i32x4_t x = dsa3d_struct_buffer_load_v4(r, vidx, lane_off, 0, 0);
  return make_uint4((uint32_t)x.x, (uint32_t)x.y, (uint32_t)x.z, (uint32_t)x.w);
}

// One sampling point of a query: corner record indices and weights (registers only).
struct Point {
  int vidx[8];                // record index of corner c = cz*4 + cy*2 + cx (out of range: zeros)
  float w[8];                 // trilinear weight of corner c (corners outside read as zero rows)
  float ax[2], ay[2], az[2];  // per-axis weights of the lower / upper corner
  int cx, cy, cz;             // floor of the (clamped) position: the trilinear cell
  bool slow;                  // a corner inside the grid lies outside the buffer window
};

// pos = (float)(integer base) + offset, clamped to [-2, size + 1] (every corner of a position
// beyond that range is outside the grid, so the clamp changes no value or gradient; it also
// sends NaN to -2 and keeps the integer conversion in range).
__device__ inline __attribute__((always_inline)) void axis(float base, float off, int size, int& i0,
                                                           float& t) {
  float p = base + off;
  p = fminf(fmaxf(p, -2.0f), (float)size + 1.0f);
  const float f = floorf(p);
  t = p - f;
  i0 = (int)f;
}

__device__ inline __attribute__((always_inline)) void make_point(const Geometry& g,
                                                                 const RowWindow& win, int t, int i,
                                                                 int j, int dz, int dy, int dx,
                                                                 float ox, float oy, float oz,
                                                                 Point& pt) {
  int ix, iy, iz;
  float tx, ty, tz;
  axis((float)(j + dx), ox, g.W, ix, tx);
  axis((float)(i + dy), oy, g.H, iy, ty);
  axis((float)(t + dz), oz, g.T, iz, tz);
  pt.ax[0] = 1.0f - tx;
  pt.ax[1] = tx;
  pt.ay[0] = 1.0f - ty;
  pt.ay[1] = ty;
  pt.az[0] = 1.0f - tz;
  pt.az[1] = tz;
  pt.cx = ix;
  pt.cy = iy;
  pt.cz = iz;
  const int HW = g.H * g.W;
  const int zr = iz - win.t0;
  const int xt[2] = {(unsigned)ix < (unsigned)g.W ? ix : kPoison,
                     (unsigned)(ix + 1) < (unsigned)g.W ? ix + 1 : kPoison};
  const int yt[2] = {(unsigned)iy < (unsigned)g.H ? iy * g.W : kPoison,
                     (unsigned)(iy + 1) < (unsigned)g.H ? (iy + 1) * g.W : kPoison};
  const int zt[2] = {(unsigned)zr < (unsigned)win.frames ? zr * HW : kPoison,
                     (unsigned)(zr + 1) < (unsigned)win.frames ? (zr + 1) * HW : kPoison};
  pt.slow = ((unsigned)iz < (unsigned)g.T && (unsigned)zr >= (unsigned)win.frames) ||
            ((unsigned)(iz + 1) < (unsigned)g.T && (unsigned)(zr + 1) >= (unsigned)win.frames);
  const float wyz[4] = {pt.ay[0] * pt.az[0], pt.ay[1] * pt.az[0], pt.ay[0] * pt.az[1],
                        pt.ay[1] * pt.az[1]};
#pragma unroll
  for (int c = 0; c < 8; ++c) {
    const int cx = c & 1, cy = (c >> 1) & 1, cz = c >> 2;
    pt.vidx[c] = xt[cx] + yt[cy] + zt[cz];
    pt.w[c] = pt.ax[cx] * wyz[c >> 1];
  }
}

// K and V rows (this lane's 16 bytes of each) at the 8 corners of a point that a lane of the
// row formed: `vidx` are its corner indices, already fetched from that owner lane (ds_bpermute
// address `src`, its point `mine`).  Corners come through the window resources; an in-grid
// corner outside the window takes a global load, and the window test and the cell that load
// needs are fetched from the owner only when some lane of the wave has such a corner (the test
// is wave-uniform and rare), so the common case exchanges the 8 indices and one flag per
// point.  KV = false: V only.
template <int ROW_BYTES, bool KV>
__device__ inline __attribute__((always_inline)) void load_shared_corners(
    const Geometry& g, const RowWindow& win, const char* kb, const char* vb, int b, int m,
    int lane_off, const Point& mine, int src, const int* vidx, uint4* kr, uint4* vr) {
#pragma unroll
  for (int c = 0; c < 8; ++c) {
    if constexpr (KV) kr[c] = buffer_row(win.k, vidx[c], lane_off);
    vr[c] = buffer_row(win.v, vidx[c], lane_off);
  }
  const bool slow = __builtin_amdgcn_ds_bpermute(src, (int)mine.slow) != 0;
  if (__builtin_amdgcn_ballot_w64(slow)) {
    const int cx = __builtin_amdgcn_ds_bpermute(src, mine.cx);
    const int cy = __builtin_amdgcn_ds_bpermute(src, mine.cy);
    const int cz = __builtin_amdgcn_ds_bpermute(src, mine.cz);
    if (slow) {
#pragma unroll
      for (int c = 0; c < 8; ++c) {
        const int x = cx + (c & 1), y = cy + ((c >> 1) & 1), z = cz + (c >> 2);
        const bool inside = (unsigned)x < (unsigned)g.W && (unsigned)y < (unsigned)g.H &&
                            (unsigned)z < (unsigned)g.T;
        if (inside && (unsigned)(z - win.t0) >= (unsigned)win.frames) {
          const int64_t row = ((((int64_t)b * g.T + z) * g.H + y) * g.W + x) * g.heads + m;
          if constexpr (KV) kr[c] = load16(kb, row * ROW_BYTES + lane_off);
          vr[c] = load16(vb, row * ROW_BYTES + lane_off);
        }
      }
    }
  }
}

// The same with the owner's point read from its LDS slot instead of from its registers:
// `cell` = (window flag, cell x, y, z) of that point, `cell_at` its place in the slot.
template <int ROW_BYTES, bool KV>
__device__ inline __attribute__((always_inline)) void load_stashed_corners(
    const Geometry& g, const RowWindow& win, const char* kb, const char* vb, int b, int m,
    int lane_off, const int4* cell_at, const int* vidx, uint4* kr, uint4* vr) {
#pragma unroll
  for (int c = 0; c < 8; ++c) {
    if constexpr (KV) kr[c] = buffer_row(win.k, vidx[c], lane_off);
    vr[c] = buffer_row(win.v, vidx[c], lane_off);
  }
  const int4 cell = *cell_at;
  const bool slow = cell.x != 0;
  if (__builtin_amdgcn_ballot_w64(slow)) {
    if (slow) {
#pragma unroll
      for (int c = 0; c < 8; ++c) {
        const int x = cell.y + (c & 1), y = cell.z + ((c >> 1) & 1), z = cell.w + (c >> 2);
        const bool inside = (unsigned)x < (unsigned)g.W && (unsigned)y < (unsigned)g.H &&
                            (unsigned)z < (unsigned)g.T;
        if (inside && (unsigned)(z - win.t0) >= (unsigned)win.frames) {
          const int64_t row = ((((int64_t)b * g.T + z) * g.H + y) * g.W + x) * g.heads + m;
          if constexpr (KV) kr[c] = load16(kb, row * ROW_BYTES + lane_off);
          vr[c] = load16(vb, row * ROW_BYTES + lane_off);
        }
      }
    }
  }
}

// LDS point slots: thread t of a block keeps N int4 (16-byte) words at slot_of<L, N>(t), with
// one word of padding after each row's L slots.  The rows of a wave read one slot each in the
// same instruction (the row's lanes read the same words: a broadcast); without the padding
// their addresses would differ by L N 16 bytes, a multiple of the 256 bytes the LDS banks span
// at L = 16, so all of them would hit the same banks.  With it they differ by L N 16 + 16
// bytes, which for the slot sizes used here (N = 5 and 9, L = 8, 16 or 32) puts each row on a
// different 16-byte bank group; an odd N keeps the writes of consecutive lanes, N 16 bytes
// apart, on different bank groups too.
template <int L, int N>
__device__ inline __attribute__((always_inline)) int slot_of(int t) {
  return t * N + t / L;
}
template <int L, int N>
constexpr int slot_words() {
  return kBlockThreads * N + kBlockThreads / L;
}

// ---------------------------------------------------------------------------- launch shape

constexpr int kMaxBlocks = 1 << 22;  // grid cap; larger problems loop over tiles

// Pencil order of the query-owned kernels: tiles of kRowsPerBlock tokens inside pencils of
// about 12 x 12 tokens of a frame.  Measured on one MI355X at 64x68x120, 24 heads x 128,
// 3x5x5, offsets U[-8,8]: forward 159 / 162 / 197 ms and sweep 199 / 201 / 220 ms with
// pencils of about 12 x 12 / 16 x 16 / 24 x 24 tokens.
template <int D, bool BF16>
inline PencilOrder query_order(const Geometry& g) {
  return plan_pencils(g.B * g.heads, g.T, g.H, g.W, Layout<D, BF16>::kRowsPerBlock, 12, 12);
}

// Workgroups for `vtiles` virtual tiles: at most kMaxBlocks, a multiple of 8 when capped so
// that a workgroup's later tiles (v += gridDim.x) stay on its XCD.
inline int grid_blocks(int64_t vtiles) {
  return (int)(vtiles < kMaxBlocks ? vtiles : kMaxBlocks);
}

}  // namespace dev
}  // namespace dsa3d
