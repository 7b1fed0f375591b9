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

namespace dsa3d {
namespace dev {

constexpr int kBlockThreads = 256;
constexpr int kWavesPerBlock = kBlockThreads / 64;
constexpr int kNumXcd = 8;
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

template <int D, bool BF16>
struct Layout {
  static constexpr int kElemBytes = BF16 ? 2 : 4;
  static constexpr int kRowBytes = D * kElemBytes;
  static constexpr int kLanes = kRowBytes / 16;  // lanes per query row
  static constexpr int kVec = 16 / kElemBytes;   // channels per lane
  static constexpr int kGroups = 64 / kLanes;    // query rows per wave
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

// One sampling point of a query: corner rows, weights and validity (registers only).
struct Point {
  int64_t row[8];  // row index of each corner in [B][T][H][W][heads]
  float w[8];      // trilinear weight (0 for corners outside the grid)
  bool ok[8];      // corner inside the grid
  float ax[2], ay[2], az[2];  // per-axis weights (lower, upper corner), before zero padding
  int cx, cy, cz;             // floor of the (clamped) position: the trilinear cell
};

// pos = (float)(integer base) + offset, clamped to [-2, size + 1] (every corner of a position
// beyond that range is outside the grid, so the clamp changes no value or gradient; it also
// sends NaN to -2 and keeps the integer conversion in range).
__device__ inline __attribute__((always_inline)) void axis(float base, float off, int size, int& i0, float& t) {
  float p = base + off;
  p = fminf(fmaxf(p, -2.0f), (float)size + 1.0f);
  const float f = floorf(p);
  t = p - f;
  i0 = (int)f;
}

__device__ inline __attribute__((always_inline)) void make_point(const Geometry& g, int b, int t, int i, int j, int m,
                                           int dz, int dy, int dx, const float* off, Point& pt) {
  int ix, iy, iz;
  float tx, ty, tz;
  axis((float)(j + dx), off[0], g.W, ix, tx);
  axis((float)(i + dy), off[1], g.H, iy, ty);
  axis((float)(t + dz), off[2], g.T, iz, tz);
  pt.ax[0] = 1.0f - tx;
  pt.ax[1] = tx;
  pt.ay[0] = 1.0f - ty;
  pt.ay[1] = ty;
  pt.az[0] = 1.0f - tz;
  pt.az[1] = tz;
  pt.cx = ix;
  pt.cy = iy;
  pt.cz = iz;
  const bool vx[2] = {(unsigned)ix < (unsigned)g.W, (unsigned)(ix + 1) < (unsigned)g.W};
  const bool vy[2] = {(unsigned)iy < (unsigned)g.H, (unsigned)(iy + 1) < (unsigned)g.H};
  const bool vz[2] = {(unsigned)iz < (unsigned)g.T, (unsigned)(iz + 1) < (unsigned)g.T};
  const int64_t sx = g.heads, sy = (int64_t)g.W * g.heads, sz = (int64_t)g.H * sy;
  const int64_t r0 = ((((int64_t)b * g.T + iz) * g.H + iy) * g.W + ix) * g.heads + m;
#pragma unroll
  for (int c = 0; c < 8; ++c) {
    const int cx = c & 1, cy = (c >> 1) & 1, cz = c >> 2;
    pt.ok[c] = vx[cx] && vy[cy] && vz[cz];
    pt.w[c] = pt.ok[c] ? pt.ax[cx] * pt.ay[cy] * pt.az[cz] : 0.0f;
    pt.row[c] = r0 + cx * sx + cy * sy + cz * sz;
  }
}

// ---------------------------------------------------------------------------- launch shape

constexpr int kMaxBlocks = 1 << 22;  // grid cap; larger problems loop over tiles

template <int D, bool BF16>
inline int tiles_for(const Geometry& g) {
  using LY = Layout<D, BF16>;
  const int64_t per = (g.N + LY::kRowsPerBlock - 1) / LY::kRowsPerBlock;
  return (int)(per * g.B * g.heads);
}

}  // namespace dev
}  // namespace dsa3d
