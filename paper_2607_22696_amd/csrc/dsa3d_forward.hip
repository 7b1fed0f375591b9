// Forward kernel of 3D Deformable Slide Attention (MegaSlide-DiT, Section 5.2, Eq. (1)).
//
// Each L-lane group owns one query row.  For every point it forms the sampling position,
// the 8 trilinear corners and their weights in registers, loads the 8 K corner rows and
// the 8 V corner rows (one 16-byte buffer load per lane per row; corners outside the grid
// come back as zeros from the buffer unit), reduces the interpolated logit
// over the group with DPP butterflies (q.K by v_dot2_f32_bf16 on bf16 data, fp32
// accumulation) and folds the point into an online (running-max, base-2) softmax, so each
// corner row is read once.  Nothing per point is written to memory; the output row and
// its LSE are stored once.
//
// Memory order: consecutive workgroups go to the 8 XCDs round-robin; blocks are renumbered
// so each XCD walks one contiguous range of (batch, head, token) tiles and its L2 holds one
// head's sliding band of K/V rows.
#include "dsa3d_device.h"

namespace dsa3d {
namespace {

using namespace dev;

template <int D, bool BF16, int NC>
__global__ __launch_bounds__(kBlockThreads) void fwd_kernel(Geometry g, const void* __restrict__ q,
                                                             const void* __restrict__ k,
                                                             const void* __restrict__ v,
                                                             const float* __restrict__ offsets,
                                                             void* __restrict__ out,
                                                             float* __restrict__ lse, int tiles) {
  using LY = Layout<D, BF16, NC>;
  constexpr int L = LY::kLanes;
  constexpr int VEC = LY::kVec;
  constexpr int CV = VEC / NC;  // channels per 16-byte chunk
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int grp = lane / L, sub = lane % L;
  const int lane_off = sub * 16 * NC;
  const char* qb = static_cast<const char*>(q);
  const char* kb = static_cast<const char*>(k);
  const char* vb = static_cast<const char*>(v);
  const int tiles_per_bh = (g.N + LY::kRowsPerBlock - 1) / LY::kRowsPerBlock;
  const int HW = g.H * g.W;
  const int rt = (g.kt - 1) / 2, rh = (g.kh - 1) / 2, rw = (g.kw - 1) / 2;

  for (int tile = xcd_tile(blockIdx.x, gridDim.x); tile < tiles; tile += gridDim.x) {
    const int bh = tile / tiles_per_bh;
    const int b = bh / g.heads, m = bh % g.heads;
    const int n0 = (tile % tiles_per_bh) * LY::kRowsPerBlock;
    const RowWindow win = make_window<LY::kRowBytes>(g, k, v, b, m, n0 / HW);
    const int n_raw = n0 + wave * LY::kGroups + grp;
    const bool active = n_raw < g.N;
    const int n = active ? n_raw : g.N - 1;
    const int j = n % g.W, i = (n / g.W) % g.H, t = n / HW;
    const int64_t row = ((int64_t)b * g.N + n) * g.heads + m;

    uint4 qr[NC];
#pragma unroll
    for (int h = 0; h < NC; ++h) qr[h] = load16(qb, row * LY::kRowBytes + lane_off + 16 * h);
    const float* off = offsets + row * g.P * 3;
    float o[VEC];
#pragma unroll
    for (int e = 0; e < VEC; ++e) o[e] = 0.0f;
    float mx = -INFINITY, l = 0.0f;
    float ox = off[0], oy = off[1], oz = off[2];

    int it = 0, ih = 0, iw = 0;
    for (int p = 0; p < g.P; ++p) {
      Point pt;
      make_point(g, win, t, i, j, it - rt, ih - rh, iw - rw, ox, oy, oz, pt);
      if (p + 1 < g.P) {  // next point's offsets, in flight with this point's corner rows
        ox = off[3 * p + 3];
        oy = off[3 * p + 4];
        oz = off[3 * p + 5];
      }
      uint4 kr[8 * NC], vr[8 * NC];
      load_corners<LY::kRowBytes, NC>(g, win, kb, vb, b, m, lane_off, pt, kr, vr);
      float sp = 0.0f;
#pragma unroll
      for (int c = 0; c < 8; ++c) {
        float d = chunk_dot<BF16>(qr[0], kr[c * NC]);
#pragma unroll
        for (int h = 1; h < NC; ++h) d += chunk_dot<BF16>(qr[h], kr[c * NC + h]);
        sp = fmaf(pt.w[c], d, sp);
      }
      const float s2 = group_sum<L>(sp) * g.scale_log2;
      // One exponential per point: a new maximum rescales the running sums by
      // 2^(old max - new max) and enters with weight exactly 1; otherwise the point enters
      // with 2^(s - max).  (The first point always takes the first branch: 2^-inf = 0.)
      const bool up = s2 > mx;
      const float ex = exp2f(up ? mx - s2 : s2 - mx);
      const float corr = up ? ex : 1.0f;
      const float e = up ? 1.0f : ex;
      l = fmaf(l, corr, e);
      mx = up ? s2 : mx;
#pragma unroll
      for (int x = 0; x < VEC; ++x) o[x] *= corr;
#pragma unroll
      for (int c = 0; c < 8; ++c) {
#pragma unroll
        for (int h = 0; h < NC; ++h) chunk_axpy<BF16>(o + h * CV, e * pt.w[c], vr[c * NC + h]);
      }
      if (++iw == g.kw) {
        iw = 0;
        if (++ih == g.kh) {
          ih = 0;
          ++it;
        }
      }
    }
    if (active) {
      const float inv = 1.0f / l;
      char* ob = static_cast<char*>(out) + row * LY::kRowBytes + lane_off;
#pragma unroll
      for (int h = 0; h < NC; ++h) {
        const float* oh = o + h * CV;
        if constexpr (BF16) {
          uint4 w;
          w.x = bf16_bits(oh[0] * inv) | (bf16_bits(oh[1] * inv) << 16);
          w.y = bf16_bits(oh[2] * inv) | (bf16_bits(oh[3] * inv) << 16);
          w.z = bf16_bits(oh[4] * inv) | (bf16_bits(oh[5] * inv) << 16);
          w.w = bf16_bits(oh[6] * inv) | (bf16_bits(oh[7] * inv) << 16);
          *reinterpret_cast<uint4*>(ob + 16 * h) = w;
        } else {
          *reinterpret_cast<float4*>(ob + 16 * h) =
              make_float4(oh[0] * inv, oh[1] * inv, oh[2] * inv, oh[3] * inv);
        }
      }
      if (lse != nullptr && sub == 0) lse[row] = (mx + log2f(l)) * kLn2;
    }
  }
}

// ---------------------------------------------------------------------------- launch

template <int D, bool BF16, int NC>
hipError_t fwd_dispatch(const Geometry& g, const void* q, const void* k, const void* v,
                        const float* off, void* out, float* lse, hipStream_t s) {
  const int tiles = tiles_for<D, BF16, NC>(g);
  const int blocks = tiles < kMaxBlocks ? tiles : kMaxBlocks;
  void* args[] = {(void*)&g, (void*)&q, (void*)&k, (void*)&v, (void*)&off, (void*)&out, (void*)&lse,
                  (void*)&tiles};
  return hipLaunchKernel(reinterpret_cast<const void*>(&fwd_kernel<D, BF16, NC>), dim3(blocks),
                         dim3(kBlockThreads), args, 0, s);
}

}  // namespace

hipError_t launch_forward(const Geometry& g, bool bf16, const void* q, const void* k,
                          const void* v, const float* offsets, void* out, float* lse,
                          hipStream_t stream) {
  switch (g.D) {
    case 32:
      return bf16 ? fwd_dispatch<32, true, 1>(g, q, k, v, offsets, out, lse, stream)
                  : fwd_dispatch<32, false, 1>(g, q, k, v, offsets, out, lse, stream);
    case 64:
      return bf16 ? fwd_dispatch<64, true, 1>(g, q, k, v, offsets, out, lse, stream)
                  : fwd_dispatch<64, false, 1>(g, q, k, v, offsets, out, lse, stream);
    case 128:
      return bf16 ? fwd_dispatch<128, true, 1>(g, q, k, v, offsets, out, lse, stream)
                  : fwd_dispatch<128, false, 1>(g, q, k, v, offsets, out, lse, stream);
    default:
      return hipErrorInvalidValue;
  }
}

}  // namespace dsa3d
