// Forward kernel of 3D Deformable Slide Attention (MegaSlide-DiT, Section 5.2, Eq. (1)).
//
// Each L-lane group owns one query row.  For every point it forms the sampling position,
// the 8 trilinear corners and their weights (computed once per row by one lane and shared
// with ds_bpermute), loads the 8 K corner rows and
// the 8 V corner rows (one 16-byte buffer load per lane per row; corners outside the grid
// come back as zeros from the buffer unit), reduces the interpolated logit
// over the group with DPP butterflies (q.K by v_dot2_f32_bf16 on bf16 data, fp32
// accumulation) and folds the point into an online (running-max, base-2) softmax, so each
// corner row is read once.  Nothing per point is written to memory; the output row and
// its LSE are stored once.
//
// Memory order: tiles are handed out in pencils (tile_order.h): each XCD walks one pencil of
// about 16 x 16 tokens of a (batch, head) frame by frame, so the K/V rows its in-flight
// queries reach stay in its L2.
#include "dsa3d_device.h"

namespace dsa3d {
namespace {

using namespace dev;

// Per-point coordinate work shared across the L lanes of a row: in each chunk of L points,
// lane `sub` of a row computes point chunk + sub once and leaves its corner indices, weights
// and cell in its LDS slot (80 bytes), and the row's lanes read each point from there (one
// broadcast read per 16 bytes) instead of every lane repeating the same arithmetic.  Against
// fetching them from the owner's registers with ds_bpermute this keeps 14 fewer registers
// live in the point loop (138) and measured 1% faster; four waves per SIMD (128 registers,
// a few spilled outside the loop) did not pay.
//
// PW (the predicted-weights variant): the logit of a point is given (`logits`, one fp32 per
// (row, point)) instead of scale <q, k_p>, so neither q nor the K corners are read.
template <int D, bool BF16, bool PW>
__global__ __launch_bounds__(kBlockThreads) void fwd_kernel(
    Geometry g, const void* __restrict__ q, const void* __restrict__ k, const void* __restrict__ v,
    const float* __restrict__ logits, const float* __restrict__ offsets, void* __restrict__ out,
    float* __restrict__ lse, PencilOrder po) {
  using LY = Layout<D, BF16>;
  constexpr int L = LY::kLanes;
  constexpr int VEC = LY::kVec;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int grp = lane / L, sub = lane % L;
  const int lane_off = sub * 16;
  const char* qb = static_cast<const char*>(q);
  const char* kb = static_cast<const char*>(k);
  const char* vb = static_cast<const char*>(v);
  const int HW = g.H * g.W;
  const int rt = (g.kt - 1) / 2, rh = (g.kh - 1) / 2, rw = (g.kw - 1) / 2;
  const int khw = g.kh * g.kw;
  // The point each lane formed for the current chunk, read back by its row's lanes: corner
  // indices, weights, and for the global-load path its window flag and cell.  A row's lanes
  // are in one wave, whose LDS accesses complete in order: no barrier.
  __shared__ int4 pts[slot_words<L, 5>()];
  int4* const mine_at = pts + slot_of<L, 5>(threadIdx.x);

  for (int64_t vt = blockIdx.x; vt < po.vtiles; vt += gridDim.x) {
    PencilTile tl;
    if (!pencil_tile(po, vt, tl)) continue;  // the whole block: no pencil left on this XCD
    const int b = tl.group / g.heads, m = tl.group % g.heads;
    const int t = tl.frame;
    const RowWindow win = make_window<LY::kRowBytes>(g, k, v, b, m, t);
    int i, j;
    const bool active = pencil_cell(po, tl, wave * LY::kGroups + grp, i, j);
    if (!active) {  // an idle row computes on a valid token and stores nothing
      i = tl.pr * po.ph;
      j = tl.pc * po.pw;
    }
    const int n = t * HW + i * g.W + j;
    const int64_t row = ((int64_t)b * g.N + n) * g.heads + m;

    uint4 qr = make_uint4(0u, 0u, 0u, 0u);
    if constexpr (!PW) qr = load16(qb, row * LY::kRowBytes + lane_off);
    const float* off = offsets + row * g.P * 3;
    float o[VEC];
#pragma unroll
    for (int e = 0; e < VEC; ++e) o[e] = 0.0f;
    float mx = -INFINITY, l = 0.0f;

    for (int p0 = 0; p0 < g.P; p0 += L) {
      // this lane's point of the chunk
      const int pm = min(p0 + sub, g.P - 1);
      const int it = pm / khw, ih = (pm - it * khw) / g.kw, iw = pm - it * khw - ih * g.kw;
      {
        Point mine;
        make_point(g, win, t, i, j, it - rt, ih - rh, iw - rw, off[3 * pm], off[3 * pm + 1],
                   off[3 * pm + 2], mine);
        mine_at[0] = make_int4(mine.vidx[0], mine.vidx[1], mine.vidx[2], mine.vidx[3]);
        mine_at[1] = make_int4(mine.vidx[4], mine.vidx[5], mine.vidx[6], mine.vidx[7]);
        mine_at[2] = make_int4(__float_as_int(mine.w[0]), __float_as_int(mine.w[1]),
                               __float_as_int(mine.w[2]), __float_as_int(mine.w[3]));
        mine_at[3] = make_int4(__float_as_int(mine.w[4]), __float_as_int(mine.w[5]),
                               __float_as_int(mine.w[6]), __float_as_int(mine.w[7]));
        mine_at[4] = make_int4((int)mine.slow, mine.cx, mine.cy, mine.cz);
      }
      float mylog2 = 0.0f;  // PW: this lane's point's logit, base 2
      if constexpr (PW) mylog2 = logits[row * g.P + pm] * kLog2e;
      const int nk = min(L, g.P - p0);
      for (int kk = 0; kk < nk; ++kk) {
        const int src = (grp * L + kk) << 2;
        const int4* at = pts + slot_of<L, 5>(wave * 64 + grp * L) + kk * 5;
        const int4 i0 = at[0], i1 = at[1], w0 = at[2], w1 = at[3];
        Point pt;
        pt.vidx[0] = i0.x; pt.vidx[1] = i0.y; pt.vidx[2] = i0.z; pt.vidx[3] = i0.w;
        pt.vidx[4] = i1.x; pt.vidx[5] = i1.y; pt.vidx[6] = i1.z; pt.vidx[7] = i1.w;
        pt.w[0] = __int_as_float(w0.x); pt.w[1] = __int_as_float(w0.y);
        pt.w[2] = __int_as_float(w0.z); pt.w[3] = __int_as_float(w0.w);
        pt.w[4] = __int_as_float(w1.x); pt.w[5] = __int_as_float(w1.y);
        pt.w[6] = __int_as_float(w1.z); pt.w[7] = __int_as_float(w1.w);
        uint4 vr[8];
        float s2;
        if constexpr (PW) {
          load_stashed_corners<LY::kRowBytes, false>(g, win, kb, vb, b, m, lane_off, at + 4,
                                                     pt.vidx, nullptr, vr);
          s2 = __int_as_float(__builtin_amdgcn_ds_bpermute(src, __float_as_int(mylog2)));
        } else {
          uint4 kr[8];
          load_stashed_corners<LY::kRowBytes, true>(g, win, kb, vb, b, m, lane_off, at + 4,
                                                    pt.vidx, kr, vr);
          float sp = 0.0f;
#pragma unroll
          for (int c = 0; c < 8; ++c) sp = fmaf(pt.w[c], chunk_dot<BF16>(qr, kr[c]), sp);
          s2 = group_sum<L>(sp) * g.scale_log2;
        }
        // One exponential per point: a new maximum rescales the running sums by
        // 2^(old max - new max) and enters with weight exactly 1; otherwise the point enters
        // with 2^(s - max).  (A first finite logit takes the first branch: 2^-inf = 0.)  A
        // given logit of -inf enters with weight 0 even while the maximum is still -inf,
        // where s - max would be NaN.
        const bool up = s2 > mx;
        float ex = exp2f(up ? mx - s2 : s2 - mx);
        if constexpr (PW) ex = s2 == -INFINITY ? 0.0f : ex;
        const float corr = up ? ex : 1.0f;
        const float e = up ? 1.0f : ex;
        l = fmaf(l, corr, e);
        mx = up ? s2 : mx;
#pragma unroll
        for (int x = 0; x < VEC; ++x) o[x] *= corr;
#pragma unroll
        for (int c = 0; c < 8; ++c) chunk_axpy<BF16>(o, e * pt.w[c], vr[c]);
      }
    }
    if (active) {
      const float inv = 1.0f / l;
      char* ob = static_cast<char*>(out) + row * LY::kRowBytes + lane_off;
      if constexpr (BF16) {
        uint4 wv;
        wv.x = bf16_bits(o[0] * inv) | (bf16_bits(o[1] * inv) << 16);
        wv.y = bf16_bits(o[2] * inv) | (bf16_bits(o[3] * inv) << 16);
        wv.z = bf16_bits(o[4] * inv) | (bf16_bits(o[5] * inv) << 16);
        wv.w = bf16_bits(o[6] * inv) | (bf16_bits(o[7] * inv) << 16);
        *reinterpret_cast<uint4*>(ob) = wv;
      } else {
        *reinterpret_cast<float4*>(ob) = make_float4(o[0] * inv, o[1] * inv, o[2] * inv, o[3] * inv);
      }
      if (lse != nullptr && sub == 0) lse[row] = (mx + log2f(l)) * kLn2;
    }
  }
}

// ---------------------------------------------------------------------------- launch

template <int D, bool BF16>
hipError_t fwd_dispatch(const Geometry& g, const void* q, const void* k, const void* v,
                        const float* logits, const float* off, void* out, float* lse,
                        hipStream_t s) {
  const PencilOrder po = query_order<D, BF16>(g);
  const int blocks = grid_blocks(po.vtiles);
  void* args[] = {(void*)&g,   (void*)&q,   (void*)&k,   (void*)&v,    (void*)&logits,
                  (void*)&off, (void*)&out, (void*)&lse, (void*)&po};
  const void* kern = logits != nullptr ? reinterpret_cast<const void*>(&fwd_kernel<D, BF16, true>)
                                       : reinterpret_cast<const void*>(&fwd_kernel<D, BF16, false>);
  return hipLaunchKernel(kern, dim3(blocks), dim3(kBlockThreads), args, 0, s);
}

}  // namespace

hipError_t launch_forward(const Geometry& g, bool bf16, const void* q, const void* k,
                          const void* v, const float* logits, const float* offsets, void* out,
                          float* lse, hipStream_t stream) {
#define DSA3D_FWD(DIM, BF) fwd_dispatch<DIM, BF>(g, q, k, v, logits, offsets, out, lse, stream)
  switch (g.D) {
    case 32: return bf16 ? DSA3D_FWD(32, true) : DSA3D_FWD(32, false);
    case 64: return bf16 ? DSA3D_FWD(64, true) : DSA3D_FWD(64, false);
    case 128: return bf16 ? DSA3D_FWD(128, true) : DSA3D_FWD(128, false);
    default: return hipErrorInvalidValue;
  }
#undef DSA3D_FWD
}

}  // namespace dsa3d
