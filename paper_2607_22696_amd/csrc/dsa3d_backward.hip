// Backward of 3D Deformable Slide Attention (MegaSlide-DiT, Section 5.2, Eq. (1)).
//
// With alpha_p = softmax weights, da_p = <dout, v_p>, Delta = sum_p alpha_p da_p and
// ds_p = alpha_p (da_p - Delta), the gradients are
//   dq            = scale sum_p ds_p k_p
//   d_offsets[p]  = sum_c dw_c/dpos (scale ds_p <q, K_c> + alpha_p <dout, V_c>)
//   dK[x]         = sum over (query, point, corner c) landing on voxel x of scale ds_p w_c q
//   dV[x]         = the same sum of alpha_p w_c dout
//
// Four phases, none with floating-point atomics:
//  1. V pass (one L-lane group per query row): loads the V corner rows of each point, forms
//     da_p and B_p = sum_c dw_c/dpos <dout, V_c> (the V half of the point's record), and
//     counts the point into the bin of its trilinear cell (the floor of its position) with
//     an integer atomic whose result, the point's rank in the bin, is kept.
//  2. exclusive scan of the bin counts -> bin starts.
//  3. K pass (one L-lane group per query row): loads the K corner rows, forms alpha_p from the
//     logit and the forward's LSE, A_p = sum_c dw_c/dpos <q, K_c>, Delta = sum_p alpha_p da_p
//     and dq, keeping the Delta-dependent part factored until the row's last point,
//       dq = scale (sum_p alpha_p da_p k_p - Delta sum_p alpha_p k_p);
//     then the row's lanes finish its points: d_offsets[p] = alpha_p (scale (da_p - Delta) A_p
//     + B_p), and the point's dK/dV coefficients (scale ds_p, alpha_p) and fractional position
//     go to slot bin start + rank, i.e. sorted by cell.  (alpha_p, A_p) wait for the row's end
//     in registers when the row has at most kHoldChunks chunks of L points, else in the K
//     half of the point's record.
//  4. gather: a voxel is corner c of exactly the points whose cell is voxel - c, so a block
//     of voxels reads the bins of the cells around it, a few runs of adjacent bins, and
//     stores the dK and dV rows of its voxels once.  bf16: one wave per 4 x 2 x 2 block, the
//     sums as matrix products (weights x q / dout rows) on the matrix cores; fp32: one
//     L-lane group per 2 x 2 block of a frame, w_c * coefficient * q and * dout accumulated
//     in registers.
// The predicted-weights variant reads no K: one sweep (phase 1 with the given logits, the
// bin counts' ranks not kept) and a finalize of one thread per point that claims its slot
// from a fill cursor take phases 1 and 3.
#include "dsa3d_device.h"

namespace dsa3d {
namespace {

using namespace dev;

// Per-point records of the backward, in two arrays so that a pass that forms one half
// writes whole lines: the half that needs the K corners (alpha_p, A_p) and the half that needs
// the V corners (da_p, B_p).
struct __align__(16) RecK {
  float alpha, ax, ay, az;
};
struct __align__(16) RecV {
  float dalpha, bx, by, bz;
};

// A point's contribution to dK/dV, stored in the bin of its cell.
struct Entry {
  int32_t n;      // query token within the batch item
  float alpha;    // dV coefficient: alpha_p
  float sds;      // dK coefficient: scale * ds_p
  float fx, fy, fz;  // fractional position inside the cell
};

static_assert(sizeof(RecK) == 16 && sizeof(RecV) == 16 && sizeof(Entry) == 24, "record layout");

// Register budget of the sweep and gather kernels: at head_dim <= 64 (8 rows per wave) three
// waves per SIMD (at most 168 VGPRs) measured faster than the compiler's own allocation; at
// head_dim 128 the unconstrained allocation (two waves) is faster.
#define DSA3D_WAVES_HINT(D) __attribute__((amdgpu_waves_per_eu((D) <= 64 ? 3 : 1)))

constexpr int kScanThreads = 256;
constexpr int kScanItems = 16;
constexpr int kScanBlockItems = kScanThreads * kScanItems;

// Cells are the integer floor positions with at least one corner inside the grid:
// x in [-1, W-1], y in [-1, H-1], z in [-1, T-1]; (T+1)(H+1)(W+1) of them per (b, head).
__host__ __device__ inline int64_t cells_per_bh(const Geometry& g) {
  return (int64_t)(g.T + 1) * (g.H + 1) * (g.W + 1);
}

__device__ inline int64_t cell_index(const Geometry& g, int bh, int x, int y, int z) {
  return (int64_t)bh * cells_per_bh(g) + ((int64_t)(z + 1) * (g.H + 1) + (y + 1)) * (g.W + 1) + (x + 1);
}

__device__ inline bool cell_inside(const Geometry& g, int x, int y, int z) {
  return x >= -1 && x < g.W && y >= -1 && y < g.H && z >= -1 && z < g.T;
}

// ---------------------------------------------------------------------------- 1. sweep

// The predicted-weights variant's sweep (the logit of a point is given, `logits`, so q and the
// K corners are not read and there is no dq; the main operator's V and K passes are below).
// The lanes of a row share each point's coordinate work: in a chunk of L points, lane `sub`
// forms point chunk + sub (position, corners, weights, cell), counts it into its bin, and
// the row's lanes pick the corner indices, fractions and cell up with ds_bpermute; the
// weights are rebuilt from the fractions with the same products.  Lane `sub` also keeps
// that point's record (alpha_p and A_p = 0; da_p and B_p), and the row stores the chunk's
// records as one contiguous block.
template <int D, bool BF16>
__global__ __launch_bounds__(kBlockThreads) DSA3D_WAVES_HINT(D) void bwd_sweep_kernel(
    Geometry g, const void* __restrict__ v, const float* __restrict__ logits,
    const float* __restrict__ offsets, const float* __restrict__ lse,
    const void* __restrict__ dout, RecK* __restrict__ reck, RecV* __restrict__ recv,
    float* __restrict__ delta_out, uint32_t* __restrict__ counts, PencilOrder po) {
  using LY = Layout<D, BF16>;
  constexpr int L = LY::kLanes;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int grp = lane / L, sub = lane % L;
  const int lane_off = sub * 16;
  const char* vb = static_cast<const char*>(v);
  const char* gb = static_cast<const char*>(dout);
  const int HW = g.H * g.W;
  const int rt = (g.kt - 1) / 2, rh = (g.kh - 1) / 2, rw = (g.kw - 1) / 2;
  const int khw = g.kh * g.kw;

  for (int64_t vt = blockIdx.x; vt < po.vtiles; vt += gridDim.x) {
    PencilTile tl;
    if (!pencil_tile(po, vt, tl)) continue;  // the whole block: no pencil left on this XCD
    const int bh = tl.group;
    const int b = bh / g.heads, m = bh % g.heads;
    const int t = tl.frame;
    const RowWindow win = make_window<LY::kRowBytes>(g, v, v, b, m, t);  // V rows only
    int i, j;
    // All lanes of a group share the token: a whole group is idle or active, so neither the
    // group reductions nor the point sharing ever mix an idle group into an active one.
    if (!pencil_cell(po, tl, wave * LY::kGroups + grp, i, j)) continue;
    const int n = t * HW + i * g.W + j;
    const int64_t row = ((int64_t)b * g.N + n) * g.heads + m;

    const uint4 gr = load16(gb, row * LY::kRowBytes + lane_off);
    const float lse2 = lse[row] * kLog2e;
    const float* off = offsets + row * g.P * 3;
    float delta = 0.0f;

    int pm = min(sub, g.P - 1);  // this lane's point of the chunk (clamped in the last one)
    float ox = off[3 * pm], oy = off[3 * pm + 1], oz = off[3 * pm + 2];
    for (int p0 = 0; p0 < g.P; p0 += L) {
      const int it = pm / khw, ih = (pm - it * khw) / g.kw, iw = pm - it * khw - ih * g.kw;
      Point mine;
      make_point(g, win, t, i, j, it - rt, ih - rh, iw - rw, ox, oy, oz, mine);
      const float mylog2 = logits[row * g.P + pm] * kLog2e;  // this lane's point's logit, base 2
      const bool own = p0 + sub < g.P;
      if (own && cell_inside(g, mine.cx, mine.cy, mine.cz))  // result unused: no wait
        __hip_atomic_fetch_add(counts + cell_index(g, bh, mine.cx, mine.cy, mine.cz), 1u,
                               __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      pm = min(p0 + L + sub, g.P - 1);  // next chunk's offsets, in flight during this one
      ox = off[3 * pm];
      oy = off[3 * pm + 1];
      oz = off[3 * pm + 2];
      const int nk = min(L, g.P - p0);
      float4 rec0 = make_float4(0.0f, 0.0f, 0.0f, 0.0f), rec1 = rec0;
      for (int kk = 0; kk < nk; ++kk) {
        const int src = (grp * L + kk) << 2;
        Point pt;
#pragma unroll
        for (int c = 0; c < 8; ++c) pt.vidx[c] = __builtin_amdgcn_ds_bpermute(src, mine.vidx[c]);
        const float tx = __int_as_float(__builtin_amdgcn_ds_bpermute(src, __float_as_int(mine.ax[1])));
        const float ty = __int_as_float(__builtin_amdgcn_ds_bpermute(src, __float_as_int(mine.ay[1])));
        const float tz = __int_as_float(__builtin_amdgcn_ds_bpermute(src, __float_as_int(mine.az[1])));
        pt.ax[0] = 1.0f - tx;
        pt.ax[1] = tx;
        pt.ay[0] = 1.0f - ty;
        pt.ay[1] = ty;
        pt.az[0] = 1.0f - tz;
        pt.az[1] = tz;
        {
          const float wyz[4] = {pt.ay[0] * pt.az[0], pt.ay[1] * pt.az[0], pt.ay[0] * pt.az[1],
                                pt.ay[1] * pt.az[1]};
#pragma unroll
          for (int c = 0; c < 8; ++c) pt.w[c] = pt.ax[c & 1] * wyz[c >> 1];
        }
        uint4 vr[8];
        load_shared_corners<LY::kRowBytes, false>(g, win, vb, vb, b, m, lane_off, mine, src,
                                                  pt.vidx, nullptr, vr);
        float dap = 0.0f, b3[3] = {0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int c = 0; c < 8; ++c) {
          const int cx = c & 1, cy = (c >> 1) & 1, cz = c >> 2;
          const float dvv = chunk_dot<BF16>(gr, vr[c]);
          dap = fmaf(pt.w[c], dvv, dap);
          // d w_c / d pos along each axis (corners outside the grid have zero rows, so zero dots)
          const float wx = cx ? pt.ay[cy] * pt.az[cz] : -(pt.ay[cy] * pt.az[cz]);
          const float wy = cy ? pt.ax[cx] * pt.az[cz] : -(pt.ax[cx] * pt.az[cz]);
          const float wz = cz ? pt.ax[cx] * pt.ay[cy] : -(pt.ax[cx] * pt.ay[cy]);
          b3[0] = fmaf(wx, dvv, b3[0]);
          b3[1] = fmaf(wy, dvv, b3[1]);
          b3[2] = fmaf(wz, dvv, b3[2]);
        }
        const float alpha =
            exp2f(__int_as_float(__builtin_amdgcn_ds_bpermute(src, __float_as_int(mylog2))) - lse2);
        const float da = group_sum<L>(dap);
        delta = fmaf(alpha, da, delta);
#pragma unroll
        for (int a = 0; a < 3; ++a) b3[a] = group_sum<L>(b3[a]);
        if (sub == kk) {
          rec0 = make_float4(alpha, 0.0f, 0.0f, 0.0f);
          rec1 = make_float4(da, b3[0], b3[1], b3[2]);
        }
      }
      if (own) {
        *reinterpret_cast<float4*>(reck + row * g.P + p0 + sub) = rec0;
        *reinterpret_cast<float4*>(recv + row * g.P + p0 + sub) = rec1;
      }
    }
    if (sub == 0) delta_out[row] = delta;
  }
}

// ---------------------------------------------------------------------------- 1b. split sweep
//
// The same work as the sweep in two passes over the points, one over the V corners and one
// over the K corners, so that each pass keeps only one of the two tensors' rows in the L2s.
// The V pass forms da_p = <dout, v_p> and B_p and counts the bins, keeping each point's rank
// in its bin; after the scan, the K pass forms alpha_p, A_p, dq and Delta, and once a row's
// Delta is known its lanes finish the row's points: d_offsets and the point's entry, placed
// at its bin's start + its rank (what the finalize pass does in the one-sweep order).

// The row's points once its Delta is known, NB per lane at a time so that their loads
// (V record halves, offsets, ranks) and then their bin-start lookups are in flight together:
// d_offsets of each point and its entry in the bin of its cell, at slot starts[cell] + rank
// (the point's rank in its bin, from the V pass).  Lane `sub` takes the points sub + c L of
// the row's chunks c; p[u] >= P marks a lane with no point in that chunk.  rk holds the K
// halves of the records (alpha_p, A_p) of those points.  (t, i, j): the query token; n its
// index in the batch item; bh its (batch, head) group.
constexpr int kFinish = 4;
// Chunks of a row whose K record halves the K pass holds in registers (4 VGPRs each): rows of
// up to 80 points at head_dim 128 and 40 at 64 in bf16.
constexpr int kHoldChunks = 5;

template <int NB>
__device__ inline __attribute__((always_inline)) void finish_points(
    const Geometry& g, const RecK (&rk)[NB], const int (&p)[NB],
    const RecV* __restrict__ vrow, const float* __restrict__ off,
    const uint32_t* __restrict__ rrow, float delta, int bh, int n, int t, int i, int j,
    float* __restrict__ drow, const uint32_t* __restrict__ starts, Entry* __restrict__ entries) {
  const int rt = (g.kt - 1) / 2, rh = (g.kh - 1) / 2, rw = (g.kw - 1) / 2;
  RecV rv[NB];
  float o[NB][3];
  uint32_t rank[NB];
#pragma unroll
  for (int u = 0; u < NB; ++u) {
    const int q = min(p[u], g.P - 1);  // no point: a repeat, not stored
    rv[u] = vrow[q];
    o[u][0] = off[3 * q];
    o[u][1] = off[3 * q + 1];
    o[u][2] = off[3 * q + 2];
    rank[u] = rrow[q];
  }
  int cx[NB], cy[NB], cz[NB];
  float fx[NB], fy[NB], fz[NB];
  uint32_t slot[NB];
#pragma unroll
  for (int u = 0; u < NB; ++u) {
    const int q = min(p[u], g.P - 1);
    const int iw = q % g.kw, ih = (q / g.kw) % g.kh, it = q / (g.kw * g.kh);
    axis((float)(j + iw - rw), o[u][0], g.W, cx[u], fx[u]);
    axis((float)(i + ih - rh), o[u][1], g.H, cy[u], fy[u]);
    axis((float)(t + it - rt), o[u][2], g.T, cz[u], fz[u]);
    slot[u] = 0xffffffffu;
    if (cell_inside(g, cx[u], cy[u], cz[u]))
      slot[u] = starts[cell_index(g, bh, cx[u], cy[u], cz[u])] + rank[u];
  }
#pragma unroll
  for (int u = 0; u < NB; ++u) {
    if (p[u] >= g.P) continue;
    const float dd = rv[u].dalpha - delta;
    const float sa = g.scale * dd;
    float* d = drow + 3 * p[u];
    d[0] = rk[u].alpha * fmaf(sa, rk[u].ax, rv[u].bx);
    d[1] = rk[u].alpha * fmaf(sa, rk[u].ay, rv[u].by);
    d[2] = rk[u].alpha * fmaf(sa, rk[u].az, rv[u].bz);
    if (slot[u] == 0xffffffffu) continue;
    Entry e;
    e.n = (int32_t)n;
    e.alpha = rk[u].alpha;
    e.sds = g.scale * rk[u].alpha * dd;
    e.fx = fx[u];
    e.fy = fy[u];
    e.fz = fz[u];
    entries[slot[u]] = e;
  }
}

// All of a row's points.  HOLD > 0: the lane kept the K halves of its points of the row's
// (at most HOLD) chunks in registers, the latest chunk first (hold[h] is chunk nch - 1 - h);
// it finishes them two at a time at 16 or more lanes per row, where the kernel has 128
// registers (four at a time: 129.3 against 127.0 ms at 64x68x120, 3x5x5, head_dim 128, on
// one box).
// HOLD == 0: it stored them in the row's records (krow), and program order makes its own
// stores visible to its loads.
template <int L, int HOLD>
__device__ inline __attribute__((always_inline)) void finish_row(
    const Geometry& g, const RecK* __restrict__ krow, const float4 (&hold)[HOLD > 0 ? HOLD : 1],
    const RecV* __restrict__ vrow, const float* __restrict__ off,
    const uint32_t* __restrict__ rrow, float delta, int bh, int n, int t, int i, int j, int sub,
    float* __restrict__ drow, const uint32_t* __restrict__ starts, Entry* __restrict__ entries) {
  const int nch = (g.P + L - 1) / L;
  // The points' index arithmetic depends only on the lane and the geometry: left visible, the
  // compiler hoists it out of the tile loop for every held chunk and spills it there.
  asm volatile("" : "+v"(sub));
  if constexpr (HOLD > 0) {
    // NB held points per batch of kFinish slots, the other slots empty (p = P): as a batch of
    // two the compiler spills more (125.6 against 123.7 ms at 64x68x120, 3x5x5, head_dim 128)
    constexpr int NB = L >= 16 ? 2 : kFinish;
#pragma unroll
    for (int h0 = 0; h0 < HOLD; h0 += NB) {
      if (h0 >= nch) break;
      int p[kFinish];
      RecK rk[kFinish];
#pragma unroll
      for (int u = 0; u < kFinish; ++u) {
        if (u >= NB) {
          p[u] = g.P;
          rk[u] = RecK{0.0f, 0.0f, 0.0f, 0.0f};
          continue;
        }
        const int c = nch - 1 - (h0 + u);
        p[u] = c >= 0 ? sub + c * L : g.P;
        const float4 r = hold[h0 + u < HOLD ? h0 + u : HOLD - 1];
        rk[u] = RecK{r.x, r.y, r.z, r.w};
      }
      finish_points<kFinish>(g, rk, p, vrow, off, rrow, delta, bh, n, t, i, j, drow, starts,
                             entries);
    }
  } else {
    for (int c0 = 0; c0 < nch; c0 += kFinish) {
      int p[kFinish];
      RecK rk[kFinish];
#pragma unroll
      for (int u = 0; u < kFinish; ++u) {
        p[u] = sub + (c0 + u) * L;
        rk[u] = krow[min(p[u], g.P - 1)];
      }
      finish_points<kFinish>(g, rk, p, vrow, off, rrow, delta, bh, n, t, i, j, drow, starts,
                             entries);
    }
  }
}

// Point setup shared by the two passes: the row's lanes fetch point `kk` of the chunk from the
// lane that formed it (`mine`): corner indices, fractions, and the weights rebuilt from them.
__device__ inline __attribute__((always_inline)) void fetch_point(const Point& mine, int src,
                                                                 Point& pt) {
#pragma unroll
  for (int c = 0; c < 8; ++c) pt.vidx[c] = __builtin_amdgcn_ds_bpermute(src, mine.vidx[c]);
  const float tx = __int_as_float(__builtin_amdgcn_ds_bpermute(src, __float_as_int(mine.ax[1])));
  const float ty = __int_as_float(__builtin_amdgcn_ds_bpermute(src, __float_as_int(mine.ay[1])));
  const float tz = __int_as_float(__builtin_amdgcn_ds_bpermute(src, __float_as_int(mine.az[1])));
  pt.ax[0] = 1.0f - tx;
  pt.ax[1] = tx;
  pt.ay[0] = 1.0f - ty;
  pt.ay[1] = ty;
  pt.az[0] = 1.0f - tz;
  pt.az[1] = tz;
  const float wyz[4] = {pt.ay[0] * pt.az[0], pt.ay[1] * pt.az[0], pt.ay[0] * pt.az[1],
                        pt.ay[1] * pt.az[1]};
#pragma unroll
  for (int c = 0; c < 8; ++c) pt.w[c] = pt.ax[c & 1] * wyz[c >> 1];
}

// V pass: per point da_p = <dout, v_p> and B_p = sum_c dw_c/dpos <dout, V_c> into the V half
// of the record; every point is counted into the bin of its cell.
template <int D, bool BF16>
__global__ __launch_bounds__(kBlockThreads) DSA3D_WAVES_HINT(D) void bwd_vpass_kernel(
    Geometry g, const void* __restrict__ v, const float* __restrict__ offsets,
    const void* __restrict__ dout, RecV* __restrict__ recv, uint32_t* __restrict__ counts,
    uint32_t* __restrict__ ranks, PencilOrder po) {
  using LY = Layout<D, BF16>;
  constexpr int L = LY::kLanes;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int grp = lane / L, sub = lane % L;
  const int lane_off = sub * 16;
  const char* vb = static_cast<const char*>(v);
  const char* gb = static_cast<const char*>(dout);
  const int HW = g.H * g.W;
  const int rt = (g.kt - 1) / 2, rh = (g.kh - 1) / 2, rw = (g.kw - 1) / 2;
  const int khw = g.kh * g.kw;
  // At 16 lanes per row the point each lane formed for the current chunk is read back by its
  // row's lanes from LDS (a row's lanes are one wave, whose LDS accesses complete in order):
  // corner indices, weights, the magnitudes of the weights' position derivatives, window flag
  // and cell (as in the K pass).  At 8 lanes per row (a read then serves 8 rows) the lanes
  // fetch indices and fractions with ds_bpermute and rebuild the rest, which measured faster
  // there (2.98 against 3.10 ms at 64x34x60; 88.7 against 87.2 ms at 64x68x120, head_dim 128).
  constexpr bool kSlots = L >= 16;
  __shared__ int4 pts[kSlots ? slot_words<L, 9>() : 1];  // 8 words used, 9 for the banks
  int4* const mine_at = pts + (kSlots ? slot_of<L, 9>(threadIdx.x) : 0);

  for (int64_t vt = blockIdx.x; vt < po.vtiles; vt += gridDim.x) {
    PencilTile tl;
    if (!pencil_tile(po, vt, tl)) continue;
    const int bh = tl.group;
    const int b = bh / g.heads, m = bh % g.heads;
    const int t = tl.frame;
    const RowWindow win = make_window<LY::kRowBytes>(g, v, v, b, m, t);  // V rows only
    int i, j;
    if (!pencil_cell(po, tl, wave * LY::kGroups + grp, i, j)) continue;  // a whole group idles
    const int n = t * HW + i * g.W + j;
    const int64_t row = ((int64_t)b * g.N + n) * g.heads + m;
    const uint4 gr = load16(gb, row * LY::kRowBytes + lane_off);
    const float* off = offsets + row * g.P * 3;
    int pm = min(sub, g.P - 1);  // this lane's point of the chunk (clamped in the last one)
    float ox = off[3 * pm], oy = off[3 * pm + 1], oz = off[3 * pm + 2];
    for (int p0 = 0; p0 < g.P; p0 += L) {
      const int it = pm / khw, ih = (pm - it * khw) / g.kw, iw = pm - it * khw - ih * g.kw;
      Point mine;
      make_point(g, win, t, i, j, it - rt, ih - rh, iw - rw, ox, oy, oz, mine);
      if constexpr (kSlots) {
        const float* ax = mine.ax;
        const float* ay = mine.ay;
        const float* az = mine.az;
        mine_at[0] = make_int4(mine.vidx[0], mine.vidx[1], mine.vidx[2], mine.vidx[3]);
        mine_at[1] = make_int4(mine.vidx[4], mine.vidx[5], mine.vidx[6], mine.vidx[7]);
        mine_at[2] = make_int4(__float_as_int(mine.w[0]), __float_as_int(mine.w[1]),
                               __float_as_int(mine.w[2]), __float_as_int(mine.w[3]));
        mine_at[3] = make_int4(__float_as_int(mine.w[4]), __float_as_int(mine.w[5]),
                               __float_as_int(mine.w[6]), __float_as_int(mine.w[7]));
        mine_at[4] = make_int4(__float_as_int(ay[0] * az[0]), __float_as_int(ay[1] * az[0]),
                               __float_as_int(ay[0] * az[1]), __float_as_int(ay[1] * az[1]));
        mine_at[5] = make_int4(__float_as_int(ax[0] * az[0]), __float_as_int(ax[1] * az[0]),
                               __float_as_int(ax[0] * az[1]), __float_as_int(ax[1] * az[1]));
        mine_at[6] = make_int4(__float_as_int(ax[0] * ay[0]), __float_as_int(ax[1] * ay[0]),
                               __float_as_int(ax[0] * ay[1]), __float_as_int(ax[1] * ay[1]));
        mine_at[7] = make_int4((int)mine.slow, mine.cx, mine.cy, mine.cz);
      }
      const bool own = p0 + sub < g.P;
      // the point's rank in its bin: the K pass puts its entry at bin start + rank (the
      // returning atomic's latency is covered by the chunk's corner loads)
      uint32_t rank = 0u;
      if (own && cell_inside(g, mine.cx, mine.cy, mine.cz))
        rank = __hip_atomic_fetch_add(counts + cell_index(g, bh, mine.cx, mine.cy, mine.cz), 1u,
                                      __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      pm = min(p0 + L + sub, g.P - 1);  // next chunk's offsets, in flight during this one
      ox = off[3 * pm];
      oy = off[3 * pm + 1];
      oz = off[3 * pm + 2];
      const int nk = min(L, g.P - p0);
      float4 rec = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
      for (int kk = 0; kk < nk; ++kk) {
        uint4 vr[8];
        float w[8], gx[4], gy[4], gz[4];
        if constexpr (!kSlots) {
          const int src = (grp * L + kk) << 2;
          Point pt;
          fetch_point(mine, src, pt);
          load_shared_corners<LY::kRowBytes, false>(g, win, vb, vb, b, m, lane_off, mine, src,
                                                    pt.vidx, nullptr, vr);
#pragma unroll
          for (int c = 0; c < 8; ++c) w[c] = pt.w[c];
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            gx[e] = pt.ay[e & 1] * pt.az[e >> 1];
            gy[e] = pt.ax[e & 1] * pt.az[e >> 1];
            gz[e] = pt.ax[e & 1] * pt.ay[e >> 1];
          }
        } else {
          const int4* at = pts + slot_of<L, 9>(wave * 64 + grp * L) + kk * 9;
          int vidx[8];
          const int4 i0 = at[0], i1 = at[1];
          vidx[0] = i0.x; vidx[1] = i0.y; vidx[2] = i0.z; vidx[3] = i0.w;
          vidx[4] = i1.x; vidx[5] = i1.y; vidx[6] = i1.z; vidx[7] = i1.w;
          load_stashed_corners<LY::kRowBytes, false>(g, win, vb, vb, b, m, lane_off, at + 7,
                                                     vidx, nullptr, vr);
          const int4 w0 = at[2], w1 = at[3], x4 = at[4], y4 = at[5], z4 = at[6];
          w[0] = __int_as_float(w0.x); w[1] = __int_as_float(w0.y);
          w[2] = __int_as_float(w0.z); w[3] = __int_as_float(w0.w);
          w[4] = __int_as_float(w1.x); w[5] = __int_as_float(w1.y);
          w[6] = __int_as_float(w1.z); w[7] = __int_as_float(w1.w);
          gx[0] = __int_as_float(x4.x); gx[1] = __int_as_float(x4.y);
          gx[2] = __int_as_float(x4.z); gx[3] = __int_as_float(x4.w);
          gy[0] = __int_as_float(y4.x); gy[1] = __int_as_float(y4.y);
          gy[2] = __int_as_float(y4.z); gy[3] = __int_as_float(y4.w);
          gz[0] = __int_as_float(z4.x); gz[1] = __int_as_float(z4.y);
          gz[2] = __int_as_float(z4.z); gz[3] = __int_as_float(z4.w);
        }
        float dap = 0.0f, b3[3] = {0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int c = 0; c < 8; ++c) {
          const int cx = c & 1, cy = (c >> 1) & 1, cz = c >> 2;
          const float dvv = chunk_dot<BF16>(gr, vr[c]);
          dap = fmaf(w[c], dvv, dap);
          b3[0] = fmaf(cx ? gx[c >> 1] : -gx[c >> 1], dvv, b3[0]);
          b3[1] = fmaf(cy ? gy[cx + 2 * cz] : -gy[cx + 2 * cz], dvv, b3[1]);
          b3[2] = fmaf(cz ? gz[c & 3] : -gz[c & 3], dvv, b3[2]);
        }
        const float da = group_sum<L>(dap);
#pragma unroll
        for (int a = 0; a < 3; ++a) b3[a] = group_sum<L>(b3[a]);
        if (sub == kk) rec = make_float4(da, b3[0], b3[1], b3[2]);
      }
      if (own) {
        *reinterpret_cast<float4*>(recv + row * g.P + p0 + sub) = rec;
        ranks[row * g.P + p0 + sub] = rank;
      }
    }
  }
}

// K pass: alpha_p from the logit and the forward's LSE, A_p = sum_c dw_c/dpos <q, K_c> (the
// K half of the point's record), Delta = sum_p alpha_p da_p and dq; then, with Delta known, the
// row's lanes finish its points (finish_row).  Needs the V pass's records and the bin starts.
// HOLD > 0 (rows of at most HOLD chunks of L points): each lane keeps the K halves of its
// points in registers until the row's end; HOLD == 0: it writes them to the records and reads
// them back.  Holding them measured 131.4 -> 127.0 ms at 64x68x120 (3x5x5, head_dim 128) and
// 4.76 -> 4.37 ms at 64x34x60 (3x3x3, head_dim 64).
template <int D, bool BF16, int HOLD>
// Four waves per SIMD at head_dim 128 with bf16 (128 registers, 40 bytes spilled outside the
// point loop): 133.2 -> 131.5 ms at 64x68x120 (3x5x5), 240.0 -> 236.0 ms (3x7x7); at head_dim
// 64 the same hint cost 4% (4.81 -> 5.00 ms at 64x34x60), so three stay there.
__global__ __launch_bounds__(kBlockThreads) __attribute__((
    amdgpu_waves_per_eu((D) <= 64 ? 3 : (BF16 ? 4 : 1)))) void bwd_kpass_kernel(
    Geometry g, const void* __restrict__ q, const void* __restrict__ k,
    const float* __restrict__ offsets, const float* __restrict__ lse, float* __restrict__ dq,
    RecK* __restrict__ reck, const RecV* __restrict__ recv, const uint32_t* __restrict__ starts,
    const uint32_t* __restrict__ ranks, float* __restrict__ doff, Entry* __restrict__ entries,
    PencilOrder po) {
  using LY = Layout<D, BF16>;
  constexpr int L = LY::kLanes;
  constexpr int VEC = LY::kVec;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int grp = lane / L, sub = lane % L;
  const int lane_off = sub * 16;
  const char* qb = static_cast<const char*>(q);
  const char* kb = static_cast<const char*>(k);
  const int HW = g.H * g.W;
  const int rt = (g.kt - 1) / 2, rh = (g.kh - 1) / 2, rw = (g.kw - 1) / 2;
  const int khw = g.kh * g.kw;
  // The point each lane formed for the current chunk, read back by its row's lanes (a row's
  // lanes are one wave, whose LDS accesses complete in order): corner indices, weights, the
  // magnitudes of the weights' position derivatives (the products of two axis weights),
  // window flag and cell, and the point's da_p.  The owner forms them once instead of every
  // lane of the row rebuilding them, which the VALU-bound point loop feels.
  __shared__ int4 pts[slot_words<L, 9>()];
  int4* const mine_at = pts + slot_of<L, 9>(threadIdx.x);

  for (int64_t vt = blockIdx.x; vt < po.vtiles; vt += gridDim.x) {
    PencilTile tl;
    if (!pencil_tile(po, vt, tl)) continue;
    const int bh = tl.group;
    const int b = bh / g.heads, m = bh % g.heads;
    const int t = tl.frame;
    const RowWindow win = make_window<LY::kRowBytes>(g, k, k, b, m, t);  // K rows only
    int i, j;
    if (!pencil_cell(po, tl, wave * LY::kGroups + grp, i, j)) continue;  // a whole group idles
    const int n = t * HW + i * g.W + j;
    const int64_t row = ((int64_t)b * g.N + n) * g.heads + m;
    const uint4 qr = load16(qb, row * LY::kRowBytes + lane_off);
    const float lse2 = lse[row] * kLog2e;
    const float* off = offsets + row * g.P * 3;
    RecK* krow = reck + row * g.P;
    const RecV* vrow = recv + row * g.P;
    float ak[VEC], bk[VEC];
#pragma unroll
    for (int x = 0; x < VEC; ++x) {
      ak[x] = 0.0f;
      bk[x] = 0.0f;
    }
    float delta = 0.0f;
    float4 hold[HOLD > 0 ? HOLD : 1];
#pragma unroll
    for (int h = 0; h < (HOLD > 0 ? HOLD : 1); ++h) hold[h] = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
    int pm = min(sub, g.P - 1);
    float ox = off[3 * pm], oy = off[3 * pm + 1], oz = off[3 * pm + 2];
    for (int p0 = 0; p0 < g.P; p0 += L) {
      const int it = pm / khw, ih = (pm - it * khw) / g.kw, iw = pm - it * khw - ih * g.kw;
      {
        Point mine;
        make_point(g, win, t, i, j, it - rt, ih - rh, iw - rw, ox, oy, oz, mine);
        const float my_da = vrow[pm].dalpha;  // this lane's point's da_p (V pass)
        const float* ax = mine.ax;
        const float* ay = mine.ay;
        const float* az = mine.az;
        mine_at[0] = make_int4(mine.vidx[0], mine.vidx[1], mine.vidx[2], mine.vidx[3]);
        mine_at[1] = make_int4(mine.vidx[4], mine.vidx[5], mine.vidx[6], mine.vidx[7]);
        mine_at[2] = make_int4(__float_as_int(mine.w[0]), __float_as_int(mine.w[1]),
                               __float_as_int(mine.w[2]), __float_as_int(mine.w[3]));
        mine_at[3] = make_int4(__float_as_int(mine.w[4]), __float_as_int(mine.w[5]),
                               __float_as_int(mine.w[6]), __float_as_int(mine.w[7]));
        // |dw_c/dx| = ay az, |dw_c/dy| = ax az, |dw_c/dz| = ax ay, by the corner's other two bits
        mine_at[4] = make_int4(__float_as_int(ay[0] * az[0]), __float_as_int(ay[1] * az[0]),
                               __float_as_int(ay[0] * az[1]), __float_as_int(ay[1] * az[1]));
        mine_at[5] = make_int4(__float_as_int(ax[0] * az[0]), __float_as_int(ax[1] * az[0]),
                               __float_as_int(ax[0] * az[1]), __float_as_int(ax[1] * az[1]));
        mine_at[6] = make_int4(__float_as_int(ax[0] * ay[0]), __float_as_int(ax[1] * ay[0]),
                               __float_as_int(ax[0] * ay[1]), __float_as_int(ax[1] * ay[1]));
        mine_at[7] = make_int4((int)mine.slow, mine.cx, mine.cy, mine.cz);
        mine_at[8] = make_int4(__float_as_int(my_da), 0, 0, 0);
      }
      const bool own = p0 + sub < g.P;
      pm = min(p0 + L + sub, g.P - 1);
      ox = off[3 * pm];
      oy = off[3 * pm + 1];
      oz = off[3 * pm + 2];
      const int nk = min(L, g.P - p0);
      float4 rec = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
      for (int kk = 0; kk < nk; ++kk) {
        const int4* at = pts + slot_of<L, 9>(wave * 64 + grp * L) + kk * 9;
        int vidx[8];
        {
          const int4 i0 = at[0], i1 = at[1];
          vidx[0] = i0.x; vidx[1] = i0.y; vidx[2] = i0.z; vidx[3] = i0.w;
          vidx[4] = i1.x; vidx[5] = i1.y; vidx[6] = i1.z; vidx[7] = i1.w;
        }
        uint4 kr[8];
        load_stashed_corners<LY::kRowBytes, false>(g, win, kb, kb, b, m, lane_off, at + 7, vidx,
                                                   nullptr, kr);
        float w[8], gx[4], gy[4], gz[4];
        {
          const int4 w0 = at[2], w1 = at[3], x4 = at[4], y4 = at[5], z4 = at[6];
          w[0] = __int_as_float(w0.x); w[1] = __int_as_float(w0.y);
          w[2] = __int_as_float(w0.z); w[3] = __int_as_float(w0.w);
          w[4] = __int_as_float(w1.x); w[5] = __int_as_float(w1.y);
          w[6] = __int_as_float(w1.z); w[7] = __int_as_float(w1.w);
          gx[0] = __int_as_float(x4.x); gx[1] = __int_as_float(x4.y);
          gx[2] = __int_as_float(x4.z); gx[3] = __int_as_float(x4.w);
          gy[0] = __int_as_float(y4.x); gy[1] = __int_as_float(y4.y);
          gy[2] = __int_as_float(y4.z); gy[3] = __int_as_float(y4.w);
          gz[0] = __int_as_float(z4.x); gz[1] = __int_as_float(z4.y);
          gz[2] = __int_as_float(z4.z); gz[3] = __int_as_float(z4.w);
        }
        float sp = 0.0f, a3[3] = {0.0f, 0.0f, 0.0f};
        float kp[VEC];
#pragma unroll
        for (int x = 0; x < VEC; ++x) kp[x] = 0.0f;
#pragma unroll
        for (int c = 0; c < 8; ++c) {
          const int cx = c & 1, cy = (c >> 1) & 1, cz = c >> 2;
          const float qk = chunk_dot<BF16>(qr, kr[c]);
          sp = fmaf(w[c], qk, sp);
          // dw_c/dpos: + for the upper corner of an axis, - for the lower
          a3[0] = fmaf(cx ? gx[c >> 1] : -gx[c >> 1], qk, a3[0]);
          a3[1] = fmaf(cy ? gy[cx + 2 * cz] : -gy[cx + 2 * cz], qk, a3[1]);
          a3[2] = fmaf(cz ? gz[c & 3] : -gz[c & 3], qk, a3[2]);
          chunk_axpy<BF16>(kp, w[c], kr[c]);
        }
        const float alpha = exp2f(group_sum<L>(sp) * g.scale_log2 - lse2);
        const float da = __int_as_float(at[8].x);
        delta = fmaf(alpha, da, delta);
        const float ada = alpha * da;
#pragma unroll
        for (int x = 0; x < VEC; ++x) {
          ak[x] = fmaf(ada, kp[x], ak[x]);
          bk[x] = fmaf(alpha, kp[x], bk[x]);
        }
#pragma unroll
        for (int a = 0; a < 3; ++a) a3[a] = group_sum<L>(a3[a]);
        if (sub == kk) rec = make_float4(alpha, a3[0], a3[1], a3[2]);
      }
      if constexpr (HOLD > 0) {
#pragma unroll
        for (int h = HOLD - 1; h > 0; --h) hold[h] = hold[h - 1];
        hold[0] = rec;
      } else {
        if (own) *reinterpret_cast<float4*>(krow + p0 + sub) = rec;
      }
    }
    float* dqr = dq + row * D + sub * VEC;
#pragma unroll
    for (int x = 0; x < VEC; x += 4)
      *reinterpret_cast<float4*>(dqr + x) =
          make_float4(g.scale * fmaf(-delta, bk[x], ak[x]), g.scale * fmaf(-delta, bk[x + 1], ak[x + 1]),
                      g.scale * fmaf(-delta, bk[x + 2], ak[x + 2]),
                      g.scale * fmaf(-delta, bk[x + 3], ak[x + 3]));
    // Delta is known: finish the row's points
    finish_row<L, HOLD>(g, krow, hold, vrow, off, ranks + row * g.P, delta, bh, n, t, i, j, sub,
                        doff + row * g.P * 3, starts, entries);
  }
}

// ---------------------------------------------------------------------------- 2. scan

__global__ __launch_bounds__(kBlockThreads) void fill_u32_kernel(uint32_t* __restrict__ a, int64_t n,
                                                                  uint32_t value) {
  for (int64_t x = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; x < n;
       x += (int64_t)gridDim.x * blockDim.x)
    a[x] = value;
}

// Exclusive scan of one 256-thread block's per-thread values; returns the block total.
__device__ inline uint32_t block_exclusive_scan(uint32_t v, uint32_t* lds_waves, uint32_t& excl) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  uint32_t incl = v;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const uint32_t o = __shfl_up(incl, d);
    if (lane >= d) incl += o;
  }
  if (lane == 63) lds_waves[wave] = incl;
  __syncthreads();
  uint32_t wave_off = 0, total = 0;
#pragma unroll
  for (int w = 0; w < kScanThreads / 64; ++w) {
    const uint32_t s = lds_waves[w];
    if (w < wave) wave_off += s;
    total += s;
  }
  __syncthreads();
  excl = wave_off + incl - v;
  return total;
}

// Block sums of kScanBlockItems items each.
__global__ __launch_bounds__(kScanThreads) void scan_reduce_kernel(const uint32_t* __restrict__ in,
                                                                    uint32_t* __restrict__ sums,
                                                                    int64_t n) {
  __shared__ uint32_t lds[kScanThreads / 64];
  const int64_t base = (int64_t)blockIdx.x * kScanBlockItems + (int64_t)threadIdx.x * kScanItems;
  uint32_t s = 0;
#pragma unroll
  for (int e = 0; e < kScanItems; ++e)
    if (base + e < n) s += in[base + e];
  uint32_t excl;
  const uint32_t total = block_exclusive_scan(s, lds, excl);
  if (threadIdx.x == 0) sums[blockIdx.x] = total;
}

// Exclusive scan of the block sums in place (one block, chunk by chunk); writes the grand
// total to *grand.
__global__ __launch_bounds__(kScanThreads) void scan_sums_kernel(uint32_t* __restrict__ sums,
                                                                  int64_t nsums,
                                                                  uint32_t* __restrict__ grand) {
  __shared__ uint32_t lds[kScanThreads / 64];
  uint32_t carry = 0;
  for (int64_t base = 0; base < nsums; base += kScanThreads) {
    const int64_t x = base + threadIdx.x;
    const uint32_t v = x < nsums ? sums[x] : 0u;
    uint32_t excl;
    const uint32_t total = block_exclusive_scan(v, lds, excl);
    if (x < nsums) sums[x] = carry + excl;
    carry += total;
  }
  if (threadIdx.x == 0) *grand = carry;
}

// starts[x] = cursor[x] = offset of block + exclusive scan inside the block.
__global__ __launch_bounds__(kScanThreads) void scan_apply_kernel(const uint32_t* __restrict__ in,
                                                                   const uint32_t* __restrict__ sums,
                                                                   uint32_t* __restrict__ out,
                                                                   uint32_t* __restrict__ cursor,
                                                                   int64_t n) {
  __shared__ uint32_t lds[kScanThreads / 64];
  const int64_t base = (int64_t)blockIdx.x * kScanBlockItems + (int64_t)threadIdx.x * kScanItems;
  uint32_t vals[kScanItems];
  uint32_t s = 0;
#pragma unroll
  for (int e = 0; e < kScanItems; ++e) {
    vals[e] = base + e < n ? in[base + e] : 0u;
    s += vals[e];
  }
  uint32_t excl;
  block_exclusive_scan(s, lds, excl);
  uint32_t run = sums[blockIdx.x] + excl;
#pragma unroll
  for (int e = 0; e < kScanItems; ++e) {
    if (base + e < n) {
      out[base + e] = run;
      cursor[base + e] = run;
    }
    run += vals[e];
  }
}

// ---------------------------------------------------------------------------- 3. finalize

// dlogits (the predicted-weights variant, else null) receives alpha_p (da_p - Delta).
__global__ __launch_bounds__(kBlockThreads) void bwd_finalize_kernel(
    Geometry g, const float* __restrict__ offsets, const RecK* __restrict__ reck,
    const RecV* __restrict__ recv,
    const float* __restrict__ delta, uint32_t* __restrict__ cursor, float* __restrict__ doff,
    float* __restrict__ dlogits, Entry* __restrict__ entries, int npoints) {
  const int rt = (g.kt - 1) / 2, rh = (g.kh - 1) / 2, rw = (g.kw - 1) / 2;
  const unsigned P = g.P, heads = g.heads, N = g.N, W = g.W, HW = g.H * g.W;
  for (unsigned idx = blockIdx.x * blockDim.x + threadIdx.x; idx < (unsigned)npoints;
       idx += gridDim.x * blockDim.x) {
    const unsigned row = idx / P;
    const unsigned p = idx - row * P;
    const RecK rk = reck[idx];
    const RecV rv = recv[idx];
    const float dd = rv.dalpha - delta[row];
    float* d = doff + (size_t)idx * 3;
    const float sa = g.scale * dd;
    d[0] = rk.alpha * fmaf(sa, rk.ax, rv.bx);
    d[1] = rk.alpha * fmaf(sa, rk.ay, rv.by);
    d[2] = rk.alpha * fmaf(sa, rk.az, rv.bz);
    if (dlogits != nullptr) dlogits[idx] = rk.alpha * dd;
    const unsigned tok = row / heads;
    const unsigned m = row - tok * heads;
    const unsigned b = tok / N;
    const unsigned n = tok - b * N;
    const unsigned t = n / HW;
    const unsigned rem = n - t * HW;
    const unsigned i = rem / W;
    const unsigned j = rem - i * W;
    const unsigned iw = p % g.kw, ih = (p / g.kw) % g.kh, it = p / (g.kw * g.kh);
    const float* o = offsets + (size_t)idx * 3;
    int x, y, z;
    float fx, fy, fz;
    axis((float)((int)j + (int)iw - rw), o[0], g.W, x, fx);
    axis((float)((int)i + (int)ih - rh), o[1], g.H, y, fy);
    axis((float)((int)t + (int)it - rt), o[2], g.T, z, fz);
    if (!cell_inside(g, x, y, z)) continue;
    const uint32_t slot = atomicAdd(cursor + cell_index(g, b * heads + m, x, y, z), 1u);
    Entry e;
    e.n = (int32_t)n;
    e.alpha = rk.alpha;
    e.sds = g.scale * rk.alpha * dd;
    e.fx = fx;
    e.fy = fy;
    e.fz = fz;
    entries[slot] = e;
  }
}

// ---------------------------------------------------------------------------- 4. gather

constexpr int kGatherUnroll = 4;  // bin entries processed per iteration

// Per-lane dK/dV accumulators of a group's 2 x 2 voxel block: voxel v = 2 * yi + xi.
template <int VEC>
struct BlockAcc {
  float k[4][VEC];
  float v[4][VEC];
};

// One run of bins: the cells (x0 - 1, x0, x0 + 1) of cell row y0 - 1 + YR in one z plane,
// contiguous in the bin order.  Cell row y0 - 1 feeds voxel row y0 (as its upper y corner),
// cell row y0 feeds both rows (lower corner of y0, upper of y0 + 1) and cell row y0 + 1 feeds
// row y0 + 1 (as its lower corner); YR is the same for every group of a wave, so each case is
// its own code and a run touches only the accumulators of the rows it feeds.  Along x the
// voxel x0 is the upper corner of cell x0 - 1 and the lower of cell x0, the voxel x0 + 1 the
// upper of x0 and the lower of x0 + 1: [s0, m1), [m1, m2), [m2, end).  `zlow` says whether
// the voxels are the lower z corner of this plane's cells.  Entries are read one batch
// ahead, so a batch waits for its rows only.
template <int D, bool BF16, bool PW, int YR>
__device__ inline __attribute__((always_inline)) void gather_run(
    const char* __restrict__ qh, const char* __restrict__ gh, uint32_t tok_bytes,
    const Entry* __restrict__ entries, uint32_t s0, uint32_t m1, uint32_t m2, uint32_t end,
    bool zlow, BlockAcc<Layout<D, BF16>::kVec>& acc) {
  using LY = Layout<D, BF16>;
  constexpr int VEC = LY::kVec;
  constexpr int U = kGatherUnroll;
  if (s0 >= end) return;
  Entry en[U];
#pragma unroll
  for (int k = 0; k < U; ++k) en[k] = entries[min(s0 + k, end - 1)];
  for (uint32_t u = s0; u < end; u += U) {
    uint4 qr[U], gr[U];
#pragma unroll
    for (int k = 0; k < U; ++k) {
      const uint64_t o = (uint64_t)(uint32_t)en[k].n * tok_bytes;
      if constexpr (!PW) qr[k] = *reinterpret_cast<const uint4*>(qh + o);
      gr[k] = *reinterpret_cast<const uint4*>(gh + o);
    }
    Entry nx[U];
#pragma unroll
    for (int k = 0; k < U; ++k) nx[k] = entries[min(u + U + k, end - 1)];
#pragma unroll
    for (int k = 0; k < U; ++k) {
      const uint32_t uk = u + k;
      const float wz = uk < end ? (zlow ? 1.0f - en[k].fz : en[k].fz) : 0.0f;
      const float lo = 1.0f - en[k].fx;
      const float tx0 = wz * (uk < m1 ? en[k].fx : (uk < m2 ? lo : 0.0f));
      const float tx1 = wz * (uk < m1 ? 0.0f : (uk < m2 ? en[k].fx : lo));
      float qf[VEC], gf[VEC];
      if constexpr (!PW) chunk_to_float<BF16>(qr[k], qf);
      chunk_to_float<BF16>(gr[k], gf);
#pragma unroll
      for (int yi = 0; yi < 2; ++yi) {
        if ((YR == 0 && yi == 1) || (YR == 2 && yi == 0)) continue;
        // lower y corner for (YR, yi) = (1, 0), (2, 1); upper for (0, 0), (1, 1)
        const float wy = (YR - yi == 1) ? 1.0f - en[k].fy : en[k].fy;
        const float sk = en[k].sds * wy, sv = en[k].alpha * wy;
        const float k0 = sk * tx0, k1 = sk * tx1, v0 = sv * tx0, v1 = sv * tx1;
#pragma unroll
        for (int e = 0; e < VEC; ++e) {
          if constexpr (!PW) {
            acc.k[2 * yi][e] = fmaf(k0, qf[e], acc.k[2 * yi][e]);
            acc.k[2 * yi + 1][e] = fmaf(k1, qf[e], acc.k[2 * yi + 1][e]);
          }
          acc.v[2 * yi][e] = fmaf(v0, gf[e], acc.v[2 * yi][e]);
          acc.v[2 * yi + 1][e] = fmaf(v1, gf[e], acc.v[2 * yi + 1][e]);
        }
      }
    }
#pragma unroll
    for (int k = 0; k < U; ++k) en[k] = nx[k];
  }
}

// Each L-lane group owns the 2 x 2 block of voxels (x0..x0+1, y0..y0+1) of one frame z.  The
// block's voxels are corners of the points in the 3 x 3 cells (x0-1..x0+1, y0-1..y0+1) of
// the planes z - 1 and z: six runs of three adjacent bins, and each entry's q and dout rows
// are loaded once per run for all the voxels it feeds.
// PW (the predicted-weights variant): dV only (there is no K).
template <int D, bool BF16, bool PW>
__global__ __launch_bounds__(kBlockThreads) DSA3D_WAVES_HINT(D) void bwd_gather_kernel(
    Geometry g, const void* __restrict__ q, const void* __restrict__ dout,
    const uint32_t* __restrict__ starts, const Entry* __restrict__ entries, float* __restrict__ dk,
    float* __restrict__ dv, PencilOrder po) {
  using LY = Layout<D, BF16>;
  constexpr int L = LY::kLanes;
  constexpr int VEC = LY::kVec;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int grp = lane / L, sub = lane % L;
  const uint32_t tok_bytes = (uint32_t)g.heads * LY::kRowBytes;  // one token's rows, all heads

  for (int64_t vt = blockIdx.x; vt < po.vtiles; vt += gridDim.x) {
    PencilTile tl;
    if (!pencil_tile(po, vt, tl)) continue;
    const int bh = tl.group;
    const int b = bh / g.heads, m = bh % g.heads;
    int by, bx;  // the group's 2 x 2 block (cell of the pencil grid)
    if (!pencil_cell(po, tl, wave * LY::kGroups + grp, by, bx)) continue;
    const int64_t head_off = ((int64_t)b * g.N * g.heads + m) * LY::kRowBytes + sub * 16;
    const char* qh = static_cast<const char*>(q) + head_off;
    const char* gh = static_cast<const char*>(dout) + head_off;
    const int x0 = 2 * bx, y0 = 2 * by, z = tl.frame;
    const bool hasx1 = x0 + 1 < g.W, hasy1 = y0 + 1 < g.H;
    BlockAcc<VEC> acc;
#pragma unroll
    for (int c = 0; c < 4; ++c) {
#pragma unroll
      for (int e = 0; e < VEC; ++e) {
        acc.k[c][e] = 0.0f;
        acc.v[c][e] = 0.0f;
      }
    }
#pragma unroll 1
    for (int cz = 0; cz < 2; ++cz) {  // cell plane z - 1 + cz; voxel z is its upper corner for cz = 0
      uint32_t r[3][4];
#pragma unroll
      for (int yr = 0; yr < 3; ++yr) {
        if (yr == 2 && !hasy1) {  // cell row y0 + 1 is outside the cell grid: nothing to gather
          r[yr][0] = r[yr][1] = r[yr][2] = r[yr][3] = 0u;
          continue;
        }
        const int64_t ci = cell_index(g, bh, x0 - 1, y0 - 1 + yr, z - 1 + cz);
        r[yr][0] = starts[ci];
        r[yr][1] = starts[ci + 1];
        r[yr][2] = starts[ci + 2];
        r[yr][3] = hasx1 ? starts[ci + 3] : r[yr][2];
      }
      const bool zlow = cz == 1;
      gather_run<D, BF16, PW, 0>(qh, gh, tok_bytes, entries, r[0][0], r[0][1], r[0][2], r[0][3], zlow, acc);
      gather_run<D, BF16, PW, 1>(qh, gh, tok_bytes, entries, r[1][0], r[1][1], r[1][2], r[1][3], zlow, acc);
      gather_run<D, BF16, PW, 2>(qh, gh, tok_bytes, entries, r[2][0], r[2][1], r[2][2], r[2][3], zlow, acc);
    }
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int xi = c & 1, yi = c >> 1;
      if ((xi == 1 && !hasx1) || (yi == 1 && !hasy1)) continue;
      const int64_t row =
          ((int64_t)b * g.N + (int64_t)(z * g.H + y0 + yi) * g.W + x0 + xi) * g.heads + m;
      float* dkr = dk + row * D + sub * VEC;
      float* dvr = dv + row * D + sub * VEC;
#pragma unroll
      for (int e = 0; e < VEC; e += 4) {
        if constexpr (!PW)
          *reinterpret_cast<float4*>(dkr + e) =
              make_float4(acc.k[c][e], acc.k[c][e + 1], acc.k[c][e + 2], acc.k[c][e + 3]);
        *reinterpret_cast<float4*>(dvr + e) =
            make_float4(acc.v[c][e], acc.v[c][e + 1], acc.v[c][e + 2], acc.v[c][e + 3]);
      }
    }
  }
}

// ------------------------------------------------------- 4b. gather on the matrix cores (bf16)
//
// For bf16 rows the gather's sums are matrix products.  For a block of voxels and a batch of
// bin entries e (points with query token n_e, coefficients sds_e and alpha_e, fractions f_e),
//   dK[voxel] += sum_e W[voxel][e] sds_e q[n_e],   dV[voxel] += sum_e W[voxel][e] alpha_e dout[n_e],
// W being the trilinear weight of the voxel as a corner of the entry's cell (zero when it is
// not one of its corners).  A wave owns the 4 x 2 x 2 voxel block (x0..x0+3, y0..y0+1,
// z0..z0+1), whose points lie in the 5 x 3 x 3 cells (x0-1..x0+3, y0-1..y0+1, z0-1..z0+1):
// nine runs of five adjacent bins.  Per batch of 32 entries of one run
//  * the lanes that own an entry (lane e for its dK coefficient, lane e + 32 for dV) form its
//    16 weighted coefficients (voxel v = vx + 4 vy + 8 vz) and store them as row e of A_hi^T
//    (the upper half of each fp32 value) and of A_lo^T (the remainder rounded to bf16):
//    hi + lo carries about 16 significant bits;
//  * the wave copies the entries' q and dout rows into LDS;
//  * v_mfma_f32_16x16x32_bf16 multiplies A_hi and A_lo (16 voxels x 32 entries) into the same
//    accumulators by the rows (32 entries x 16 channels per product), both operands read with
//    the transposing ds_read_b64_tr_b16.
// Entries are loaded two batches ahead of the products and rows one batch ahead.  Each wave
// has its own LDS and the LDS operations of a wave complete in order, so there are no barriers.

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef short s16x4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s16x4_t lds_s16x4_t;

constexpr int kGB = 32;  // entries per batch: the products' K

// Waves per workgroup.  The LDS of a wave grows with head_dim, and at head_dim 128 LDS and
// registers both bound the waves per compute unit.  The gather waits on its rows' loads, so
// waves are worth their LDS: one-wave workgroups of 20 KB (the rows and A^T only) let eight
// waves share a compute unit, against six for two-wave workgroups that also kept the run
// table and the batch's tokens in LDS (20.4 KB per wave): 102 -> 81 ms at 64x68x120 with a
// 3x5x5 kernel, 210 -> 152 ms with 3x7x7.  At head_dim 64 (12 KB) registers bound it at
// three waves per SIMD first.
template <int D>
constexpr int gather_waves() { return D <= 64 ? 4 : 1; }

template <int D, bool PW>
struct GatherLds {
  uint16_t q[PW ? 8 : kGB * D];  // the batch's rows, 16-byte chunks permuted per row
  uint16_t g[kGB * D];
  uint16_t a[PW ? 2 : 4][kGB * 16];  // A^T: (dV hi, dV lo[, dK hi, dK lo]), 32 rows of 16 bf16
};
// The rows and A^T only (the run table stays in the registers of the lanes that read it, the
// tokens are broadcast with ds_bpermute): 20 KB per wave at head_dim 128, so that eight waves
// fit in a compute unit's 160 KB.

// The 16-byte chunks of row e are permuted by XOR with 2 s(e), so that each half-wave of a
// transposing read (for groups G = 0, 1 or 2, 3: rows 8 G + {0..3}, or 8 G + {4..7}, 32 bytes
// each) covers 256 distinct bytes of banks; the row-wise 16-byte writes stay conflict-free since
// a row keeps its bytes.
template <int D>
__device__ inline int gather_row_at(int e, int chunk) {
  int s;
  if constexpr (D == 32) s = (e >> 3) & 1;
  else if constexpr (D == 64) s = ((e >> 1) & 1) | (((e >> 3) & 1) << 1);
  else s = (e & 3) | (((e >> 3) & 1) << 2);
  return e * 2 * D + ((chunk ^ (2 * s)) << 4);
}
// A^T row e (32 bytes); rows 8..15 and 24..31 move to the other 128-byte half of the banks,
// and keep voxels 8..15 in their first 16 bytes and voxels 0..7 in the second, so that the
// 16-byte writes of 16 consecutive rows (first half, then second) fall on distinct banks.
__device__ inline int gather_at_at(int e) { return (e * 32) ^ (((e >> 3) & 1) << 7); }
__device__ inline int gather_at_half(int e) { return ((e >> 3) & 1) << 4; }

__device__ inline bf16x8_t tr_pair(const char* lo, const char* hi) {
  const s16x4_t a = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4_t*)lo);
  const s16x4_t b = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4_t*)hi);
  const uint2 ua = __builtin_bit_cast(uint2, a), ub = __builtin_bit_cast(uint2, b);
  return __builtin_bit_cast(bf16x8_t, make_uint4(ua.x, ua.y, ub.x, ub.y));
}

// Operand with entries 8 G .. 8 G + 7 (G = lane / 16) as its K and column lane % 16: lane j of
// a group reads 4 values of row 8 G + j / 4 (then + 4) at column 4 (j % 4), and the transposing
// read hands lane i column i of those four rows.
template <int D>
__device__ inline bf16x8_t gather_b_frag(const uint16_t* rows, int db) {
  const int lane = threadIdx.x & 63, grp = lane >> 4, j = lane & 15;
  const int e = 8 * grp + (j >> 2), chunk = 2 * db + ((j & 3) >> 1), in = (j & 1) * 8;
  const char* base = reinterpret_cast<const char*>(rows);
  return tr_pair(base + gather_row_at<D>(e, chunk) + in, base + gather_row_at<D>(e + 4, chunk) + in);
}
__device__ inline bf16x8_t gather_a_frag(const uint16_t* at) {
  const int lane = threadIdx.x & 63, grp = lane >> 4, j = lane & 15;
  const int e = 8 * grp + (j >> 2), in = ((j & 3) * 8) ^ gather_at_half(e);
  const char* base = reinterpret_cast<const char*>(at);
  return tr_pair(base + gather_at_at(e) + in, base + gather_at_at(e + 4) + in);
}

// Weights of voxel coordinates 0 and 1 of the block along y or z for a cell at offset rc
// (-1, 0, 1) from the block: the cell's lower corner takes 1 - f, its upper corner f.
__device__ inline void axis_weights(float f, int rc, float& w0, float& w1) {
  const float lo = 1.0f - f;
  w0 = rc < 0 ? f : (rc == 0 ? lo : 0.0f);
  w1 = rc < 0 ? 0.0f : (rc == 0 ? f : lo);
}

// Rows of A_hi^T and A_lo^T for one entry: c times the weights of the block's 16 voxels.
__device__ inline void weight_rows(float c, float fx, float fy, float fz, int rcx, int rcy,
                                   int rcz, uint32_t (&hi)[8], uint32_t (&lo)[8]) {
  float x[4], y[2], z[2];
  const float fl = 1.0f - fx;
#pragma unroll
  for (int vx = 0; vx < 4; ++vx) x[vx] = vx == rcx ? fl : (vx == rcx + 1 ? fx : 0.0f);
  axis_weights(fy, rcy, y[0], y[1]);
  axis_weights(fz, rcz, z[0], z[1]);
  float w[16];
#pragma unroll
  for (int v = 0; v < 16; ++v) w[v] = x[v & 3] * (y[(v >> 2) & 1] * (c * z[v >> 3]));
#pragma unroll
  for (int p = 0; p < 8; ++p) {
    const uint32_t u0 = __float_as_uint(w[2 * p]), u1 = __float_as_uint(w[2 * p + 1]);
    hi[p] = __builtin_amdgcn_perm(u1, u0, 0x07060302u);  // upper halves of w0 (low), w1 (high)
    const float l0 = w[2 * p] - __uint_as_float(u0 & 0xffff0000u);
    const float l1 = w[2 * p + 1] - __uint_as_float(u1 & 0xffff0000u);
    lo[p] = __builtin_bit_cast(uint32_t, bf16x2_t{(__bf16)l0, (__bf16)l1});
  }
}

// A batch position: entries [u, min(u + 32, end)) of run r, whose cells x0 .. x0 + 3 start at
// m1 .. m4 (cell x0 - 1 starts at or before u); u >= end once the runs are exhausted.
struct GatherPos {
  uint32_t u, end, m1, m2, m3, m4;
  int rc;         // the run's cell row / plane: (y - y0 + 1) + 3 (z - z0 + 1)
  uint64_t left;  // lanes holding the runs after this one
};

// This lane's 16 bytes of an entry: lanes 0-31 read (n, alpha, sds, fx), lanes 32-63 read
// (sds, fx, fy, fz) of the same entry; the halves then swap what the other one holds.
struct GatherEntry {
  uint4 raw;
  uint32_t idx;
};

template <int D, bool PW>
__global__ __launch_bounds__(64 * gather_waves<D>()) __attribute__((amdgpu_waves_per_eu(D <= 64 ? 3 : 2)))
void bwd_gather_mfma_kernel(Geometry g, const void* __restrict__ q, const void* __restrict__ dout,
                            const uint32_t* __restrict__ starts, const Entry* __restrict__ entries,
                            float* __restrict__ dk, float* __restrict__ dv, PencilOrder po) {
  constexpr int NW = gather_waves<D>();
  constexpr int DB = D / 16;     // 16-channel blocks: two products each (hi, lo) per tensor
  constexpr int LPR = D / 8;     // lanes per row when copying rows (16 bytes each)
  constexpr int RPI = 64 / LPR;  // rows per copy instruction
  constexpr int NI = kGB / RPI;  // copy instructions per tensor and batch
  __shared__ GatherLds<D, PW> lds[NW];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  GatherLds<D, PW>& L = lds[wave];
  const uint32_t tok_bytes = (uint32_t)g.heads * 2 * D;
  const bool upper = lane >= 32;  // dV coefficients (else dK)
  const int own = lane & 31;      // the entry whose coefficients this lane forms

  for (int64_t vt = blockIdx.x; vt < po.vtiles; vt += gridDim.x) {
    PencilTile tl;
    if (!pencil_tile(po, vt, tl)) continue;
    int by, bx;  // the wave's 4 x 2 x 2 block: cell (by, bx) of the pencil grid, frame pair tl.frame
    if (!pencil_cell(po, tl, wave, by, bx)) continue;
    const int bh = tl.group;
    const int b = bh / g.heads, m = bh % g.heads;
    const int x0 = 4 * bx, y0 = 2 * by, z0 = 2 * tl.frame;
    const int nx = min(5, g.W - x0 + 1);  // cells x0 - 1 .. x0 + nx - 2 exist
    const bool hasy1 = y0 + 1 < g.H, hasz1 = z0 + 1 < g.T;
    const int64_t head_off = ((int64_t)b * g.N * g.heads + m) * (2 * D) + (lane % LPR) * 16;
    const char* qh = static_cast<const char*>(q) + head_off;
    const char* gh = static_cast<const char*>(dout) + head_off;

    // the non-empty runs, in order: lane r < 9 looks at cell row y0 - 1 + r % 3, plane z0 - 1 + r / 3
    bool has = false;
    uint32_t c[6] = {0u, 0u, 0u, 0u, 0u, 0u};
    if (lane < 9) {
      const int yr = lane % 3, zr = lane / 3;
      if ((yr < 2 || hasy1) && (zr < 2 || hasz1)) {
        const int64_t ci = cell_index(g, bh, x0 - 1, y0 - 1 + yr, z0 - 1 + zr);
#pragma unroll
        for (int i = 0; i < 6; ++i) c[i] = starts[ci + min(i, nx)];
        has = c[0] < c[5];
      }
    }
    // lane r < 9 keeps its run's bounds in c[]; the wave reads the runs in lane order with
    // readlane, `left` marking the lanes whose runs are still ahead
    const uint64_t hm = __builtin_amdgcn_ballot_w64(has);
    auto next_run = [&](GatherPos& d) {
      if (d.left != 0ull) {
        const int lr = __builtin_amdgcn_readfirstlane(__builtin_ctzll(d.left));
        d.left &= d.left - 1ull;
        d.u = __builtin_amdgcn_readlane(c[0], lr);
        d.m1 = __builtin_amdgcn_readlane(c[1], lr);
        d.m2 = __builtin_amdgcn_readlane(c[2], lr);
        d.m3 = __builtin_amdgcn_readlane(c[3], lr);
        d.m4 = __builtin_amdgcn_readlane(c[4], lr);
        d.end = __builtin_amdgcn_readlane(c[5], lr);
        d.rc = lr;
      } else {
        d.u = d.end = d.m1 = d.m2 = d.m3 = d.m4 = 0u;
        d.rc = 0;
      }
    };
    auto advance = [&](GatherPos& d) {
      d.u += kGB;
      if (d.u >= d.end) next_run(d);
    };
    // this lane's part of its entry (clamped to the run; the coefficient is zeroed outside it)
    auto fetch = [&](const GatherPos& d, GatherEntry& en) {
      en.idx = d.u + own;
      const char* p = reinterpret_cast<const char*>(entries + min(en.idx, d.end - 1u));
      en.raw = *reinterpret_cast<const uint4*>(p + (upper ? 8 : 0));
    };
    auto weights = [&](const GatherPos& d, const GatherEntry& en) {
      // the other half's words: lanes 0-31 get (fy, fz), lanes 32-63 get alpha
      const auto sz = __builtin_amdgcn_permlane32_swap(en.raw.z, en.raw.z, false, false);
      const auto sw = __builtin_amdgcn_permlane32_swap(en.raw.w, en.raw.w, false, false);
      const auto sy = __builtin_amdgcn_permlane32_swap(en.raw.y, en.raw.y, false, false);
      const float coef = __uint_as_float(upper ? sy[0] : en.raw.z);
      const float fx = __uint_as_float(upper ? en.raw.y : en.raw.w);
      const float fy = __uint_as_float(upper ? en.raw.z : sz[1]);
      const float fz = __uint_as_float(upper ? en.raw.w : sw[1]);
      const uint32_t i = en.idx;
      const int rcx = -1 + (i >= d.m1 ? 1 : 0) + (i >= d.m2 ? 1 : 0) + (i >= d.m3 ? 1 : 0) +
                      (i >= d.m4 ? 1 : 0);
      if (PW && !upper) return;
      uint32_t hi[8], lo[8];
      weight_rows(i < d.end ? coef : 0.0f, fx, fy, fz, rcx, d.rc % 3 - 1, d.rc / 3 - 1, hi, lo);
      const int sel = upper ? 0 : 2;
      const int h0 = gather_at_half(own), h1 = 16 - h0;  // bytes of voxels 0..7 and 8..15
      char* ah = reinterpret_cast<char*>(L.a[sel]) + gather_at_at(own);
      char* al = reinterpret_cast<char*>(L.a[sel + 1]) + gather_at_at(own);
      *reinterpret_cast<uint4*>(ah + h0) = make_uint4(hi[0], hi[1], hi[2], hi[3]);
      *reinterpret_cast<uint4*>(ah + h1) = make_uint4(hi[4], hi[5], hi[6], hi[7]);
      *reinterpret_cast<uint4*>(al + h0) = make_uint4(lo[0], lo[1], lo[2], lo[3]);
      *reinterpret_cast<uint4*>(al + h1) = make_uint4(lo[4], lo[5], lo[6], lo[7]);
    };
    uint4 rq[NI], rg[NI];
    bool part = false;  // the batch ends inside: its rows past the end are zeroed in LDS
    auto issue_rows = [&](const GatherPos& d, const GatherEntry& en) {
      part = d.end - d.u < (uint32_t)kGB;
#pragma unroll
      for (int t = 0; t < NI; ++t) {
        const int e = lane / LPR + RPI * t;
        // entry e's token, from lane e (lanes 0-31 hold n), for the LPR lanes of its row
        const uint32_t n = (uint32_t)__builtin_amdgcn_ds_bpermute(e << 2, (int)en.raw.x);
        const uint64_t o = (uint64_t)n * tok_bytes;
        if (d.u + e < d.end) {  // rows past the run's end are not loaded
          if constexpr (!PW) rq[t] = *reinterpret_cast<const uint4*>(qh + o);
          rg[t] = *reinterpret_cast<const uint4*>(gh + o);
        }
      }
    };
    auto store_rows = [&](const GatherPos& d) {
      if (part) {
#pragma unroll
        for (int t = 0; t < NI; ++t) {
          if (d.u + lane / LPR + RPI * t >= d.end) {
            rq[t] = make_uint4(0, 0, 0, 0);
            rg[t] = make_uint4(0, 0, 0, 0);
          }
        }
      }
#pragma unroll
      for (int t = 0; t < NI; ++t) {
        const int at = gather_row_at<D>(lane / LPR + RPI * t, lane % LPR);
        if constexpr (!PW) *reinterpret_cast<uint4*>(reinterpret_cast<char*>(L.q) + at) = rq[t];
        *reinterpret_cast<uint4*>(reinterpret_cast<char*>(L.g) + at) = rg[t];
      }
    };

    f32x4_t ck[DB], cv[DB];
#pragma unroll
    for (int db = 0; db < DB; ++db) ck[db] = cv[db] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};

    // Per batch i: store its rows, fetch the entries of batch i + 2, load the rows of batch
    // i + 1, take batch i's products, then form batch i + 1's weights (p0, p1, p2: batches i,
    // i + 1, i + 2).
    GatherPos p0, p1, p2;
    p0.left = hm;
    next_run(p0);
    if (p0.u < p0.end) {
      GatherEntry e1, e2;
      {
        GatherEntry e0;
        fetch(p0, e0);
        weights(p0, e0);
        issue_rows(p0, e0);
      }
      p1 = p0;
      advance(p1);
      if (p1.u < p1.end) fetch(p1, e1);
      p2 = p1;
      advance(p2);
      while (p0.u < p0.end) {
        store_rows(p0);
        if (p2.u < p2.end) fetch(p2, e2);
        if (p1.u < p1.end) issue_rows(p1, e1);
        const bf16x8_t avh = gather_a_frag(L.a[0]), avl = gather_a_frag(L.a[1]);
        bf16x8_t akh, akl;
        if constexpr (!PW) {
          akh = gather_a_frag(L.a[2]);
          akl = gather_a_frag(L.a[3]);
        }
#pragma unroll
        for (int db = 0; db < DB; ++db) {
          if constexpr (!PW) {
            const bf16x8_t bq = gather_b_frag<D>(L.q, db);
            ck[db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(akh, bq, ck[db], 0, 0, 0);
            ck[db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(akl, bq, ck[db], 0, 0, 0);
          }
          const bf16x8_t bg = gather_b_frag<D>(L.g, db);
          cv[db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(avh, bg, cv[db], 0, 0, 0);
          cv[db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(avl, bg, cv[db], 0, 0, 0);
        }
        if (p1.u < p1.end) weights(p1, e1);
        e1 = e2;
        p0 = p1;
        p1 = p2;
        advance(p2);
      }
    }

    // result rows 4 G + vx (G = lane / 16 = vy + 2 vz), column lane % 16 of each channel block
    const int grp = lane >> 4, col = lane & 15;
    const int vy = grp & 1, vz = grp >> 1;
    if ((vy == 0 || hasy1) && (vz == 0 || hasz1)) {
      const int64_t row0 =
          ((int64_t)b * g.N + (int64_t)((z0 + vz) * g.H + y0 + vy) * g.W + x0) * g.heads + m;
#pragma unroll
      for (int vx = 0; vx < 4; ++vx) {
        if (vx > 0 && x0 + vx >= g.W) break;
        const int64_t row = row0 + (int64_t)vx * g.heads;
#pragma unroll
        for (int db = 0; db < DB; ++db) {
          if constexpr (!PW) dk[row * D + db * 16 + col] = ck[db][vx];
          dv[row * D + db * 16 + col] = cv[db][vx];
        }
      }
    }
  }
}

// ---------------------------------------------------------------------------- launch

struct Workspace {
  uint32_t* counts;   // [cells]
  uint32_t* starts;   // [cells + 1]
  uint32_t* cursor;   // [cells]
  uint32_t* sums;     // [ceil(cells / kScanBlockItems)]
  RecK* reck;         // [rows * P]
  RecV* recv;         // [rows * P]
  float* delta;       // [rows]
  Entry* entries;     // [rows * P]
  uint32_t* ranks;    // [rows * P]: a point's rank in its bin (the split sweep's slots)
  size_t bytes;
};

inline size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

Workspace carve(const Geometry& g, void* base) {
  const int64_t rows = (int64_t)g.B * g.N * g.heads;
  const int64_t cells = cells_per_bh(g) * g.B * g.heads;
  const int64_t nsums = (cells + kScanBlockItems - 1) / kScanBlockItems;
  const int64_t points = rows * g.P;
  Workspace w{};
  size_t off = 0;
  char* p = static_cast<char*>(base);
  auto take = [&](size_t bytes) {
    char* r = p ? p + off : nullptr;
    off += align256(bytes);
    return r;
  };
  w.counts = reinterpret_cast<uint32_t*>(take(cells * 4));
  w.starts = reinterpret_cast<uint32_t*>(take((cells + 1) * 4));
  w.cursor = reinterpret_cast<uint32_t*>(take(cells * 4));
  w.sums = reinterpret_cast<uint32_t*>(take(nsums * 4));
  w.reck = reinterpret_cast<RecK*>(take(points * sizeof(RecK)));
  w.recv = reinterpret_cast<RecV*>(take(points * sizeof(RecV)));
  w.delta = reinterpret_cast<float*>(take(rows * 4));
  w.entries = reinterpret_cast<Entry*>(take(points * sizeof(Entry)));
  w.ranks = reinterpret_cast<uint32_t*>(take(points * 4));
  w.bytes = off;
  return w;
}

int grid_for(int64_t items, int per_block = kBlockThreads, int cap = 1 << 20) {
  const int64_t b = (items + per_block - 1) / per_block;
  return (int)(b < 1 ? 1 : (b < cap ? b : cap));
}

template <int D, bool BF16>
// logits != null: the predicted-weights variant (q, k, dq and dk unused; dlogits written).
hipError_t bwd_dispatch(const Geometry& g, const void* q, const void* k, const void* v,
                        const float* logits, const float* off, const float* lse, const void* dout,
                        float* dq, float* dk, float* dv, float* doff, float* dlogits,
                        void* workspace, hipStream_t s, hipEvent_t const* ev) {
  const bool pw = logits != nullptr;
  // phase marks for the caller's timing events (none when ev is null)
  auto mark = [&](int i) { return ev == nullptr ? hipSuccess : hipEventRecord(ev[i], s); };
  Workspace w = carve(g, workspace);
  const int64_t rows = (int64_t)g.B * g.N * g.heads;
  const int64_t cells = cells_per_bh(g) * g.B * g.heads;
  const int64_t nsums = (cells + kScanBlockItems - 1) / kScanBlockItems;
  const int64_t points = rows * g.P;
  hipError_t e;
  {
    uint32_t zero = 0;
    void* a[] = {(void*)&w.counts, (void*)&cells, (void*)&zero};
    e = hipLaunchKernel(reinterpret_cast<const void*>(&fill_u32_kernel), dim3(grid_for(cells)),
                        dim3(kBlockThreads), a, 0, s);
    if (e != hipSuccess) return e;
  }
  const PencilOrder po = query_order<D, BF16>(g);
  const int blocks = grid_blocks(po.vtiles);
  // The main operator sweeps the points twice (V pass, then K pass with the finish of each
  // row's points); the predicted-weights variant, which reads no K, sweeps them once and
  // finishes them in the finalize pass.
  const bool split = !pw;
  if ((e = mark(0)) != hipSuccess) return e;
  if (split) {
    void* a[] = {(void*)&g, (void*)&v, (void*)&off, (void*)&dout, (void*)&w.recv,
                 (void*)&w.counts, (void*)&w.ranks, (void*)&po};
    e = hipLaunchKernel(reinterpret_cast<const void*>(&bwd_vpass_kernel<D, BF16>), dim3(blocks),
                        dim3(kBlockThreads), a, 0, s);
    if (e != hipSuccess) return e;
  } else {
    void* a[] = {(void*)&g,      (void*)&v,      (void*)&logits,  (void*)&off,
                 (void*)&lse,    (void*)&dout,   (void*)&w.reck,  (void*)&w.recv,
                 (void*)&w.delta, (void*)&w.counts, (void*)&po};
    e = hipLaunchKernel(reinterpret_cast<const void*>(&bwd_sweep_kernel<D, BF16>), dim3(blocks),
                        dim3(kBlockThreads), a, 0, s);
    if (e != hipSuccess) return e;
  }
  if ((e = mark(1)) != hipSuccess) return e;
  {
    void* a[] = {(void*)&w.counts, (void*)&w.sums, (void*)&cells};
    e = hipLaunchKernel(reinterpret_cast<const void*>(&scan_reduce_kernel), dim3((unsigned)nsums),
                        dim3(kScanThreads), a, 0, s);
    if (e != hipSuccess) return e;
    uint32_t* grand = w.starts + cells;
    void* b2[] = {(void*)&w.sums, (void*)&nsums, (void*)&grand};
    e = hipLaunchKernel(reinterpret_cast<const void*>(&scan_sums_kernel), dim3(1),
                        dim3(kScanThreads), b2, 0, s);
    if (e != hipSuccess) return e;
    void* c3[] = {(void*)&w.counts, (void*)&w.sums, (void*)&w.starts, (void*)&w.cursor,
                  (void*)&cells};
    e = hipLaunchKernel(reinterpret_cast<const void*>(&scan_apply_kernel), dim3((unsigned)nsums),
                        dim3(kScanThreads), c3, 0, s);
    if (e != hipSuccess) return e;
  }
  if ((e = mark(2)) != hipSuccess) return e;
  if (split) {
    void* a[] = {(void*)&g,    (void*)&q,       (void*)&k,       (void*)&off,
                 (void*)&lse,  (void*)&dq,      (void*)&w.reck,  (void*)&w.recv, (void*)&w.starts,
                 (void*)&w.ranks, (void*)&doff, (void*)&w.entries, (void*)&po};
    constexpr int L = Layout<D, BF16>::kLanes;
    const void* kern = (g.P + L - 1) / L <= kHoldChunks
                           ? reinterpret_cast<const void*>(&bwd_kpass_kernel<D, BF16, kHoldChunks>)
                           : reinterpret_cast<const void*>(&bwd_kpass_kernel<D, BF16, 0>);
    e = hipLaunchKernel(kern, dim3(blocks), dim3(kBlockThreads), a, 0, s);
    if (e != hipSuccess) return e;
  } else {
    const int npoints = (int)points;
    void* a[] = {(void*)&g,      (void*)&off,     (void*)&w.reck,  (void*)&w.recv,  (void*)&w.delta,
                 (void*)&w.cursor, (void*)&doff, (void*)&dlogits, (void*)&w.entries,
                 (void*)&npoints};
    e = hipLaunchKernel(reinterpret_cast<const void*>(&bwd_finalize_kernel), dim3(grid_for(points)),
                        dim3(kBlockThreads), a, 0, s);
    if (e != hipSuccess) return e;
  }
  if ((e = mark(3)) != hipSuccess) return e;
  if constexpr (BF16) {
    constexpr int NW = gather_waves<D>();
    // cells: 4 x 2 voxel blocks of a frame pair; pencils of about 16 x 16 voxels at head_dim
    // 128 and 32 x 32 below.  Measured (with two-wave workgroups at head_dim 128) at
    // 64x68x120 (head_dim 128) / 64x34x60 (64): 108.8 / 3.68 ms for 16 x 16, 108.3 / 3.42
    // for 32 x 32, 110.6 / 3.76 for 8 x 8, 132.5 / 3.25 for whole frames; at 64x68x120
    // 32 x 32 pencils hit L2 on 31% of its requests against 58%, the same time only
    // because the gather then reads past L2 at the ceiling of such misses.
    const PencilOrder go = plan_pencils(g.B * g.heads, (g.T + 1) / 2, (g.H + 1) / 2,
                                        (g.W + 3) / 4, NW, D >= 128 ? 8 : 16, D >= 128 ? 4 : 8);
    const int gblocks = grid_blocks(go.vtiles);
    void* a[] = {(void*)&g,         (void*)&q,  (void*)&dout, (void*)&w.starts,
                 (void*)&w.entries, (void*)&dk, (void*)&dv,   (void*)&go};
    const void* kern = pw ? reinterpret_cast<const void*>(&bwd_gather_mfma_kernel<D, true>)
                          : reinterpret_cast<const void*>(&bwd_gather_mfma_kernel<D, false>);
    e = hipLaunchKernel(kern, dim3(gblocks), dim3(64 * NW), a, 0, s);
    if (e != hipSuccess) return e;
  } else {
    using LY = Layout<D, BF16>;
    // cells: 2 x 2 voxel blocks of a frame; pencils of about 32 x 32 voxels
    const PencilOrder go = plan_pencils(g.B * g.heads, g.T, (g.H + 1) / 2, (g.W + 1) / 2,
                                        LY::kRowsPerBlock, 16, 16);
    const int gblocks = grid_blocks(go.vtiles);
    void* a[] = {(void*)&g,         (void*)&q,  (void*)&dout, (void*)&w.starts,
                 (void*)&w.entries, (void*)&dk, (void*)&dv,   (void*)&go};
    const void* kern = pw ? reinterpret_cast<const void*>(&bwd_gather_kernel<D, BF16, true>)
                          : reinterpret_cast<const void*>(&bwd_gather_kernel<D, BF16, false>);
    e = hipLaunchKernel(kern, dim3(gblocks), dim3(kBlockThreads), a, 0, s);
    if (e != hipSuccess) return e;
  }
  return mark(4);
}

}  // namespace

size_t backward_workspace_bytes(const Geometry& g) { return carve(g, nullptr).bytes; }

hipError_t launch_backward(const Geometry& g, bool bf16, const void* q, const void* k,
                           const void* v, const float* logits, const float* offsets,
                           const float* lse, const void* dout, float* dq, float* dk, float* dv,
                           float* d_offsets, float* dlogits, void* workspace, hipStream_t stream,
                           hipEvent_t const* events) {
#define DSA3D_BWD(DIM, BF)                                                                      \
  bwd_dispatch<DIM, BF>(g, q, k, v, logits, offsets, lse, dout, dq, dk, dv, d_offsets, dlogits, \
                        workspace, stream, events)
  switch (g.D) {
    case 32:
      return bf16 ? DSA3D_BWD(32, true) : DSA3D_BWD(32, false);
    case 64:
      return bf16 ? DSA3D_BWD(64, true) : DSA3D_BWD(64, false);
    case 128:
      return bf16 ? DSA3D_BWD(128, true) : DSA3D_BWD(128, false);
    default:
      return hipErrorInvalidValue;
  }
#undef DSA3D_BWD
}

}  // namespace dsa3d
