// Fixed / shifted 3D window attention (the Swin-DiT baseline of Section 6.2), gfx950 kernels.
//
// The shifted-window partition is handled as a partition of the grid into boxes: along each
// axis the cut points are off + n * window, clipped to the grid, and every box attends densely
// within itself (the keys a rolled window's mask keeps for a query are exactly the real tokens
// of the query's box).  A workgroup takes one (batch, box, head) group and one tile of 128 of
// its queries; the tiles of a group are given blocks of one XCD, so its K and V rows are
// served from that XCD's L2 after the first read.
//
// Matrix products use v_mfma_f32_32x32x16_bf16.  For A (32 x 16), B (16 x 32) and C (32 x 32)
// lane l holds row (of A) or column (of B) l % 32 with k = 8 (l / 32) .. +7, and C column
// l % 32 with rows 8 (i / 4) + 4 (l / 32) + i % 4 in its element i.  The kernels compute the
// transposed products (S^T = K Q^T, O^T = V^T P^T and so on) so that a lane owns one query's
// (or key's) column: the softmax statistics then need only one exchange with lane l ^ 32, and
// the logits in C layout are already the B operand of the next product once the keys are
// taken in the order lane l's 8 registers hold them (the A operand, read from a transposed LDS
// tile, uses the same order).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>
#include <cmath>

#include "dsa3d_internal.h"

namespace dsa3d {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr int kThreads = 256;
constexpr int kQTile = 128;  // queries per workgroup: 4 waves x 32
constexpr int kTile = 64;    // rows per LDS tile of the dq (keys) and dk/dv (queries) passes
constexpr int kFwdTile = 64;   // keys per LDS tile of the forward
constexpr int kXcd = 8;
constexpr float kLn2 = 0.6931471805599453f;
constexpr float kSlack = 8.0f;  // base-2 headroom of the forward's running maximum

struct Box {
  int t0, i0, j0, lh, lw, n;
  float inv_hw, inv_w;
};

__device__ inline void axis_cut(int a, int off, int win, int size, int& lo, int& len) {
  const int s = off + a * win, e = s + win;
  lo = s > 0 ? s : 0;
  len = (e < size ? e : size) - lo;
}

__device__ inline Box box_of(const WinGeometry& g, int box) {
  const int aw = box % g.nw, r = box / g.nw, ah = r % g.nh, at = r / g.nh;
  Box bx;
  int lt;
  axis_cut(at, g.off_t, g.wt, g.T, bx.t0, lt);
  axis_cut(ah, g.off_h, g.wh, g.H, bx.i0, bx.lh);
  axis_cut(aw, g.off_w, g.ww, g.W, bx.j0, bx.lw);
  bx.n = lt * bx.lh * bx.lw;
  bx.inv_hw = 1.0f / (float)(bx.lh * bx.lw);
  bx.inv_w = 1.0f / (float)bx.lw;
  return bx;
}

// Token (t * H + i) * W + j of box-local index u, box-major (t, then i, then j).  u is below
// 2^16, so the float quotients (u + 1/2) / d, whose distance to an integer is at least 1/(2d),
// are floored exactly.
__device__ inline int box_token(const WinGeometry& g, const Box& bx, int u) {
  const int a = (int)(((float)u + 0.5f) * bx.inv_hw);
  const int rem = u - a * bx.lh * bx.lw;
  const int e = (int)(((float)rem + 0.5f) * bx.inv_w);
  return ((bx.t0 + a) * g.H + bx.i0 + e) * g.W + bx.j0 + (rem - e * bx.lw);
}

struct Group {
  int b, m, qt;
  Box bx;
};

// Block -> (batch, box, head) group and query tile.  Dispatch hands block x to XCD x % 8, so
// the tiles of a group are given blocks congruent modulo 8.  Returns false for padding blocks.
__device__ inline bool group_of(const WinGeometry& g, int tiles, Group& gr) {
  const int x = blockIdx.x % kXcd, r = blockIdx.x / kXcd;
  gr.qt = r % tiles;
  const int grp = (r / tiles) * kXcd + x;
  if (grp >= g.groups) return false;
  gr.m = grp % g.heads;
  const int r2 = grp / g.heads;
  gr.b = r2 / g.boxes;
  gr.bx = box_of(g, r2 % g.boxes);
  return true;
}

__device__ inline int64_t row_of(const WinGeometry& g, int b, int tok, int m) {
  return ((int64_t)b * g.N + tok) * g.heads + m;
}

// x combined with the value of lane l ^ 32 by v_permlane32_swap, which moves data between the
// two halves of the wave without going through LDS (so it does not wait for outstanding LDS
// reads).  Applied to (x, x) it returns, in each lane, the lane's own value and its partner's
// (in either order), so max and sum come out identical in both lanes of a pair.
__device__ inline float pair_max(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                  false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ inline float pair_sum(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                  false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

__device__ inline f32x16_t mfma(const bf16x8_t& a, const bf16x8_t& b, const f32x16_t& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ inline bf16x8_t as_bf16x8(const uint4& u) { return __builtin_bit_cast(bf16x8_t, u); }

// Tensor rows of tile rows base .. base + ROWS - 1 of the group's box, computed by the first
// ROWS threads for the whole workgroup.  Tile rows past the box end get the box's last row (a
// valid address: the loads need no branch; the staging zeroes what they read).
template <int ROWS>
__device__ inline void fill_rows(int* tab, const WinGeometry& g, const Group& gr, int base) {
  if (threadIdx.x < ROWS) {
    const int u = min(base + (int)threadIdx.x, gr.bx.n - 1);
    tab[threadIdx.x] = (int)row_of(g, gr.b, box_token(g, gr.bx, u), gr.m);
  }
}

// A tile of ROWS box rows (box-local indices base .. base + ROWS - 1; rows past the box end
// read as zero) of a [rows][D] bf16 tensor in LDS, gathered through the box's token order.
// Rows are D channels long, unpadded, and the 16-byte chunks of a row are XOR-permuted by a
// function of the row so that both operand reads cover the 256 bytes the LDS serves per
// cycle without a repeated bank: the 16-byte reads of one chunk of 16 consecutive rows (the
// row-major operand) and the transposing 8-byte reads of 4 consecutive rows x 64 bytes (the
// column operand).  D = 128 (16 chunks, one row per 256 bytes): f = 4 (row % 4) + (row / 4) % 4;
// D = 64 (8 chunks, the row's parity picks the 128-byte half):
// f = 4 ((row / 2) % 2) + (row / 4) % 4.  Each thread stages NL 16-byte chunks.
template <int D, int ROWS>
struct Tile {
  static constexpr int KCH = D / 8;                 // 16-byte chunks per row
  static constexpr int NL = ROWS * KCH / kThreads;  // chunks per thread
  static constexpr int kElems = ROWS * D;
  static_assert(NL == 2 || NL == 4 || NL == 8, "unsupported tile");

  // element offset of (row, channel), channel a multiple of 4
  static __device__ inline int at(int row, int chan) {
    static_assert(D == 64 || D == 128, "head_dim 64 or 128");
    const int f = D == 128 ? 4 * (row & 3) + ((row >> 2) & 3)
                           : 4 * ((row >> 1) & 1) + ((row >> 2) & 3);
    return row * D + (((chan >> 3) ^ f) << 3) + (chan & 7);
  }

  // Thread t moves chunk t % KCH of tile rows t / KCH + i * (kThreads / KCH).  tab[r] is the
  // tensor row of tile row r; `valid` tile rows (those inside the box) are kept, the others
  // zeroed.  The loads are issued together, without branches.
  static __device__ inline void load(uint4 (&r)[NL], const uint16_t* src, const int* tab,
                                     int valid) {
    const int t = threadIdx.x;
    int row[NL];
#pragma unroll
    for (int i = 0; i < NL; ++i) row[i] = tab[t / KCH + i * (kThreads / KCH)];
#pragma unroll
    for (int i = 0; i < NL; ++i)
      r[i] = *reinterpret_cast<const uint4*>(src + (int64_t)row[i] * D + (t % KCH) * 8);
    if (valid < ROWS) {
#pragma unroll
      for (int i = 0; i < NL; ++i)
        if (t / KCH + i * (kThreads / KCH) >= valid) r[i] = make_uint4(0, 0, 0, 0);
    }
  }
  static __device__ inline void store(uint16_t* lds, const uint4 (&r)[NL]) {
    const int t = threadIdx.x;
#pragma unroll
    for (int i = 0; i < NL; ++i)
      *reinterpret_cast<uint4*>(lds + at(t / KCH + i * (kThreads / KCH), (t % KCH) * 8)) = r[i];
  }

  // A operand with tile rows as its rows: row r0 + l % 32, channels 16 ks + 8 (l / 32) .. +7.
  static __device__ inline bf16x8_t a_rows(const uint16_t* lds, int r0, int ks) {
    const int lane = threadIdx.x & 63;
    return as_bf16x8(
        *reinterpret_cast<const uint4*>(lds + at(r0 + (lane & 31), ks * 16 + (lane >> 5) * 8)));
  }
  // A operand with channels as its rows: channel d0 + l % 32; tile rows 32 kb + 16 p + 4 (l / 32)
  // + {0..3, 8..11}, the order in which a C-layout block's elements 8 p .. 8 p + 7 hold them.
  // ds_read_b64_tr_b16 transposes within each 16-lane group: lane i receives element i % 4 of
  // the 4-element reads of lanes i / 4 + {0, 4, 8, 12}; so lane j reads 4 channels starting at
  // c0 + 4 (j % 4) of row base + j / 4, and lane i gets channel c0 + i of rows base .. base + 3.
  static __device__ inline bf16x8_t a_cols(const uint16_t* lds, int d0, int kb, int p) {
    typedef short s4_t __attribute__((ext_vector_type(4)));
    typedef __attribute__((address_space(3))) s4_t lds_s4_t;
    const int lane = threadIdx.x & 63, j = lane & 15;
    const int row = kb * 32 + 16 * p + 4 * (lane >> 5) + (j >> 2);
    const int chan = d0 + 16 * ((lane >> 4) & 1) + 4 * (j & 3);
    const s4_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s4_t*)(lds + at(row, chan)));
    const s4_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s4_t*)(lds + at(row + 8, chan)));
    const uint2 ul = __builtin_bit_cast(uint2, lo), uh = __builtin_bit_cast(uint2, hi);
    return as_bf16x8(make_uint4(ul.x, ul.y, uh.x, uh.y));
  }
};

// Fragment of this lane's row as the B operand: channels 16 ks + 8 (l / 32) .. +7 (zero for a
// row past the box end).
template <int D>
__device__ inline void load_frag(bf16x8_t (&f)[D / 16], const uint16_t* src, int64_t row, bool ok) {
  const int hh = (threadIdx.x & 63) >> 5;
#pragma unroll
  for (int ks = 0; ks < D / 16; ++ks) {
    uint4 u = make_uint4(0, 0, 0, 0);
    if (ok) u = *reinterpret_cast<const uint4*>(src + row * D + ks * 16 + hh * 8);
    f[ks] = as_bf16x8(u);
  }
}

// Sixteen C-layout values as B-operand fragments (elements 8 p .. 8 p + 7) of a bf16 pair
// hi + lo carrying about 16 significant bits, so a product taken as two MFMAs (hi and lo)
// loses almost nothing to the bf16 operand.
__device__ inline void to_frags(const float (&x)[16], bf16x8_t (&hi)[2], bf16x8_t (&lo)[2]) {
  // hi = x truncated to its upper 16 bits (two of them packed by one byte permute); lo = x - hi
  // is exact in fp32 and rounded once to bf16, so hi + lo is x to within 2^-17 |x|.
  uint32_t h[8], l[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const uint32_t u0 = __float_as_uint(x[2 * i]), u1 = __float_as_uint(x[2 * i + 1]);
    h[i] = __builtin_amdgcn_perm(u1, u0, 0x07060302u);
    const float l0 = x[2 * i] - __uint_as_float(u0 & 0xffff0000u);
    const float l1 = x[2 * i + 1] - __uint_as_float(u1 & 0xffff0000u);
    typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
    l[i] = __builtin_bit_cast(uint32_t, bf16x2_t{(__bf16)l0, (__bf16)l1});
  }
  hi[0] = __builtin_bit_cast(bf16x8_t, make_uint4(h[0], h[1], h[2], h[3]));
  hi[1] = __builtin_bit_cast(bf16x8_t, make_uint4(h[4], h[5], h[6], h[7]));
  lo[0] = __builtin_bit_cast(bf16x8_t, make_uint4(l[0], l[1], l[2], l[3]));
  lo[1] = __builtin_bit_cast(bf16x8_t, make_uint4(l[4], l[5], l[6], l[7]));
}

// Stores this lane's 16 fp32 C-layout values of channel block db (channels 32 db + 8 blk +
// 4 (l / 32) + j) times `mul` to a float row.
__device__ inline void store_f32_block(float* row, int db, const f32x16_t& acc, float mul) {
  const int hh = (threadIdx.x & 63) >> 5;
#pragma unroll
  for (int blk = 0; blk < 4; ++blk)
    *reinterpret_cast<float4*>(row + db * 32 + 8 * blk + 4 * hh) =
        make_float4(acc[4 * blk] * mul, acc[4 * blk + 1] * mul, acc[4 * blk + 2] * mul,
                    acc[4 * blk + 3] * mul);
}

// ---------------------------------------------------------------------------- forward

// Online-softmax state of one query (lanes l and l ^ 32 keep identical copies): running
// maximum of the base-2 logits and the partial sum over this lane's half of the keys.
struct Softmax {
  float m = -INFINITY, l = 0.0f;
};

// One workgroup: 128 queries of one (batch, box, head) group against every key of the box,
// kFwdTile keys per LDS tile, online base-2 softmax.  Wave w owns queries 32 w .. 32 w + 31 of the
// tile; lanes l and l ^ 32 share query l % 32 and hold 16 of each 32-key block's logits each.
// Within a tile the logits of block b + 1 are issued to the matrix cores before the softmax of
// block b runs on the vector ALUs, so the two overlap.
template <int D>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2, 2))) void
win_fwd_kernel(WinGeometry g, const uint16_t* __restrict__ q, const uint16_t* __restrict__ k,
               const uint16_t* __restrict__ v, uint16_t* __restrict__ out,
               uint16_t* __restrict__ out_res, float* __restrict__ lse) {
  constexpr int KT = kFwdTile;
  using Tl = Tile<D, KT>;
  constexpr int KS = D / 16;  // MFMA k-steps over head_dim
  constexpr int DB = D / 32;  // 32-channel blocks of the output
  constexpr int NB = KT / 32; // 32-key blocks per tile
  __shared__ __attribute__((aligned(16))) uint16_t Ks[2][Tl::kElems];
  __shared__ __attribute__((aligned(16))) uint16_t Vs[2][Tl::kElems];
  __shared__ int tab[3][KT];  // key rows of tile i in slot i % 3

  Group gr;
  if (!group_of(g, g.qtiles, gr)) return;
  const int q0 = gr.qt * kQTile, n = gr.bx.n;
  if (q0 >= n) return;  // the box has fewer tiles than the largest one
  const int ntiles = (n + KT - 1) / KT;
  for (int i = 0; i < 3 && i < ntiles; ++i) fill_rows<KT>(tab[i], g, gr, i * KT);

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, hh = lane >> 5;
  const int uq = q0 + wave * 32 + (lane & 31);
  const bool qok = uq < n;
  const int64_t qrow = qok ? row_of(g, gr.b, box_token(g, gr.bx, uq), gr.m) : 0;
  bf16x8_t qf[KS];  // Q^T as the B operand
  load_frag<D>(qf, q, qrow, qok);

  f32x16_t o[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) o[db] = f32x16_t{};
  Softmax sm;

  // S^T = K Q^T for 32-key block b of the tile in LDS buffer kb
  auto logits = [&](const uint16_t* kb, int b) {
    bf16x8_t a[KS];  // all operands read before the products, so the reads overlap
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) a[ks] = Tl::a_rows(kb, b * 32, ks);
    __builtin_amdgcn_sched_barrier(0);
    f32x16_t acc = f32x16_t{};
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) acc = mfma(a[ks], qf[ks], acc);
    return acc;
  };

  // Tile i is staged in LDS buffer i & 1; its global loads go out one tile ahead and its row
  // table is filled three tiles ahead.  One barrier per tile: a buffer or table slot is
  // rewritten only after the barrier that follows its last read, and read only after the
  // barrier that follows its write.
  uint4 kr[Tl::NL], vr[Tl::NL];
  __syncthreads();
  Tl::load(kr, k, tab[0], n);
  Tl::load(vr, v, tab[0], n);
  Tl::store(Ks[0], kr);
  Tl::store(Vs[0], vr);
  if (ntiles > 1) {
    Tl::load(kr, k, tab[1], n - KT);
    Tl::load(vr, v, tab[1], n - KT);
  }
  __syncthreads();
  for (int kt = 0; kt < ntiles; ++kt) {
    const uint16_t *kc = Ks[kt & 1], *vc = Vs[kt & 1];
    if (kt + 1 < ntiles) {
      Tl::store(Ks[(kt + 1) & 1], kr);
      Tl::store(Vs[(kt + 1) & 1], vr);
    }
    if (kt + 2 < ntiles) {
      const int* t2 = tab[(kt + 2) % 3];
      Tl::load(kr, k, t2, n - (kt + 2) * KT);
      Tl::load(vr, v, t2, n - (kt + 2) * KT);
    }
    if (kt + 3 < ntiles) fill_rows<KT>(tab[kt % 3], g, gr, (kt + 3) * KT);
    const int kbase = kt * KT;
    const int nb = min(NB, (n - kbase + 31) / 32);  // blocks holding at least one key
    f32x16_t cur = logits(kc, 0);
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      if (b >= nb) break;
      f32x16_t nxt;
      if (b + 1 < nb) nxt = logits(kc, b + 1);
      // V^T operands of this block, read now so that the softmax below hides their latency
      bf16x8_t av[DB][2];
#pragma unroll
      for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int p = 0; p < 2; ++p) av[db][p] = Tl::a_cols(vc, db * 32, b, p);
      float s[16];
#pragma unroll
      for (int i = 0; i < 16; ++i) s[i] = cur[i];
      if (kbase + b * 32 + 32 > n) {  // ragged block: keys past the box end get -inf
#pragma unroll
        for (int i = 0; i < 16; ++i)
          if (kbase + b * 32 + 8 * (i / 4) + 4 * hh + (i % 4) >= n) s[i] = -INFINITY;
      }
      float mx = fmaxf(fmaxf(s[0], s[1]), s[2]);
#pragma unroll
      for (int i = 3; i < 16; ++i) mx = fmaxf(mx, s[i]);
      mx = pair_max(mx) * g.scale_log2;  // scale > 0
      // The running maximum is raised only when a logit exceeds it by more than kSlack
      // (base 2), so P stays below 2^kSlack and the rescale of O is skipped by whole waves
      // most of the time; the result does not depend on which maximum was used.
      const bool raise = mx > sm.m + kSlack;
      if (__any(raise)) {
        const float mnew = raise ? mx : sm.m;
        const float corr = __builtin_amdgcn_exp2f(sm.m - mnew);
        sm.m = mnew;
        sm.l *= corr;
#pragma unroll
        for (int db = 0; db < DB; ++db) o[db] *= corr;
      }
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        s[i] = __builtin_amdgcn_exp2f(fmaf(s[i], g.scale_log2, -sm.m));
        sm.l += s[i];
      }
      bf16x8_t ph[2], pl[2];  // P^T as B-operand fragments (hi + lo)
      to_frags(s, ph, pl);
      // O^T += V^T P^T
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int p = 0; p < 2; ++p) {
          o[db] = mfma(av[db][p], ph[p], o[db]);
          o[db] = mfma(av[db][p], pl[p], o[db]);
        }
      cur = nxt;
    }
    __syncthreads();
  }

  const float ltot = pair_sum(sm.l);
  if (!qok) return;
  const float inv = 1.0f / ltot;
  const int64_t obase = qrow * D + 4 * hh;
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int blk = 0; blk < 4; ++blk) {
      __bf16 h[4], r[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const float x = o[db][4 * blk + j] * inv;
        h[j] = (__bf16)x;
        r[j] = (__bf16)(x - (float)h[j]);
      }
      const int64_t at = obase + db * 32 + 8 * blk;
      *reinterpret_cast<uint2*>(out + at) = __builtin_bit_cast(uint2, h);
      if (out_res != nullptr) *reinterpret_cast<uint2*>(out_res + at) = __builtin_bit_cast(uint2, r);
    }
  if (hh == 0 && lse != nullptr) lse[qrow] = (sm.m + __builtin_amdgcn_logf(ltot)) * kLn2;
}

// ---------------------------------------------------------------------------- backward

// dq pass: 128 queries of one group against every key of the box (as the forward), with
//   P = exp2(s log2(e) scale - lse log2(e)),  dP^T = V dout^T,  dS = P (dP - Delta),
//   dq^T += K^T dS^T  (scaled by `scale` at the end),
// and Delta = <dout, out + out_res> of each query (out alone without the residual), written
// to `delta` for the dk/dv pass.
template <int D>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2, 2))) void
win_dq_kernel(WinGeometry g, const uint16_t* __restrict__ q, const uint16_t* __restrict__ k,
              const uint16_t* __restrict__ v, const uint16_t* __restrict__ out,
              const uint16_t* __restrict__ out_res, const float* __restrict__ lse,
              const uint16_t* __restrict__ dout, float* __restrict__ dq,
              float* __restrict__ delta) {
  using Tl = Tile<D, kTile>;
  constexpr int KS = D / 16, DB = D / 32;
  __shared__ __attribute__((aligned(16))) uint16_t Ks[2][Tl::kElems];
  __shared__ __attribute__((aligned(16))) uint16_t Vs[2][Tl::kElems];
  __shared__ int tab[3][kTile];  // key rows of tile i in slot i % 3

  Group gr;
  if (!group_of(g, g.qtiles, gr)) return;
  const int q0 = gr.qt * kQTile, n = gr.bx.n;
  if (q0 >= n) return;
  const int ntiles = (n + kTile - 1) / kTile;
  for (int i = 0; i < 3 && i < ntiles; ++i) fill_rows<kTile>(tab[i], g, gr, i * kTile);

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, hh = lane >> 5;
  const int uq = q0 + wave * 32 + (lane & 31);
  const bool qok = uq < n;
  const int64_t qrow = qok ? row_of(g, gr.b, box_token(g, gr.bx, uq), gr.m) : 0;
  bf16x8_t qf[KS], gf[KS];
  load_frag<D>(qf, q, qrow, qok);
  load_frag<D>(gf, dout, qrow, qok);
  float dl;
  {
    bf16x8_t of[KS], rf[KS];
    load_frag<D>(of, out, qrow, qok);
    load_frag<D>(rf, out_res, qrow, qok && out_res != nullptr);
    float part = 0.0f;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
#pragma unroll
      for (int e = 0; e < 8; ++e)
        part = fmaf((float)gf[ks][e], (float)of[ks][e] + (float)rf[ks][e], part);
    dl = pair_sum(part);
  }
  if (qok && hh == 0) delta[qrow] = dl;
  const float lse2 = qok ? lse[qrow] * 1.4426950408889634f : 0.0f;

  f32x16_t acc[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) acc[db] = f32x16_t{};

  // staging as in the forward: tile i in LDS buffer i & 1, loads one tile ahead, row table
  // three tiles ahead, one barrier per tile
  uint4 kr[Tl::NL], vr[Tl::NL];
  __syncthreads();
  Tl::load(kr, k, tab[0], n);
  Tl::load(vr, v, tab[0], n);
  Tl::store(Ks[0], kr);
  Tl::store(Vs[0], vr);
  if (ntiles > 1) {
    Tl::load(kr, k, tab[1], n - kTile);
    Tl::load(vr, v, tab[1], n - kTile);
  }
  __syncthreads();
  for (int kt = 0; kt < ntiles; ++kt) {
    const uint16_t *kc = Ks[kt & 1], *vc = Vs[kt & 1];
    if (kt + 1 < ntiles) {
      Tl::store(Ks[(kt + 1) & 1], kr);
      Tl::store(Vs[(kt + 1) & 1], vr);
    }
    if (kt + 2 < ntiles) {
      const int* t2 = tab[(kt + 2) % 3];
      Tl::load(kr, k, t2, n - (kt + 2) * kTile);
      Tl::load(vr, v, t2, n - (kt + 2) * kTile);
    }
    if (kt + 3 < ntiles) fill_rows<kTile>(tab[kt % 3], g, gr, (kt + 3) * kTile);
    const int kbase = kt * kTile;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      f32x16_t sa = f32x16_t{}, pa = f32x16_t{};
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        sa = mfma(Tl::a_rows(kc, kb * 32, ks), qf[ks], sa);
        pa = mfma(Tl::a_rows(vc, kb * 32, ks), gf[ks], pa);
      }
      float ds[16];
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const float p = __builtin_amdgcn_exp2f(fmaf(sa[i], g.scale_log2, -lse2));
        ds[i] = p * (pa[i] - dl);
      }
      if (kbase + kb * 32 + 32 > n) {  // ragged block: keys past the box end contribute nothing
#pragma unroll
        for (int i = 0; i < 16; ++i)
          if (kbase + kb * 32 + 8 * (i / 4) + 4 * hh + (i % 4) >= n) ds[i] = 0.0f;
      }
      bf16x8_t dh[2], dlo[2];
      to_frags(ds, dh, dlo);
#pragma unroll
      for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int p = 0; p < 2; ++p) {
          const bf16x8_t a = Tl::a_cols(kc, db * 32, kb, p);
          acc[db] = mfma(a, dh[p], acc[db]);
          acc[db] = mfma(a, dlo[p], acc[db]);
        }
    }
    __syncthreads();
  }
  if (!qok) return;
#pragma unroll
  for (int db = 0; db < DB; ++db) store_f32_block(dq + qrow * D, db, acc[db], g.scale);
}

constexpr int kBoth = 0, kDvOnly = 1, kDkOnly = 2;

// dk/dv pass: 128 keys of one group (wave w owns keys 32 w .. 32 w + 31, lanes l and l ^ 32
// share key l % 32) against every query of the box, 64 queries per LDS tile:
//   S = Q K^T,  P = exp2(s log2(e) scale - lse log2(e)),  dP = dout V^T,  dS = P (dP - Delta),
//   dv^T += dout^T P,  dk^T += Q^T dS  (scaled by `scale` at the end).
// OUT selects the outputs: kBoth, or kDvOnly / kDkOnly, run as two launches whose accumulators
// (half of the 128 keys' dK and dV) fit two waves per SIMD instead of one; the dV launch does
// not form dP and the dK launch does not take P into a product.
template <int D, int OUT>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(OUT == kBoth ? 1 : 2, 2))) void
win_dkdv_kernel(WinGeometry g, const uint16_t* __restrict__ q, const uint16_t* __restrict__ k,
                const uint16_t* __restrict__ v, const float* __restrict__ lse,
                const uint16_t* __restrict__ dout, const float* __restrict__ delta,
                float* __restrict__ dk, float* __restrict__ dv) {
  using Tl = Tile<D, kTile>;
  constexpr int KS = D / 16, DB = D / 32;
  __shared__ __attribute__((aligned(16))) uint16_t Qs[2][Tl::kElems];
  __shared__ __attribute__((aligned(16))) uint16_t Gs[2][Tl::kElems];
  __shared__ __attribute__((aligned(16))) float Ls[2][kTile];  // lse log2(e); +inf past the end
  __shared__ __attribute__((aligned(16))) float Dl[2][kTile];  // Delta
  __shared__ int tab[3][kTile];  // query rows of tile i in slot i % 3

  Group gr;
  if (!group_of(g, g.qtiles, gr)) return;
  const int k0 = gr.qt * kQTile, n = gr.bx.n;
  if (k0 >= n) return;
  const int ntiles = (n + kTile - 1) / kTile;
  for (int i = 0; i < 3 && i < ntiles; ++i) fill_rows<kTile>(tab[i], g, gr, i * kTile);

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, hh = lane >> 5;
  const int uk = k0 + wave * 32 + (lane & 31);
  const bool kok = uk < n;
  const int64_t krow = kok ? row_of(g, gr.b, box_token(g, gr.bx, uk), gr.m) : 0;
  constexpr bool kDk = OUT != kDvOnly, kDv = OUT != kDkOnly, kLean = OUT == kDkOnly && D > 64;
  bf16x8_t kf[KS], vf[KS];  // K^T and V^T as B operands
  load_frag<D>(kf, k, krow, kok);
  if constexpr (kDk) load_frag<D>(vf, v, krow, kok);

  f32x16_t dka[DB], dva[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) dka[db] = dva[db] = f32x16_t{};

  // staging as in the forward: query tile i (q, dout, and the queries' lse and Delta) in LDS
  // buffer i & 1, loads one tile ahead, row table three tiles ahead, one barrier per tile
  uint4 rq[Tl::NL], rg[Tl::NL];
  float ls = INFINITY, de = 0.0f;
  auto fetch = [&](const int* t1, int valid) {
    Tl::load(rq, q, t1, valid);
    Tl::load(rg, dout, t1, valid);
    if (threadIdx.x < kTile) {
      const int row = t1[threadIdx.x];
      const bool ok = (int)threadIdx.x < valid;
      ls = ok ? lse[row] * 1.4426950408889634f : INFINITY;
      de = ok ? delta[row] : 0.0f;
    }
  };
  auto stage = [&](int buf) {
    Tl::store(Qs[buf], rq);
    Tl::store(Gs[buf], rg);
    if (threadIdx.x < kTile) {
      Ls[buf][threadIdx.x] = ls;
      Dl[buf][threadIdx.x] = de;
    }
  };
  __syncthreads();
  fetch(tab[0], n);
  stage(0);
  if (!kLean && ntiles > 1) fetch(tab[1], n - kTile);
  __syncthreads();
  for (int qt = 0; qt < ntiles; ++qt) {
    const uint16_t *Qc = Qs[qt & 1], *Gc = Gs[qt & 1];
    const float *Lc = Ls[qt & 1], *Dc = Dl[qt & 1];
    if constexpr (kLean) {  // no tile held in registers: the next one is loaded and stored here
      if (qt + 1 < ntiles) {
        fetch(tab[(qt + 1) % 3], n - (qt + 1) * kTile);
        stage((qt + 1) & 1);
      }
    } else {
      if (qt + 1 < ntiles) stage((qt + 1) & 1);
      if (qt + 2 < ntiles) fetch(tab[(qt + 2) % 3], n - (qt + 2) * kTile);
    }
    if (qt + 3 < ntiles) fill_rows<kTile>(tab[qt % 3], g, gr, (qt + 3) * kTile);
    // S and dP of 32-query block qb: operands read together, then the products; the lean form
    // (dK alone at D = 128, to fit two waves per SIMD) reads and multiplies one operand at a time
    auto sdp = [&](int qb, f32x16_t& sa, f32x16_t& pa) {
      if constexpr (kLean) {
        bf16x8_t a[KS];
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) a[ks] = Tl::a_rows(Qc, qb * 32, ks);
        __builtin_amdgcn_sched_barrier(0);
        sa = f32x16_t{};
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) sa = mfma(a[ks], kf[ks], sa);
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) a[ks] = Tl::a_rows(Gc, qb * 32, ks);
        __builtin_amdgcn_sched_barrier(0);
        pa = f32x16_t{};
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) pa = mfma(a[ks], vf[ks], pa);
        return;
      }
      bf16x8_t aq[KS], ag[KS];
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        aq[ks] = Tl::a_rows(Qc, qb * 32, ks);
        ag[ks] = Tl::a_rows(Gc, qb * 32, ks);
      }
      __builtin_amdgcn_sched_barrier(0);
      sa = f32x16_t{};
      pa = f32x16_t{};
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        sa = mfma(aq[ks], kf[ks], sa);
        if constexpr (kDk) pa = mfma(ag[ks], vf[ks], pa);
      }
    };
    f32x16_t sc, pc;
    if constexpr (!kLean) sdp(0, sc, pc);
#pragma unroll
    for (int qb = 0; qb < 2; ++qb) {
      // the next block's products go to the matrix cores before this block's softmax
      f32x16_t sn, pn;
      if constexpr (kLean) sdp(qb, sc, pc);
      else if (qb == 0) sdp(1, sn, pn);
      float p[16], ds[16];
#pragma unroll
      for (int blk = 0; blk < 4; ++blk) {  // the queries' lse and Delta
        const float4 l4 = *reinterpret_cast<const float4*>(Lc + qb * 32 + 8 * blk + 4 * hh);
        const float4 d4 = *reinterpret_cast<const float4*>(Dc + qb * 32 + 8 * blk + 4 * hh);
        const float lv[4] = {l4.x, l4.y, l4.z, l4.w}, dv4[4] = {d4.x, d4.y, d4.z, d4.w};
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int i = 4 * blk + j;
          p[i] = __builtin_amdgcn_exp2f(fmaf(sc[i], g.scale_log2, -lv[j]));
          ds[i] = p[i] * (pc[i] - dv4[j]);
        }
      }
      bf16x8_t ph[2], pl[2], dh[2], dlo[2];
      if constexpr (kDv) to_frags(p, ph, pl);
      if constexpr (kDk) to_frags(ds, dh, dlo);
#pragma unroll
      for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int pp = 0; pp < 2; ++pp) {
          if constexpr (kDv) {
            const bf16x8_t ag = Tl::a_cols(Gc, db * 32, qb, pp);
            dva[db] = mfma(ag, ph[pp], dva[db]);
            dva[db] = mfma(ag, pl[pp], dva[db]);
          }
          if constexpr (kDk) {
            const bf16x8_t aq = Tl::a_cols(Qc, db * 32, qb, pp);
            dka[db] = mfma(aq, dh[pp], dka[db]);
            dka[db] = mfma(aq, dlo[pp], dka[db]);
          }
        }
      if constexpr (!kLean) {
        sc = sn;
        pc = pn;
      }
    }
    __syncthreads();
  }
  if (!kok) return;
#pragma unroll
  for (int db = 0; db < DB; ++db) {
    if constexpr (kDk) store_f32_block(dk + krow * D, db, dka[db], g.scale);
    if constexpr (kDv) store_f32_block(dv + krow * D, db, dva[db], 1.0f);
  }
}

int ceil_div(int a, int b) { return (a + b - 1) / b; }

hipError_t mark(hipEvent_t const* events, int i, hipStream_t s) {
  return events != nullptr ? hipEventRecord(events[i], s) : hipSuccess;
}

template <int D>
hipError_t win_backward_d(const WinGeometry& g, const uint16_t* q, const uint16_t* k,
                          const uint16_t* v, const uint16_t* out, const uint16_t* res,
                          const float* lse,
                          const uint16_t* dout, float* dq, float* dk, float* dv, float* delta,
                          hipStream_t s, hipEvent_t const* events) {
  const dim3 grid((unsigned)win_forward_blocks(g)), block(kThreads);
  void* a1[] = {(void*)&g,   (void*)&q,    (void*)&k,  (void*)&v,    (void*)&out,
                (void*)&res, (void*)&lse, (void*)&dout, (void*)&dq, (void*)&delta};
  hipError_t e = mark(events, 0, s);
  if (e == hipSuccess)
    e = hipLaunchKernel(reinterpret_cast<const void*>(&win_dq_kernel<D>), grid, block, a1, 0, s);
  if (e == hipSuccess) e = mark(events, 1, s);
  if (e != hipSuccess) return e;
  const float* cdelta = delta;
  void* a2[] = {(void*)&g,   (void*)&q,    (void*)&k,      (void*)&v, (void*)&lse,
                (void*)&dout, (void*)&cdelta, (void*)&dk, (void*)&dv};
  e = hipLaunchKernel(reinterpret_cast<const void*>(&win_dkdv_kernel<D, kDvOnly>), grid, block,
                      a2, 0, s);
  if (e == hipSuccess)
    e = hipLaunchKernel(reinterpret_cast<const void*>(&win_dkdv_kernel<D, kDkOnly>), grid, block,
                        a2, 0, s);
  return e == hipSuccess ? mark(events, 2, s) : e;
}

}  // namespace

void win_plan(WinGeometry& g, int st, int sh, int sw) {
  g.off_t = st > 0 ? st - g.wt : 0;
  g.off_h = sh > 0 ? sh - g.wh : 0;
  g.off_w = sw > 0 ? sw - g.ww : 0;
  g.nt = ceil_div(g.T - g.off_t, g.wt);
  g.nh = ceil_div(g.H - g.off_h, g.wh);
  g.nw = ceil_div(g.W - g.off_w, g.ww);
  g.boxes = g.nt * g.nh * g.nw;
  g.max_box = std::min(g.wt, g.T) * std::min(g.wh, g.H) * std::min(g.ww, g.W);
  g.qtiles = ceil_div(g.max_box, kQTile);
  g.groups = g.B * g.boxes * g.heads;
  g.N = g.T * g.H * g.W;
}

int64_t win_forward_blocks(const WinGeometry& g) {
  return (int64_t)ceil_div(g.groups, kXcd) * kXcd * g.qtiles;
}

hipError_t launch_win_forward(const WinGeometry& g, const void* q, const void* k, const void* v,
                              void* out, void* out_res, float* lse, hipStream_t s) {
  const dim3 grid((unsigned)win_forward_blocks(g)), block(kThreads);
  const uint16_t *qq = static_cast<const uint16_t*>(q), *kk = static_cast<const uint16_t*>(k),
                 *vv = static_cast<const uint16_t*>(v);
  uint16_t *oo = static_cast<uint16_t*>(out), *rr = static_cast<uint16_t*>(out_res);
  void* a[] = {(void*)&g, (void*)&qq, (void*)&kk, (void*)&vv, (void*)&oo, (void*)&rr, (void*)&lse};
  const void* fn = g.D == 64 ? reinterpret_cast<const void*>(&win_fwd_kernel<64>)
                             : reinterpret_cast<const void*>(&win_fwd_kernel<128>);
  return hipLaunchKernel(fn, grid, block, a, 0, s);
}

hipError_t launch_win_backward(const WinGeometry& g, const void* q, const void* k, const void* v,
                               const void* out, const void* out_res, const float* lse,
                               const void* dout, float* dq, float* dk, float* dv,
                               void* workspace, hipStream_t s, hipEvent_t const* events) {
  const uint16_t *qq = static_cast<const uint16_t*>(q), *kk = static_cast<const uint16_t*>(k),
                 *vv = static_cast<const uint16_t*>(v), *oo = static_cast<const uint16_t*>(out),
                 *rr = static_cast<const uint16_t*>(out_res),
                 *gg = static_cast<const uint16_t*>(dout);
  float* delta = static_cast<float*>(workspace);
  return g.D == 64
             ? win_backward_d<64>(g, qq, kk, vv, oo, rr, lse, gg, dq, dk, dv, delta, s, events)
             : win_backward_d<128>(g, qq, kk, vv, oo, rr, lse, gg, dq, dk, dv, delta, s, events);
}

}  // namespace dsa3d
