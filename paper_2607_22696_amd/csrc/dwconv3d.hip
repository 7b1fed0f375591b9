// Depthwise 3D convolution of 3D-DSA: the DWConv3D term of MegaSlide-DiT's Eq. (1) (Section
// 5.2), also the depthwise nn.Conv3d (groups = channels) of the offset network (Section 5.3).
//
//   y[b,t,i,j,c] = bias[c] + sum_(a,e,f) w[c][a][e][f] x[b, t+a-rt, i+e-rh, j+f-rw, c]
//
// with zero padding ("same" size), channels last ([B][T][H][W][C], the activation layout).
//
// Lane layout: a lane owns 2 adjacent channels (one dword of bf16 or a float2), so a wave
// covers 128 channels of a token with one coalesced 256-byte (bf16) load.  A tile is 4 grid
// rows (one per wave of the block) by 8 consecutive tokens along x, for one 128-channel chunk.
// For its 8 tokens a wave reads each in-grid filter row (t+a-rt, i+e-rh) once, as the
// 8 + kw - 1 input columns the tokens need, and applies all kw taps of that row from
// registers.  The block's filter taps sit in LDS as [tap][lane] float2, staged when the
// channel chunk changes.  Outside the grid the filter rows are skipped and the columns read as
// zero.
//
// Work order: the grid holds only the blocks the chip can keep resident, and each block
// strides through the tiles, which are ordered channel chunk, batch, brick column (5 tiles =
// 40 tokens wide), frame, row quad, tile within the brick.  At any moment the tiles in flight
// on one XCD (one contiguous range of the order) then lie within a brick of about 1.5 frames x
// the grid height x 40 tokens, whose 3 x 3 x 3 neighbourhood (about 2.6 MB at 128 bf16
// channels) stays in that XCD's 4 MB L2 while every row of it is read by 9 output rows.
//
// dx is the same convolution of dy with the spatially reversed filter.  dw and dbias are
// reductions over the grid: a block owns one channel chunk and one filter plane a, sweeps its
// share of the tiles (the blocks of one (chunk, plane) interleave tile by tile, so they move
// through the grid together) and keeps the plane's taps summed in registers; each wave writes
// its sums to a workspace slot of its own, and a second kernel adds the slots in a fixed
// order, so the weight gradients are deterministic and no float atomics are used.
#include <type_traits>

#include "dsa3d_device.h"
#include "dsa3d_internal.h"

namespace dsa3d {
namespace {

using namespace dev;

constexpr int kChunk = 128;  // channels per wave (2 per lane)
constexpr int kTok = 8;      // consecutive tokens per tile along x
constexpr int kRows = 4;     // grid rows per tile (one per wave)

// Position of tile `q` (within one channel chunk and batch item) in the brick order.
struct TilePos {
  int t, i, j0;  // frame, this wave's row, first token
  bool valid;    // false for tiles past the grid's right edge (brick padding)
};

__device__ inline __attribute__((always_inline)) TilePos tile_pos(const ConvGeometry& g, int q,
                                                                  int wave) {
  const int s_in = q % g.sg;
  int r = q / g.sg;
  const int iq = r % g.hq;
  r /= g.hq;
  const int t = r % g.T;
  const int brick = r / g.T;
  TilePos p;
  p.t = t;
  p.i = iq * kRows + wave;
  p.j0 = (brick * g.sg + s_in) * kTok;
  p.valid = p.j0 < g.W;
  return p;
}

template <bool BF16>
__device__ inline __attribute__((always_inline)) float2 load2(const char* p) {
  if constexpr (BF16) {
    const uint32_t u = *reinterpret_cast<const uint32_t*>(p);
    return make_float2(__uint_as_float(u << 16), __uint_as_float(u & 0xffff0000u));
  } else {
    return *reinterpret_cast<const float2*>(p);
  }
}

// Stages the taps of channel chunk cc ([C][taps] in memory, the chunk contiguous) as
// wl[tap * 64 + lane] = (channel 2 lane, channel 2 lane + 1) of the chunk, reversed along the
// taps when FLIP; the global reads are consecutive.  Whole-block barrier before and after.
template <bool FLIP>
__device__ inline void stage_weights(const ConvGeometry& g, const float* __restrict__ w, int cc,
                                     float2* wl) {
  float* wf = reinterpret_cast<float*>(wl);
  const int64_t base = (int64_t)cc * kChunk * g.taps;
  const int n = min(kChunk, g.C - cc * kChunk) * g.taps;
  __syncthreads();
  for (int idx = threadIdx.x; idx < kChunk * g.taps; idx += kBlockThreads) {
    const int cl = idx / g.taps, tap = idx - cl * g.taps;
    const int dst = FLIP ? g.taps - 1 - tap : tap;
    wf[(dst * 64 + (cl >> 1)) * 2 + (cl & 1)] = idx < n ? w[base + idx] : 0.0f;
  }
  __syncthreads();
}

// out = conv(in) [+ bias] [+ out]; FLIP reverses the filter (the transposed convolution).
// Tiles are numbered chunk-major: tile = (cc * B + b) * g.tiles_per_bc + q.
// Two fp32 values rounded to nearest even as a bf16 pair (v_cvt_pk_bf16_f32), x in the low half.
__device__ inline __attribute__((always_inline)) uint32_t pack_bf16x2(float x, float y) {
  return __builtin_bit_cast(uint32_t, bf16x2_t{(__bf16)x, (__bf16)y});
}

template <bool IN_BF16, bool OUT_BF16, bool FLIP, int KW>
__global__ __launch_bounds__(kBlockThreads) void dwconv_kernel(ConvGeometry g,
                                                               const void* __restrict__ in,
                                                               const float* __restrict__ w,
                                                               const float* __restrict__ bias,
                                                               void* __restrict__ out,
                                                               int accumulate, int tiles) {
  extern __shared__ float2 wl[];
  constexpr int IS = IN_BF16 ? 2 : 4, OS = OUT_BF16 ? 2 : 4;
  constexpr int NX = kTok + KW - 1;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int rt = (g.kt - 1) / 2, rh = (g.kh - 1) / 2, rw = (KW - 1) / 2;
  const int64_t tok_in = (int64_t)g.C * IS;
  int staged = -1;
  for (int tile = xcd_tile(blockIdx.x, gridDim.x); tile < tiles; tile += gridDim.x) {
    const int bc = tile / g.tiles_per_bc;
    const int cc = bc / g.B, b = bc % g.B;
    if (cc != staged) {  // the same for every wave of the block: the barriers are uniform
      stage_weights<FLIP>(g, w, cc, wl);
      staged = cc;
    }
    const TilePos p = tile_pos(g, tile % g.tiles_per_bc, wave);
    const int c = cc * kChunk + 2 * lane;
    const bool active = c < g.C;
    if (!p.valid || p.i >= g.H) continue;
    float2 b2 = make_float2(0.0f, 0.0f);
    if (bias != nullptr && active) b2 = make_float2(bias[c], bias[c + 1]);
    float2 acc[kTok];
#pragma unroll
    for (int k = 0; k < kTok; ++k) acc[k] = b2;
    for (int a = 0; a < g.kt; ++a) {
      const int tt = p.t + a - rt;
      if ((unsigned)tt >= (unsigned)g.T) continue;
      for (int e = 0; e < g.kh; ++e) {
        const int ii = p.i + e - rh;
        if ((unsigned)ii >= (unsigned)g.H) continue;
        const char* row = static_cast<const char*>(in) +
                          (((int64_t)b * g.T + tt) * g.H + ii) * g.W * tok_in + (int64_t)c * IS;
        float2 xv[NX];
#pragma unroll
        for (int q = 0; q < NX; ++q) {
          const int col = p.j0 - rw + q;
          xv[q] = ((unsigned)col < (unsigned)g.W && active) ? load2<IN_BF16>(row + col * tok_in)
                                                             : make_float2(0.0f, 0.0f);
        }
        const float2* wr = wl + ((a * g.kh + e) * KW) * 64 + lane;
#pragma unroll
        for (int f = 0; f < KW; ++f) {
          const float2 wv = wr[f * 64];
#pragma unroll
          for (int k = 0; k < kTok; ++k) {
            acc[k].x = fmaf(wv.x, xv[k + f].x, acc[k].x);
            acc[k].y = fmaf(wv.y, xv[k + f].y, acc[k].y);
          }
        }
      }
    }
    if (!active) continue;
    char* orow = static_cast<char*>(out) +
                 ((((int64_t)b * g.T + p.t) * g.H + p.i) * g.W) * g.C * OS + (int64_t)c * OS;
#pragma unroll
    for (int k = 0; k < kTok; ++k) {
      const int j = p.j0 + k;
      if (j >= g.W) break;
      char* o = orow + (int64_t)j * g.C * OS;
      float2 v = acc[k];
      if (accumulate) {
        const float2 old = load2<OUT_BF16>(o);
        v.x += old.x;
        v.y += old.y;
      }
      if constexpr (OUT_BF16)
        *reinterpret_cast<uint32_t*>(o) = pack_bf16x2(v.x, v.y);
      else
        *reinterpret_cast<float2*>(o) = v;
    }
  }
}

// Weight and bias gradient partial sums.  Block (cc, a, p) for p < g.wg_blocks: filter plane a
// of channel chunk cc, tiles q = p, p + wg_blocks, ... of every batch item; each wave sums
//   acc[e][f] += dy[t, i, j] * x[t+a-rt, i+e-rh, j+f-rw]   over its rows of those tiles,
//   db += dy (plane 0 only)
// and writes slot (p * 4 + wave): part[slot][c][tap] (the plane's taps) and part_b[slot][c].
template <bool BF16, int KH, int KW>
__global__ __launch_bounds__(kBlockThreads) void dwconv_wgrad_kernel(
    ConvGeometry g, const void* __restrict__ x, const void* __restrict__ dy,
    float* __restrict__ part, float* __restrict__ part_b) {
  constexpr int IS = BF16 ? 2 : 4;
  constexpr int NX = kTok + KW - 1;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int rt = (g.kt - 1) / 2, rh = (KH - 1) / 2, rw = (KW - 1) / 2;
  const int64_t tok = (int64_t)g.C * IS;
  const int blk = xcd_tile(blockIdx.x, gridDim.x);
  const int pblk = blk % g.wg_blocks;
  const int a = (blk / g.wg_blocks) % g.kt;
  const int cc = blk / (g.wg_blocks * g.kt);
  const int c = cc * kChunk + 2 * lane;
  const bool active = c < g.C;
  float2 acc[KH][KW];
#pragma unroll
  for (int e = 0; e < KH; ++e)
#pragma unroll
    for (int f = 0; f < KW; ++f) acc[e][f] = make_float2(0.0f, 0.0f);
  float2 db = make_float2(0.0f, 0.0f);
  const int per_b = g.tiles_per_bc;
  for (int qq = pblk; qq < g.B * per_b && active; qq += g.wg_blocks) {
    const int b = qq / per_b;
    const TilePos p = tile_pos(g, qq % per_b, wave);
    if (!p.valid || p.i >= g.H) continue;
    const int tt = p.t + a - rt;
    const bool plane_in = (unsigned)tt < (unsigned)g.T;
    if (!plane_in && a != 0) continue;
    const char* dyrow = static_cast<const char*>(dy) +
                        ((((int64_t)b * g.T + p.t) * g.H + p.i) * g.W) * tok + (int64_t)c * IS;
    float2 d[kTok];
#pragma unroll
    for (int k = 0; k < kTok; ++k)
      d[k] = p.j0 + k < g.W ? load2<BF16>(dyrow + (int64_t)(p.j0 + k) * tok)
                            : make_float2(0.0f, 0.0f);
    if (a == 0) {
#pragma unroll
      for (int k = 0; k < kTok; ++k) {
        db.x += d[k].x;
        db.y += d[k].y;
      }
    }
    if (!plane_in) continue;
#pragma unroll
    for (int e = 0; e < KH; ++e) {
      const int ii = p.i + e - rh;
      if ((unsigned)ii >= (unsigned)g.H) continue;
      const char* xrow = static_cast<const char*>(x) +
                         (((int64_t)b * g.T + tt) * g.H + ii) * g.W * tok + (int64_t)c * IS;
      float2 xv[NX];
#pragma unroll
      for (int q = 0; q < NX; ++q) {
        const int col = p.j0 - rw + q;
        xv[q] = (unsigned)col < (unsigned)g.W ? load2<BF16>(xrow + col * tok)
                                              : make_float2(0.0f, 0.0f);
      }
#pragma unroll
      for (int f = 0; f < KW; ++f)
#pragma unroll
        for (int k = 0; k < kTok; ++k) {
          acc[e][f].x = fmaf(d[k].x, xv[k + f].x, acc[e][f].x);
          acc[e][f].y = fmaf(d[k].y, xv[k + f].y, acc[e][f].y);
        }
    }
  }
  if (!active) return;
  const int64_t slot = (int64_t)pblk * kWavesPerBlock + wave;
  float* pc0 = part + (slot * g.C + c) * g.taps + a * KH * KW;
  float* pc1 = pc0 + g.taps;
#pragma unroll
  for (int e = 0; e < KH; ++e)
#pragma unroll
    for (int f = 0; f < KW; ++f) {
      pc0[e * KW + f] = acc[e][f].x;
      pc1[e * KW + f] = acc[e][f].y;
    }
  if (a == 0) {
    part_b[slot * g.C + c] = db.x;
    part_b[slot * g.C + c + 1] = db.y;
  }
}

// dw[c][tap] = sum over slots of part[slot][c][tap] (slots in order); db likewise.
__global__ __launch_bounds__(kBlockThreads) void dwconv_wgrad_reduce_kernel(
    const float* __restrict__ part, const float* __restrict__ part_b, int64_t per_slot,
    int64_t per_slot_b, int slots, float* __restrict__ dw, float* __restrict__ db) {
  const int64_t n = per_slot + per_slot_b;
  for (int64_t o = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; o < n;
       o += (int64_t)gridDim.x * blockDim.x) {
    const bool is_b = o >= per_slot;
    if (is_b ? db == nullptr : dw == nullptr) continue;
    const float* src = is_b ? part_b + (o - per_slot) : part + o;
    const int64_t stride = is_b ? per_slot_b : per_slot;
    float s = 0.0f;
    for (int k = 0; k < slots; ++k) s += src[k * stride];
    if (is_b)
      db[o - per_slot] = s;
    else
      dw[o] = s;
  }
}

// ---------------------------------------------------------------------------- time streaming

// Fast path for bf16 data and filters of at most 3 along every axis.  A block owns a brick of
// 4 grid rows x 8 tokens x 128 channels and walks all frames.  One input slice of the brick (its
// rows and columns plus the filter's halo, zero outside the grid) is staged per frame, in one of
// two LDS buffers; while a slice is used, the next one is stored into the other buffer and the
// one after that is in flight into registers, so every input element comes from HBM about once
// (the halo columns and rows are re-read, mostly from L2, by the neighbouring bricks, which walk
// the frames at the same time).  The filter taps are in registers.
template <int KT, int KH, int KW>
struct SliceShape {
  static constexpr int RY = kRows + KH - 1;  // slice rows
  static constexpr int RX = kTok + KW - 1;   // slice columns
  static constexpr int POS = RY * RX;        // token positions per slice
  static constexpr int PER_WAVE = (POS + kWavesPerBlock - 1) / kWavesPerBlock;
  static constexpr int TAPS = KT * KH * KW;
};

// The slice positions this wave loads: 32-bit byte offsets within a frame (UINT32_MAX, which the
// buffer unit reads as zero, outside the grid or the channel range), computed once per brick.
template <int KT, int KH, int KW>
__device__ inline void slice_offsets(const ConvGeometry& g, int i0, int j0, int c, int wave,
                                     uint32_t (&off)[SliceShape<KT, KH, KW>::PER_WAVE]) {
  using RG = SliceShape<KT, KH, KW>;
  const int rh = (KH - 1) / 2, rw = (KW - 1) / 2;
#pragma unroll
  for (int k = 0; k < RG::PER_WAVE; ++k) {
    const int pos = wave + kWavesPerBlock * k;
    const int y = pos / RG::RX, x = pos % RG::RX;
    const int ii = i0 - rh + y, jj = j0 - rw + x;
    const bool in = pos < RG::POS && c < g.C && (unsigned)ii < (unsigned)g.H &&
                    (unsigned)jj < (unsigned)g.W;
    off[k] = in ? (uint32_t)(((uint32_t)ii * g.W + jj) * (uint32_t)g.C + c) * 2u : 0xffffffffu;
  }
}

// Raw buffer over frame f of one batch item (f outside [0, T): zero records, so every load of
// it returns zero); offsets at or beyond the frame's size also read as zero.
__device__ inline __attribute__((always_inline)) __amdgpu_buffer_rsrc_t frame_rsrc(
    const char* batch_base, int frame_bytes, int f, int T) {
  const bool fin = (unsigned)f < (unsigned)T;
  return __builtin_amdgcn_make_buffer_rsrc(
      (void*)(batch_base + (int64_t)(fin ? f : 0) * frame_bytes), (short)0, fin ? frame_bytes : 0,
      kBufferFlags);
}

template <int KT, int KH, int KW>
__device__ inline __attribute__((always_inline)) void load_slice(
    const char* batch_base, int frame_bytes, int f, int T,
    const uint32_t (&off)[SliceShape<KT, KH, KW>::PER_WAVE], uint32_t (&v)[SliceShape<KT, KH, KW>::PER_WAVE]) {
  const __amdgpu_buffer_rsrc_t r = frame_rsrc(batch_base, frame_bytes, f, T);
#pragma unroll
  for (int k = 0; k < SliceShape<KT, KH, KW>::PER_WAVE; ++k)
    v[k] = (uint32_t)__builtin_amdgcn_raw_buffer_load_b32(r, (int)off[k], 0, 0);
}

__device__ inline __attribute__((always_inline)) float2 bf16x2(uint32_t u) {
  return make_float2(__uint_as_float(u << 16), __uint_as_float(u & 0xffff0000u));
}

// out = conv(in) [+ bias] [+ out] for bf16 `in`; bricks ordered chunk, batch, row quad, strip.
// The brick walks the input frames once: slice s (its rows and columns plus the filter halo)
// sits in LDS buffer s & 1, each wave widens the KH rows it needs to fp32 once, and adds them
// through filter plane a into output frame s + rt - a, for every a.  The KT output frames in
// progress are held in registers and shift down by one slot per slice; frame t is stored once
// slice t + rt has been added.
template <bool OUT_BF16, bool FLIP, int KT, int KH, int KW>
__global__ __launch_bounds__(kBlockThreads) __attribute__((amdgpu_waves_per_eu(2))) void dwconv_stream_kernel(
    ConvGeometry g, const void* __restrict__ in, const float* __restrict__ w,
    const float* __restrict__ bias, void* __restrict__ out, int accumulate, int bricks) {
  using RG = SliceShape<KT, KH, KW>;
  static_assert(KT == 1 || KT == 3, "time extent 1 or 3");
  __shared__ uint32_t slices[2][RG::POS * 64];
  constexpr int OS = OUT_BF16 ? 2 : 4;
  constexpr int rt = (KT - 1) / 2;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int frame_bytes = g.H * g.W * g.C * 2;  // below 2^31 on this path
  for (int brick = xcd_tile(blockIdx.x, gridDim.x); brick < bricks; brick += gridDim.x) {
    const int strip = brick % g.strips;
    int r = brick / g.strips;
    const int iq = r % g.hq;
    r /= g.hq;
    const int b = r % g.B, cc = r / g.B;
    const int c = cc * kChunk + 2 * lane;
    const bool active = c < g.C;
    const int i0 = iq * kRows, j0 = strip * kTok, i = i0 + wave;
    float2 wt[RG::TAPS];
#pragma unroll
    for (int tap = 0; tap < RG::TAPS; ++tap) {
      const int src = FLIP ? RG::TAPS - 1 - tap : tap;
      wt[tap] = active ? make_float2(w[(int64_t)c * RG::TAPS + src], w[(int64_t)(c + 1) * RG::TAPS + src])
                       : make_float2(0.0f, 0.0f);
    }
    float2 b2 = make_float2(0.0f, 0.0f);
    if (bias != nullptr && active) b2 = make_float2(bias[c], bias[c + 1]);
    uint32_t off[RG::PER_WAVE];
    slice_offsets<KT, KH, KW>(g, i0, j0, c, wave, off);
    const char* base = static_cast<const char*>(in) + (int64_t)b * g.T * frame_bytes;
    char* obase = static_cast<char*>(out) + (int64_t)b * g.T * g.H * g.W * g.C * OS;

    // While slice s is added, slot j holds output frame s - rt + j: plane a carries the slice
    // into slot KT - 1 - a, slot 0 is then complete, and the slots shift down by one.
    float2 acc[KT][kTok];
#pragma unroll
    for (int sl = 0; sl < KT; ++sl)
#pragma unroll
      for (int k = 0; k < kTok; ++k) acc[sl][k] = b2;
    auto put = [&](int buf, const uint32_t (&v)[RG::PER_WAVE]) {
#pragma unroll
      for (int k = 0; k < RG::PER_WAVE; ++k) {
        const int pos = wave + kWavesPerBlock * k;
        if (pos < RG::POS) slices[buf][pos * 64 + lane] = v[k];
      }
    };
    // stores output frame t (slot 0) of this wave's row
    auto emit = [&](int t) {
      if (!active || i >= g.H) return;
      char* orow = obase + (((int64_t)t * g.H + i) * g.W) * g.C * OS + (int64_t)c * OS;
#pragma unroll
      for (int k = 0; k < kTok; ++k) {
        if (j0 + k >= g.W) break;
        char* o = orow + (int64_t)(j0 + k) * g.C * OS;
        float2 v = acc[0][k];
        if (accumulate) {
          const float2 old = load2<OUT_BF16>(o);
          v.x += old.x;
          v.y += old.y;
        }
        if constexpr (OUT_BF16)
          *reinterpret_cast<uint32_t*>(o) = pack_bf16x2(v.x, v.y);
        else
          *reinterpret_cast<float2*>(o) = v;
      }
    };
    uint32_t nxt[RG::PER_WAVE];
    load_slice<KT, KH, KW>(base, frame_bytes, 0, g.T, off, nxt);
    put(0, nxt);  // the previous brick ended on a barrier after its last read
    if (g.T > 1) load_slice<KT, KH, KW>(base, frame_bytes, 1, g.T, off, nxt);
    __syncthreads();
#pragma unroll 1
    for (int s = 0; s < g.T; ++s) {
      // store slice s + 1, request slice s + 2, add slice s
      if (s + 1 < g.T) {
        put((s + 1) & 1, nxt);
        if (s + 2 < g.T) load_slice<KT, KH, KW>(base, frame_bytes, s + 2, g.T, off, nxt);
      }
      const uint32_t* cur = slices[s & 1];
#pragma unroll
      for (int e = 0; e < KH; ++e) {
        const uint32_t* src = cur + (wave + e) * RG::RX * 64 + lane;
        float2 xv[RG::RX];
#pragma unroll
        for (int x = 0; x < RG::RX; ++x) xv[x] = bf16x2(src[x * 64]);
#pragma unroll
        for (int a = 0; a < KT; ++a) {
          if (s + rt - a >= g.T) continue;  // that output frame is past the end
#pragma unroll
          for (int f = 0; f < KW; ++f) {
            const float2 wv = wt[(a * KH + e) * KW + f];
#pragma unroll
            for (int k = 0; k < kTok; ++k) {
              acc[KT - 1 - a][k].x = fmaf(wv.x, xv[k + f].x, acc[KT - 1 - a][k].x);
              acc[KT - 1 - a][k].y = fmaf(wv.y, xv[k + f].y, acc[KT - 1 - a][k].y);
            }
          }
        }
        asm volatile("" ::: "memory");  // one row's reads in flight at a time (registers)
      }
      if (s - rt >= 0) emit(s - rt);
#pragma unroll
      for (int sl = 0; sl + 1 < KT; ++sl)
#pragma unroll
        for (int k = 0; k < kTok; ++k) acc[sl][k] = acc[sl + 1][k];
#pragma unroll
      for (int k = 0; k < kTok; ++k) acc[KT - 1][k] = b2;
      __syncthreads();  // slice s is read; its buffer takes slice s + 2 next
    }
    // frames T - rt .. T - 1 are complete after the last slice (slots 0 .. rt - 1)
    if constexpr (rt == 1) emit(g.T - 1);
  }
}

// Weight and bias gradient partial sums on the streaming path: one brick per block; wave w of
// brick (cc, b, iq, strip) writes slot ((b * hq + iq) * strips + strip) * 4 + w, its sums
// over all frames of its row of the brick.  As in the forward, the x slices are walked once
// (LDS buffer s & 1, each row widened once per wave): slice s meets dy frame s + rt - a through
// filter plane a, and the KT dy frames in use are held in registers (slot j: frame s - rt + j),
// shifting down by one per slice.
template <int KT, int KH, int KW>
__global__ __launch_bounds__(kBlockThreads) void dwconv_stream_wgrad_kernel(
    ConvGeometry g, const void* __restrict__ x, const void* __restrict__ dy,
    float* __restrict__ part, float* __restrict__ part_b) {
  using RG = SliceShape<KT, KH, KW>;
  static_assert(KT == 1 || KT == 3, "time extent 1 or 3");
  __shared__ uint32_t slices[2][RG::POS * 64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  constexpr int rt = (KT - 1) / 2;
  const int frame_bytes = g.H * g.W * g.C * 2;  // below 2^31 on this path
  const int brick = xcd_tile(blockIdx.x, gridDim.x);
  const int strip = brick % g.strips;
  int r = brick / g.strips;
  const int iq = r % g.hq;
  r /= g.hq;
  const int b = r % g.B, cc = r / g.B;
  const int c = cc * kChunk + 2 * lane;
  const bool active = c < g.C;
  const int i0 = iq * kRows, j0 = strip * kTok, i = i0 + wave;
  uint32_t off[RG::PER_WAVE];
  slice_offsets<KT, KH, KW>(g, i0, j0, c, wave, off);
  // this wave's dy row: 8 tokens at byte offsets within a frame (UINT32_MAX outside)
  uint32_t doff[kTok];
#pragma unroll
  for (int k = 0; k < kTok; ++k)
    doff[k] = (active && i < g.H && j0 + k < g.W)
                  ? (uint32_t)(((uint32_t)i * g.W + j0 + k) * (uint32_t)g.C + c) * 2u
                  : 0xffffffffu;
  const char* xbase = static_cast<const char*>(x) + (int64_t)b * g.T * frame_bytes;
  const char* dbase = static_cast<const char*>(dy) + (int64_t)b * g.T * frame_bytes;
  auto load_dy = [&](int f, uint32_t (&v)[kTok]) {  // zeros outside [0, T)
    const __amdgpu_buffer_rsrc_t rs = frame_rsrc(dbase, frame_bytes, f, g.T);
#pragma unroll
    for (int k = 0; k < kTok; ++k) v[k] = (uint32_t)__builtin_amdgcn_raw_buffer_load_b32(rs, (int)doff[k], 0, 0);
  };
  auto put = [&](int buf, const uint32_t (&v)[RG::PER_WAVE]) {
#pragma unroll
    for (int k = 0; k < RG::PER_WAVE; ++k) {
      const int pos = wave + kWavesPerBlock * k;
      if (pos < RG::POS) slices[buf][pos * 64 + lane] = v[k];
    }
  };
  float2 acc[RG::TAPS];
#pragma unroll
  for (int tap = 0; tap < RG::TAPS; ++tap) acc[tap] = make_float2(0.0f, 0.0f);
  float2 db = make_float2(0.0f, 0.0f);
  // dy window: slot j = frame s - rt + j (frames below 0 are zero)
  float2 d[KT][kTok];
#pragma unroll
  for (int j = 0; j < KT; ++j) {
    uint32_t v[kTok];
    load_dy(j - rt, v);
#pragma unroll
    for (int k = 0; k < kTok; ++k) {
      d[j][k] = bf16x2(v[k]);
      if (j >= rt) {  // frames 0 .. rt enter the bias sum here, later ones as they arrive
        db.x += d[j][k].x;
        db.y += d[j][k].y;
      }
    }
  }
  uint32_t dnxt[kTok];
  load_dy(rt + 1, dnxt);
  uint32_t nxt[RG::PER_WAVE];
  load_slice<KT, KH, KW>(xbase, frame_bytes, 0, g.T, off, nxt);
  put(0, nxt);
  if (g.T > 1) load_slice<KT, KH, KW>(xbase, frame_bytes, 1, g.T, off, nxt);
  __syncthreads();
#pragma unroll 1
  for (int s = 0; s < g.T; ++s) {
    if (s + 1 < g.T) {
      put((s + 1) & 1, nxt);
      if (s + 2 < g.T) load_slice<KT, KH, KW>(xbase, frame_bytes, s + 2, g.T, off, nxt);
    }
    const uint32_t* cur = slices[s & 1];
#pragma unroll
    for (int e = 0; e < KH; ++e) {
      const uint32_t* src = cur + (wave + e) * RG::RX * 64 + lane;
      float2 xv[RG::RX];
#pragma unroll
      for (int q = 0; q < RG::RX; ++q) xv[q] = bf16x2(src[q * 64]);
#pragma unroll
      for (int a = 0; a < KT; ++a) {
#pragma unroll
        for (int f = 0; f < KW; ++f)
#pragma unroll
          for (int k = 0; k < kTok; ++k) {
            const float2 dv = d[KT - 1 - a][k];  // dy frame s + rt - a (zero outside the grid)
            acc[(a * KH + e) * KW + f].x = fmaf(dv.x, xv[k + f].x, acc[(a * KH + e) * KW + f].x);
            acc[(a * KH + e) * KW + f].y = fmaf(dv.y, xv[k + f].y, acc[(a * KH + e) * KW + f].y);
          }
      }
      asm volatile("" ::: "memory");  // one row's reads in flight at a time (registers)
    }
    // shift the dy window; frame s + rt + 1 enters (and the bias sum)
#pragma unroll
    for (int j = 0; j + 1 < KT; ++j)
#pragma unroll
      for (int k = 0; k < kTok; ++k) d[j][k] = d[j + 1][k];
#pragma unroll
    for (int k = 0; k < kTok; ++k) {
      d[KT - 1][k] = bf16x2(dnxt[k]);
      db.x += d[KT - 1][k].x;
      db.y += d[KT - 1][k].y;
    }
    load_dy(s + rt + 2, dnxt);
    __syncthreads();  // slice s is read; its buffer takes slice s + 2 next
  }
  if (!active) return;
  const int64_t slot = (((int64_t)b * g.hq + iq) * g.strips + strip) * kWavesPerBlock + wave;
  float* pc0 = part + (slot * g.C + c) * RG::TAPS;
  float* pc1 = pc0 + RG::TAPS;
#pragma unroll
  for (int tap = 0; tap < RG::TAPS; ++tap) {
    pc0[tap] = acc[tap].x;
    pc1[tap] = acc[tap].y;
  }
  part_b[slot * g.C + c] = db.x;
  part_b[slot * g.C + c + 1] = db.y;
}

// ---------------------------------------------------------------------------- launch

// Blocks of `kernel` the device keeps resident at once (all CUs), at least 1.
int resident_blocks(const void* kernel, size_t lds) {
  int dev = 0, cus = 0, per_cu = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel, kBlockThreads, lds) !=
          hipSuccess)
    return 1;
  const int n = cus * per_cu;
  return n > 0 ? n : 1;
}

template <bool IN_BF16, bool OUT_BF16, bool FLIP, int KW>
hipError_t launch_conv(const ConvGeometry& g, const void* in, const float* w, const float* bias,
                       void* out, int accumulate, hipStream_t s) {
  const void* k = reinterpret_cast<const void*>(&dwconv_kernel<IN_BF16, OUT_BF16, FLIP, KW>);
  const int tiles = g.chunks * g.B * g.tiles_per_bc;
  const size_t lds = (size_t)g.taps * 64 * sizeof(float2);
  const int res = resident_blocks(k, lds);
  const int blocks = tiles < res ? tiles : res;
  void* a[] = {(void*)&g, (void*)&in, (void*)&w, (void*)&bias, (void*)&out, (void*)&accumulate,
               (void*)&tiles};
  return hipLaunchKernel(k, dim3(blocks), dim3(kBlockThreads), a, lds, s);
}

template <bool IN_BF16, bool OUT_BF16, bool FLIP>
hipError_t conv_kw(const ConvGeometry& g, const void* in, const float* w, const float* bias,
                   void* out, int accumulate, hipStream_t s) {
  switch (g.kw) {
    case 1: return launch_conv<IN_BF16, OUT_BF16, FLIP, 1>(g, in, w, bias, out, accumulate, s);
    case 3: return launch_conv<IN_BF16, OUT_BF16, FLIP, 3>(g, in, w, bias, out, accumulate, s);
    case 5: return launch_conv<IN_BF16, OUT_BF16, FLIP, 5>(g, in, w, bias, out, accumulate, s);
    case 7: return launch_conv<IN_BF16, OUT_BF16, FLIP, 7>(g, in, w, bias, out, accumulate, s);
    default: return hipErrorInvalidValue;
  }
}

template <bool BF16, int KH, int KW>
hipError_t launch_wgrad(const ConvGeometry& g, const void* x, const void* dy, float* part,
                        float* part_b, hipStream_t s) {
  const int blocks = g.chunks * g.kt * g.wg_blocks;
  void* a[] = {(void*)&g, (void*)&x, (void*)&dy, (void*)&part, (void*)&part_b};
  return hipLaunchKernel(reinterpret_cast<const void*>(&dwconv_wgrad_kernel<BF16, KH, KW>),
                         dim3(blocks), dim3(kBlockThreads), a, 0, s);
}

template <bool BF16, int KH>
hipError_t wgrad_kw(const ConvGeometry& g, const void* x, const void* dy, float* part,
                    float* part_b, hipStream_t s) {
  switch (g.kw) {
    case 1: return launch_wgrad<BF16, KH, 1>(g, x, dy, part, part_b, s);
    case 3: return launch_wgrad<BF16, KH, 3>(g, x, dy, part, part_b, s);
    case 5: return launch_wgrad<BF16, KH, 5>(g, x, dy, part, part_b, s);
    case 7: return launch_wgrad<BF16, KH, 7>(g, x, dy, part, part_b, s);
    default: return hipErrorInvalidValue;
  }
}

template <bool BF16>
hipError_t wgrad_kh(const ConvGeometry& g, const void* x, const void* dy, float* part,
                    float* part_b, hipStream_t s) {
  switch (g.kh) {
    case 1: return wgrad_kw<BF16, 1>(g, x, dy, part, part_b, s);
    case 3: return wgrad_kw<BF16, 3>(g, x, dy, part, part_b, s);
    case 5: return wgrad_kw<BF16, 5>(g, x, dy, part, part_b, s);
    case 7: return wgrad_kw<BF16, 7>(g, x, dy, part, part_b, s);
    default: return hipErrorInvalidValue;
  }
}

int stream_bricks(const ConvGeometry& g) { return g.chunks * g.B * g.hq * g.strips; }

template <bool OUT_BF16, bool FLIP, int KT, int KH, int KW>
hipError_t launch_stream(const ConvGeometry& g, const void* in, const float* w, const float* bias,
                         void* out, int accumulate, hipStream_t s) {
  const int bricks = stream_bricks(g);
  const int blocks = bricks < kMaxBlocks ? bricks : kMaxBlocks;
  void* a[] = {(void*)&g, (void*)&in, (void*)&w, (void*)&bias, (void*)&out, (void*)&accumulate,
               (void*)&bricks};
  return hipLaunchKernel(
      reinterpret_cast<const void*>(&dwconv_stream_kernel<OUT_BF16, FLIP, KT, KH, KW>),
      dim3(blocks), dim3(kBlockThreads), a, 0, s);
}

template <int KT, int KH, int KW>
hipError_t launch_stream_wgrad(const ConvGeometry& g, const void* x, const void* dy, float* part,
                               float* part_b, hipStream_t s) {
  void* a[] = {(void*)&g, (void*)&x, (void*)&dy, (void*)&part, (void*)&part_b};
  return hipLaunchKernel(reinterpret_cast<const void*>(&dwconv_stream_wgrad_kernel<KT, KH, KW>),
                         dim3(stream_bricks(g)), dim3(kBlockThreads), a, 0, s);
}

// The filter shapes the streaming path covers: every extent 1 or 3.
#define DSA3D_STREAM_SHAPES(X) \
  X(1, 1, 1) X(1, 1, 3) X(1, 3, 1) X(1, 3, 3) X(3, 1, 1) X(3, 1, 3) X(3, 3, 1) X(3, 3, 3)

template <bool OUT_BF16, bool FLIP>
hipError_t stream_conv(const ConvGeometry& g, const void* in, const float* w, const float* bias,
                       void* out, int accumulate, hipStream_t s) {
#define DSA3D_CASE(KT, KH, KW)                    \
  if (g.kt == KT && g.kh == KH && g.kw == KW)     \
    return launch_stream<OUT_BF16, FLIP, KT, KH, KW>(g, in, w, bias, out, accumulate, s);
  DSA3D_STREAM_SHAPES(DSA3D_CASE)
#undef DSA3D_CASE
  return hipErrorInvalidValue;
}

hipError_t stream_wgrad(const ConvGeometry& g, const void* x, const void* dy, float* part,
                        float* part_b, hipStream_t s) {
#define DSA3D_CASE(KT, KH, KW)                \
  if (g.kt == KT && g.kh == KH && g.kw == KW) \
    return launch_stream_wgrad<KT, KH, KW>(g, x, dy, part, part_b, s);
  DSA3D_STREAM_SHAPES(DSA3D_CASE)
#undef DSA3D_CASE
  return hipErrorInvalidValue;
}

}  // namespace

// Blocks per (chunk, plane) of the weight-gradient sweep: about 768 blocks in all, which the
// 256 CUs keep resident at once (three per CU at the 3 x 3 kernel's register use), so the
// blocks of one (chunk, plane) move through the grid together; at most one per tile.
constexpr int kWgradBlocksTarget = 768;

void conv_plan(ConvGeometry& g) {
  g.taps = g.kt * g.kh * g.kw;
  // the streaming path: bf16 data, every filter extent 1 or 3, frames below 2 GB (a raw buffer
  // of one frame)
  g.stream = g.bf16 && g.kt <= 3 && g.kh <= 3 && g.kw <= 3 &&
             (uint64_t)g.H * g.W * g.C * 2 < 0x7fffffffull;
  g.chunks = (g.C + kChunk - 1) / kChunk;
  g.strips = (g.W + kTok - 1) / kTok;
  g.sg = g.strips < 5 ? g.strips : 5;
  g.hq = (g.H + kRows - 1) / kRows;
  const int bricks = (g.strips + g.sg - 1) / g.sg;
  g.tiles_per_bc = bricks * g.T * g.hq * g.sg;
  const int want = kWgradBlocksTarget / (g.chunks * g.kt);
  const int64_t per_pair = (int64_t)g.B * g.tiles_per_bc;
  g.wg_blocks = (int)(want < 1 ? 1 : (want > per_pair ? per_pair : want));
}

// Partial-sum slots of the weight-gradient sweep: one per wave of a brick on the streaming path,
// one per wave of a sweep block otherwise.
size_t conv_slots(const ConvGeometry& g) {
  return g.stream ? (size_t)g.B * g.hq * g.strips * kWavesPerBlock
                  : (size_t)g.wg_blocks * kWavesPerBlock;
}

size_t conv_workspace_bytes(const ConvGeometry& g) {
  const size_t slots = conv_slots(g);
  const size_t part = slots * g.C * g.taps * sizeof(float);
  const size_t part_b = slots * g.C * sizeof(float);
  return ((part + 255) & ~size_t(255)) + ((part_b + 255) & ~size_t(255));
}

hipError_t launch_conv_forward(const ConvGeometry& g, bool bf16, const void* x, const float* w,
                               const float* bias, void* y, int accumulate, hipStream_t s) {
  if (g.stream) return stream_conv<true, false>(g, x, w, bias, y, accumulate, s);
  return bf16 ? conv_kw<true, true, false>(g, x, w, bias, y, accumulate, s)
              : conv_kw<false, false, false>(g, x, w, bias, y, accumulate, s);
}

hipError_t launch_conv_backward(const ConvGeometry& g, bool bf16, const void* x, const float* w,
                                const void* dy, float* dx, int accumulate_dx, float* dw, float* db,
                                void* workspace, hipStream_t s) {
  hipError_t e = hipSuccess;
  if (dx != nullptr) {
    if (g.stream)
      e = stream_conv<false, true>(g, dy, w, nullptr, dx, accumulate_dx, s);
    else
      e = bf16 ? conv_kw<true, false, true>(g, dy, w, nullptr, dx, accumulate_dx, s)
               : conv_kw<false, false, true>(g, dy, w, nullptr, dx, accumulate_dx, s);
    if (e != hipSuccess) return e;
  }
  if (dw == nullptr && db == nullptr) return e;
  const size_t slots = conv_slots(g);
  const size_t part_bytes = slots * g.C * g.taps * sizeof(float);
  float* part = static_cast<float*>(workspace);
  float* part_b = reinterpret_cast<float*>(static_cast<char*>(workspace) +
                                           ((part_bytes + 255) & ~size_t(255)));
  if (g.stream)
    e = stream_wgrad(g, x, dy, part, part_b, s);
  else
    e = bf16 ? wgrad_kh<true>(g, x, dy, part, part_b, s) : wgrad_kh<false>(g, x, dy, part, part_b, s);
  if (e != hipSuccess) return e;
  const int64_t per_slot = (int64_t)g.C * g.taps, per_slot_b = g.C;
  const int nslots = (int)slots;
  const int64_t n = per_slot + per_slot_b;
  const int blocks = (int)((n + kBlockThreads - 1) / kBlockThreads);
  void* a[] = {(void*)&part, (void*)&part_b, (void*)&per_slot, (void*)&per_slot_b,
               (void*)&nslots, (void*)&dw, (void*)&db};
  return hipLaunchKernel(reinterpret_cast<const void*>(&dwconv_wgrad_reduce_kernel), dim3(blocks),
                         dim3(kBlockThreads), a, 0, s);
}

}  // namespace dsa3d
