// Internal interface between the C-ABI host code and the gfx950 kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace dsa3d {

// Problem geometry as the kernels see it (validated on the host).
struct Geometry {
  int B, T, H, W;     // batch, frames, grid height, grid width
  int heads, D;       // heads, head_dim
  int kt, kh, kw, P;  // neighbourhood and its point count
  int N;              // tokens per batch item, T*H*W
  float scale;        // logit scale (natural-log units)
  float scale_log2;   // scale * log2(e): logits are kept in base 2 inside the kernels
  int win_frames;     // frames per K/V buffer window (0: corners are read with global loads)
};

// Frames of a K/V buffer window: a structured buffer addresses < 4 GB from its base and its
// record stride (the rows of all heads of one token) must fit the descriptor's 14-bit field.
int window_frames(const Geometry& g, int row_bytes);

// All launches return the hipError_t of the launch itself.
// logits != null: the predicted-weights variant (q and k are not read; pass valid pointers).
hipError_t launch_forward(const Geometry& g, bool bf16, const void* q, const void* k,
                          const void* v, const float* logits, const float* offsets, void* out,
                          float* lse, hipStream_t stream);

// Device workspace (bytes) the backward needs for this geometry.
size_t backward_workspace_bytes(const Geometry& g);

// logits != null: the predicted-weights variant (q, k, dq, dk are not used; pass valid
// pointers for q and k; dlogits receives alpha_p (da_p - Delta)).
hipError_t launch_backward(const Geometry& g, bool bf16, const void* q, const void* k,
                           const void* v, const float* logits, const float* offsets,
                           const float* lse, const void* dout, float* dq, float* dk, float* dv,
                           float* d_offsets, float* dlogits, void* workspace, hipStream_t stream,
                           hipEvent_t const* events);

// ---------------------------------------------------------------------------- depthwise conv

// Depthwise 3D convolution geometry (validated on the host; filled by conv_plan).
struct ConvGeometry {
  int B, T, H, W, C;         // batch, frames, height, width, channels
  int bf16;                  // storage of x, y and dy (set before conv_plan)
  int stream;                // the time-streaming kernels apply (set by conv_plan)
  int kt, kh, kw, taps;      // odd filter size and its tap count
  int chunks;                // 128-channel chunks
  int strips, sg, hq;        // 8-token strips along x, strips per brick, 4-row quads along y
  int tiles_per_bc;          // tiles per (channel chunk, batch item), brick padding included
  int wg_blocks;             // weight-gradient blocks per (channel chunk, filter plane)
};

void conv_plan(ConvGeometry& g);
size_t conv_workspace_bytes(const ConvGeometry& g);
hipError_t launch_conv_forward(const ConvGeometry& g, bool bf16, const void* x, const float* w,
                               const float* bias, void* y, int accumulate, hipStream_t stream);
hipError_t launch_conv_backward(const ConvGeometry& g, bool bf16, const void* x, const float* w,
                                const void* dy, float* dx, int accumulate_dx, float* dw, float* db,
                                void* workspace, hipStream_t stream);

// ---------------------------------------------------------------------------- window attention

// Shifted-window attention geometry (validated on the host; filled by win_plan).  Along each
// axis the cut points of the box partition are off + n * window (off = shift - window for a
// non-zero shift, else 0), clipped to the grid.
struct WinGeometry {
  int B, T, H, W, heads, D;
  int wt, wh, ww;            // window
  int off_t, off_h, off_w;   // first cut point minus one window
  int nt, nh, nw, boxes;     // boxes per axis and in all
  int max_box;               // largest box volume
  int qtiles;                // query tiles of the largest box
  int groups;                // (batch, box, head) groups, B * boxes * heads
  int N;                     // tokens per batch item
  float scale, scale_log2;   // logit scale (natural-log units) and scale * log2(e)
};

// Fills the cut points, box counts and launch sizes from B..D, the window and the shifts.
void win_plan(WinGeometry& g, int st, int sh, int sw);
int64_t win_forward_blocks(const WinGeometry& g);
// out_res may be null (not written / not read).
hipError_t launch_win_forward(const WinGeometry& g, const void* q, const void* k, const void* v,
                              void* out, void* out_res, float* lse, hipStream_t stream);
hipError_t launch_win_backward(const WinGeometry& g, const void* q, const void* k, const void* v,
                               const void* out, const void* out_res, const float* lse,
                               const void* dout, float* dq, float* dk, float* dv,
                               void* workspace, hipStream_t stream, hipEvent_t const* events);

}  // namespace dsa3d
