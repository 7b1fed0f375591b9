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
hipError_t launch_forward(const Geometry& g, bool bf16, const void* q, const void* k,
                          const void* v, const float* offsets, void* out, float* lse,
                          hipStream_t stream);

// Device workspace (bytes) the backward needs for this geometry.
size_t backward_workspace_bytes(const Geometry& g);

hipError_t launch_backward(const Geometry& g, bool bf16, const void* q, const void* k,
                           const void* v, const float* offsets, const float* lse, const void* dout,
                           float* dq, float* dk, float* dv, float* d_offsets, void* workspace,
                           hipStream_t stream, hipEvent_t const* events);

}  // namespace dsa3d
