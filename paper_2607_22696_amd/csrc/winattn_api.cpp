// C-ABI entry points of the shifted-window attention: argument validation and dispatch.
// The operation and the conventions are described in include/dsa3d_win.h.
#include "dsa3d_win.h"

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>

#include "api_util.h"
#include "dsa3d_internal.h"

namespace {

using dsa3d::api::aligned;
using dsa3d::api::overlaps;
using dsa3d::api::Span;
using dsa3d::api::span_of;

// Checks the descriptor and fills the geometry, the row count and the byte size of q.
dsa3d_status check_win(const dsa3d_win_desc* d, dsa3d::WinGeometry* g, uint64_t* rows,
                       uint64_t* io_bytes) {
  if (d == nullptr) return DSA3D_ERR_NULL_POINTER;
  const int32_t dims[] = {d->batch, d->frames, d->height, d->width, d->heads, d->head_dim,
                          d->wt,    d->wh,     d->ww};
  for (int32_t v : dims)
    if (v < 1) return DSA3D_ERR_INVALID_SHAPE;
  if (d->st < 0 || d->sh < 0 || d->sw < 0 || d->st >= d->wt || d->sh >= d->wh || d->sw >= d->ww)
    return DSA3D_ERR_INVALID_SHAPE;
  if (!std::isfinite(d->scale) || d->scale < 0.0f) return DSA3D_ERR_INVALID_SHAPE;
  if (d->frames >= (1 << 24) || d->height >= (1 << 24) || d->width >= (1 << 24))
    return DSA3D_ERR_INVALID_SHAPE;
  const uint64_t r = (uint64_t)d->batch * d->frames * d->height * d->width * d->heads;
  if (r >= (1ull << 31)) return DSA3D_ERR_INVALID_SHAPE;
  if ((uint64_t)d->wt * d->wh * d->ww > DSA3D_WIN_MAX_TOKENS) return DSA3D_ERR_INVALID_SHAPE;
  if (d->dtype != DSA3D_BF16) return DSA3D_ERR_UNSUPPORTED;
  if (d->head_dim != 64 && d->head_dim != 128) return DSA3D_ERR_UNSUPPORTED;
  g->B = d->batch;
  g->T = d->frames;
  g->H = d->height;
  g->W = d->width;
  g->heads = d->heads;
  g->D = d->head_dim;
  g->wt = d->wt;
  g->wh = d->wh;
  g->ww = d->ww;
  g->scale = d->scale != 0.0f ? d->scale : 1.0f / std::sqrt((float)d->head_dim);
  g->scale_log2 = g->scale * 1.4426950408889634f;
  dsa3d::win_plan(*g, d->st, d->sh, d->sw);
  if (dsa3d::win_forward_blocks(*g) >= (1ll << 31)) return DSA3D_ERR_INVALID_SHAPE;
  *rows = r;
  *io_bytes = r * d->head_dim * 2;
  return DSA3D_OK;
}

uint64_t workspace_need(uint64_t rows) { return (rows * 4 + 255) & ~uint64_t(255); }

}  // namespace

extern "C" {

dsa3d_status dsa3d_win_forward(const dsa3d_win_desc* desc, const void* q, const void* k,
                               const void* v, void* out, void* out_res, float* lse,
                               hipStream_t stream) {
  dsa3d::WinGeometry g;
  uint64_t rows, io_bytes;
  const dsa3d_status st = check_win(desc, &g, &rows, &io_bytes);
  if (st != DSA3D_OK) return st;
  if (!q || !k || !v || !out) return DSA3D_ERR_NULL_POINTER;
  if (!aligned(q, 16) || !aligned(k, 16) || !aligned(v, 16) || !aligned(out, 16) ||
      (out_res && !aligned(out_res, 16)) || (lse && !aligned(lse, 4)))
    return DSA3D_ERR_MISALIGNED;
  const Span in[] = {span_of(q, io_bytes), span_of(k, io_bytes), span_of(v, io_bytes)};
  const Span outs[] = {span_of(out, io_bytes), span_of(out_res, out_res ? io_bytes : 0),
                       span_of(lse, lse ? rows * 4 : 0)};
  for (int a = 0; a < 3; ++a) {
    for (const Span& s : in)
      if (overlaps(outs[a], s)) return DSA3D_ERR_ALIAS;
    for (int b = a + 1; b < 3; ++b)
      if (overlaps(outs[a], outs[b])) return DSA3D_ERR_ALIAS;
  }
  const hipError_t e = dsa3d::launch_win_forward(g, q, k, v, out, out_res, lse,
                                                 stream);
  return e == hipSuccess ? DSA3D_OK : DSA3D_ERR_DEVICE;
}

size_t dsa3d_win_backward_workspace_size(const dsa3d_win_desc* desc) {
  dsa3d::WinGeometry g;
  uint64_t rows, io_bytes;
  if (check_win(desc, &g, &rows, &io_bytes) != DSA3D_OK) return 0;
  return workspace_need(rows);
}

dsa3d_status dsa3d_win_backward(const dsa3d_win_desc* desc, const void* q, const void* k,
                                const void* v, const void* out, const void* out_res,
                                const float* lse, const void* dout, float* dq, float* dk, float* dv,
                                void* workspace, size_t workspace_bytes, hipStream_t stream,
                                const hipEvent_t* events) {
  dsa3d::WinGeometry g;
  uint64_t rows, io_bytes;
  const dsa3d_status st = check_win(desc, &g, &rows, &io_bytes);
  if (st != DSA3D_OK) return st;
  if (!q || !k || !v || !out || !lse || !dout || !dq || !dk || !dv)
    return DSA3D_ERR_NULL_POINTER;
  const uint64_t ws_need = workspace_need(rows);
  if (workspace == nullptr || workspace_bytes < ws_need) return DSA3D_ERR_WORKSPACE;
  if (!aligned(q, 16) || !aligned(k, 16) || !aligned(v, 16) || !aligned(out, 16) ||
      (out_res && !aligned(out_res, 16)) || !aligned(dout, 16) || !aligned(lse, 4) ||
      !aligned(dq, 16) || !aligned(dk, 16) || !aligned(dv, 16) || !aligned(workspace, 256))
    return DSA3D_ERR_MISALIGNED;
  const uint64_t f32_bytes = io_bytes * 2;
  const Span in[] = {span_of(q, io_bytes),    span_of(k, io_bytes),
                     span_of(v, io_bytes),    span_of(out, io_bytes),
                     span_of(dout, io_bytes), span_of(lse, rows * 4),
                     span_of(out_res, out_res ? io_bytes : 0)};
  const Span outs[] = {span_of(dq, f32_bytes), span_of(dk, f32_bytes), span_of(dv, f32_bytes),
                       span_of(workspace, ws_need)};
  for (int a = 0; a < 4; ++a) {
    for (const Span& s : in)
      if (overlaps(outs[a], s)) return DSA3D_ERR_ALIAS;
    for (int b = a + 1; b < 4; ++b)
      if (overlaps(outs[a], outs[b])) return DSA3D_ERR_ALIAS;
  }
  const hipError_t e = dsa3d::launch_win_backward(
      g, q, k, v, out, out_res, lse, dout, dq, dk, dv, workspace, stream,
      events);
  return e == hipSuccess ? DSA3D_OK : DSA3D_ERR_DEVICE;
}

}  // extern "C"
