// C-ABI entry points of the 3D-DSA library: argument validation and kernel dispatch.
// The operator and the conventions are described in include/dsa3d.h.
#include "dsa3d.h"
#include "dsa3d_pw.h"

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>

#include "api_util.h"
#include "backward_entry.h"
#include "dsa3d_internal.h"

namespace {

using dsa3d::api::aligned;
using dsa3d::api::overlaps;
using dsa3d::api::Span;
using dsa3d::api::span_of;

// Checks the descriptor and fills the kernel geometry and the tensor sizes.
dsa3d_status check_desc(const dsa3d_desc* d, dsa3d::Geometry* g, uint64_t* rows, uint64_t* io_bytes,
                        uint64_t* f32_bytes, uint64_t* off_bytes) {
  if (d == nullptr) return DSA3D_ERR_NULL_POINTER;
  const int32_t dims[] = {d->batch, d->frames, d->height, d->width, d->heads, d->head_dim,
                          d->kt, d->kh, d->kw};
  for (int32_t x : dims)
    if (x < 1) return DSA3D_ERR_INVALID_SHAPE;
  if (d->kt % 2 == 0 || d->kh % 2 == 0 || d->kw % 2 == 0) return DSA3D_ERR_INVALID_SHAPE;
  if (!std::isfinite(d->scale)) return DSA3D_ERR_INVALID_SHAPE;
  // token coordinates must be exact in fp32
  if (d->frames >= (1 << 24) || d->height >= (1 << 24) || d->width >= (1 << 24))
    return DSA3D_ERR_INVALID_SHAPE;
  const uint64_t N = (uint64_t)d->frames * d->height * d->width;
  const uint64_t R = N * d->batch * d->heads;
  if (N >= (1ull << 31) || R >= (1ull << 31)) return DSA3D_ERR_INVALID_SHAPE;
  const uint64_t P = (uint64_t)d->kt * d->kh * d->kw;
  if (d->dtype != DSA3D_F32 && d->dtype != DSA3D_BF16) return DSA3D_ERR_UNSUPPORTED;
  if (d->head_dim != 32 && d->head_dim != 64 && d->head_dim != 128) return DSA3D_ERR_UNSUPPORTED;
  if (P > DSA3D_MAX_POINTS) return DSA3D_ERR_UNSUPPORTED;
  const uint64_t esz = d->dtype == DSA3D_BF16 ? 2 : 4;
  g->B = d->batch;
  g->T = d->frames;
  g->H = d->height;
  g->W = d->width;
  g->heads = d->heads;
  g->D = d->head_dim;
  g->kt = d->kt;
  g->kh = d->kh;
  g->kw = d->kw;
  g->P = (int)P;
  g->N = (int)N;
  g->scale = d->scale != 0.0f ? d->scale : 1.0f / std::sqrt((float)d->head_dim);
  g->scale_log2 = g->scale * 1.4426950408889634f;
  g->win_frames = dsa3d::window_frames(*g, (int)(d->head_dim * esz));
  *rows = R;
  *io_bytes = R * d->head_dim * esz;
  *f32_bytes = R * d->head_dim * 4;
  *off_bytes = R * P * 3 * 4;
  return DSA3D_OK;
}

}  // namespace

namespace dsa3d {

int window_frames(const Geometry& g, int row_bytes) {
  const uint64_t stride = (uint64_t)g.heads * row_bytes;
  if (stride > 16383) return 0;  // the record stride field is 14 bits wide
  const uint64_t frame_bytes = (uint64_t)g.H * g.W * stride;
  const uint64_t frames = ((1ull << 32) - 4096) / frame_bytes;
  return (int)(frames < (uint64_t)g.T ? frames : (uint64_t)g.T);
}

// The backward bins every (query row, point) pair by its trilinear cell; bin ranks and entry
// slots are 32-bit, so rows * P and the number of cells must stay below 2^31.
static dsa3d_status check_backward_range(const dsa3d::Geometry& g, uint64_t rows) {
  const uint64_t cells = (uint64_t)(g.T + 1) * (g.H + 1) * (g.W + 1) * g.B * g.heads;
  if (rows * (uint64_t)g.P >= (1ull << 31) || cells >= (1ull << 31)) return DSA3D_ERR_INVALID_SHAPE;
  return DSA3D_OK;
}

dsa3d_status check_backward_call(const dsa3d_desc* desc, const BackwardArgs& a,
                                 const void* workspace, size_t workspace_bytes,
                                 size_t scratch_limit, Geometry* gp) {
  Geometry& g = *gp;
  uint64_t rows, io_bytes, f32_bytes, off_bytes;
  dsa3d_status st = check_desc(desc, &g, &rows, &io_bytes, &f32_bytes, &off_bytes);
  if (st != DSA3D_OK) return st;
  if (!a.q || !a.k || !a.v || !a.offsets || !a.lse || !a.dout || !a.dq || !a.dk || !a.dv ||
      !a.d_offsets)
    return DSA3D_ERR_NULL_POINTER;
  st = check_backward_range(g, rows);
  if (st != DSA3D_OK) return st;
  const size_t ws_need = backward_workspace_bytes(g);
  if (scratch_limit > 0) {
    if (ws_need > scratch_limit) return DSA3D_ERR_SCRATCH;
  } else {
    if (workspace == nullptr || workspace_bytes < ws_need) return DSA3D_ERR_WORKSPACE;
    if (!aligned(workspace, 256)) return DSA3D_ERR_MISALIGNED;
  }
  if (!aligned(a.q, 16) || !aligned(a.k, 16) || !aligned(a.v, 16) || !aligned(a.dout, 16) ||
      !aligned(a.dq, 16) || !aligned(a.dk, 16) || !aligned(a.dv, 16) ||
      (a.out && !aligned(a.out, 16)) || !aligned(a.offsets, 4) || !aligned(a.lse, 4) ||
      !aligned(a.d_offsets, 4))
    return DSA3D_ERR_MISALIGNED;
  // out (optional, not read) counts as an input: outputs and the workspace must avoid it
  const Span in[] = {span_of(a.q, io_bytes),       span_of(a.k, io_bytes),
                     span_of(a.v, io_bytes),       span_of(a.offsets, off_bytes),
                     span_of(a.lse, rows * 4),     span_of(a.dout, io_bytes),
                     span_of(a.out, a.out ? io_bytes : 0)};
  const Span outs[] = {span_of(a.dq, f32_bytes), span_of(a.dk, f32_bytes),
                       span_of(a.dv, f32_bytes), span_of(a.d_offsets, off_bytes)};
  // the library's own scratch is a separate allocation: it overlaps nothing of the caller's
  const Span sw = span_of(scratch_limit > 0 ? nullptr : workspace, scratch_limit > 0 ? 0 : ws_need);
  for (int i = 0; i < 4; ++i) {
    for (const Span& s : in)
      if (overlaps(outs[i], s)) return DSA3D_ERR_ALIAS;
    for (int j = i + 1; j < 4; ++j)
      if (overlaps(outs[i], outs[j])) return DSA3D_ERR_ALIAS;
    if (overlaps(outs[i], sw)) return DSA3D_ERR_ALIAS;
  }
  for (const Span& s : in)
    if (overlaps(sw, s)) return DSA3D_ERR_ALIAS;
  return DSA3D_OK;
}

}  // namespace dsa3d

extern "C" {

int dsa3d_abi_version(void) { return 1; }

const char* dsa3d_status_string(dsa3d_status s) {
  switch (s) {
    case DSA3D_OK:
      return "ok";
    case DSA3D_ERR_NULL_POINTER:
      return "a required pointer is NULL";
    case DSA3D_ERR_INVALID_SHAPE:
      return "invalid problem shape or scale";
    case DSA3D_ERR_UNSUPPORTED:
      return "unsupported dtype, head_dim or neighbourhood size";
    case DSA3D_ERR_MISALIGNED:
      return "misaligned pointer";
    case DSA3D_ERR_WORKSPACE:
      return "workspace too small";
    case DSA3D_ERR_ALIAS:
      return "an output overlaps another argument";
    case DSA3D_ERR_DEVICE:
      return "HIP launch failed";
    case DSA3D_ERR_SCRATCH:
      return "problem needs more workspace than the library's fixed scratch buffer";
  }
  return "unknown status";
}

dsa3d_status dsa3d_forward(const dsa3d_desc* desc, const void* q, const void* k, const void* v,
                           const float* offsets, void* out, float* lse, hipStream_t stream) {
  dsa3d::Geometry g;
  uint64_t rows, io_bytes, f32_bytes, off_bytes;
  dsa3d_status st = check_desc(desc, &g, &rows, &io_bytes, &f32_bytes, &off_bytes);
  if (st != DSA3D_OK) return st;
  if (!q || !k || !v || !offsets || !out) return DSA3D_ERR_NULL_POINTER;
  if (!aligned(q, 16) || !aligned(k, 16) || !aligned(v, 16) || !aligned(out, 16) ||
      !aligned(offsets, 4) || (lse && !aligned(lse, 4)))
    return DSA3D_ERR_MISALIGNED;
  const Span in[] = {span_of(q, io_bytes), span_of(k, io_bytes), span_of(v, io_bytes),
                     span_of(offsets, off_bytes)};
  const Span so = span_of(out, io_bytes);
  for (const Span& s : in)
    if (overlaps(so, s)) return DSA3D_ERR_ALIAS;
  if (lse) {
    const Span sl = span_of(lse, rows * 4);
    if (overlaps(sl, so)) return DSA3D_ERR_ALIAS;
    for (const Span& s : in)
      if (overlaps(sl, s)) return DSA3D_ERR_ALIAS;
  }
  const hipError_t e = dsa3d::launch_forward(g, desc->dtype == DSA3D_BF16, q, k, v, nullptr,
                                             offsets, out, lse, stream);
  return e == hipSuccess ? DSA3D_OK : DSA3D_ERR_DEVICE;
}

size_t dsa3d_backward_workspace_size(const dsa3d_desc* desc) {
  dsa3d::Geometry g;
  uint64_t rows, io_bytes, f32_bytes, off_bytes;
  if (check_desc(desc, &g, &rows, &io_bytes, &f32_bytes, &off_bytes) != DSA3D_OK) return 0;
  if (dsa3d::check_backward_range(g, rows) != DSA3D_OK) return 0;
  return dsa3d::backward_workspace_bytes(g);
}

dsa3d_status dsa3d_backward_timed(const dsa3d_desc* desc, const void* q, const void* k,
                                  const void* v, const float* offsets, const void* out,
                                  const float* lse, const void* dout, float* dq, float* dk,
                                  float* dv, float* d_offsets, void* workspace,
                                  size_t workspace_bytes, hipStream_t stream,
                                  const hipEvent_t* events) {
  const dsa3d::BackwardArgs a{q, k, v, offsets, out, lse, dout, dq, dk, dv, d_offsets};
  dsa3d::Geometry g;
  const dsa3d_status st = dsa3d::check_backward_call(desc, a, workspace, workspace_bytes, 0, &g);
  if (st != DSA3D_OK) return st;
  const hipError_t e = dsa3d::launch_backward(g, desc->dtype == DSA3D_BF16, q, k, v, nullptr,
                                              offsets, lse, dout, dq, dk, dv, d_offsets, nullptr,
                                              workspace, stream, events);
  return e == hipSuccess ? DSA3D_OK : DSA3D_ERR_DEVICE;
}

dsa3d_status dsa3d_backward(const dsa3d_desc* desc, const void* q, const void* k, const void* v,
                            const float* offsets, const void* out, const float* lse,
                            const void* dout, float* dq, float* dk, float* dv, float* d_offsets,
                            void* workspace, size_t workspace_bytes, hipStream_t stream) {
  return dsa3d_backward_timed(desc, q, k, v, offsets, out, lse, dout, dq, dk, dv, d_offsets,
                              workspace, workspace_bytes, stream, nullptr);
}

// ---------------------------------------------------------------------------- predicted weights

// The variant takes its logits as given: a descriptor scale other than 0 or 1 is rejected.
static dsa3d_status check_pw(const dsa3d_desc* desc, dsa3d::Geometry* g, uint64_t* rows,
                             uint64_t* io_bytes, uint64_t* f32_bytes, uint64_t* off_bytes,
                             uint64_t* logit_bytes) {
  const dsa3d_status st = check_desc(desc, g, rows, io_bytes, f32_bytes, off_bytes);
  if (st != DSA3D_OK) return st;
  if (desc->scale != 0.0f && desc->scale != 1.0f) return DSA3D_ERR_INVALID_SHAPE;
  g->scale = 1.0f;
  g->scale_log2 = 1.4426950408889634f;
  *logit_bytes = *rows * g->P * 4;
  return DSA3D_OK;
}

dsa3d_status dsa3d_pw_forward(const dsa3d_desc* desc, const float* logits, const void* v,
                              const float* offsets, void* out, float* lse, hipStream_t stream) {
  dsa3d::Geometry g;
  uint64_t rows, io_bytes, f32_bytes, off_bytes, logit_bytes;
  dsa3d_status st = check_pw(desc, &g, &rows, &io_bytes, &f32_bytes, &off_bytes, &logit_bytes);
  if (st != DSA3D_OK) return st;
  if (!logits || !v || !offsets || !out) return DSA3D_ERR_NULL_POINTER;
  if (!aligned(v, 16) || !aligned(out, 16) || !aligned(logits, 4) || !aligned(offsets, 4) ||
      (lse && !aligned(lse, 4)))
    return DSA3D_ERR_MISALIGNED;
  const Span in[] = {span_of(logits, logit_bytes), span_of(v, io_bytes),
                     span_of(offsets, off_bytes)};
  const Span so = span_of(out, io_bytes);
  for (const Span& s : in)
    if (overlaps(so, s)) return DSA3D_ERR_ALIAS;
  if (lse) {
    const Span sl = span_of(lse, rows * 4);
    if (overlaps(sl, so)) return DSA3D_ERR_ALIAS;
    for (const Span& s : in)
      if (overlaps(sl, s)) return DSA3D_ERR_ALIAS;
  }
  // q and k are not read: v stands in for them so that every pointer the kernel forms is valid
  const hipError_t e = dsa3d::launch_forward(g, desc->dtype == DSA3D_BF16, v, v, v, logits,
                                             offsets, out, lse, stream);
  return e == hipSuccess ? DSA3D_OK : DSA3D_ERR_DEVICE;
}

size_t dsa3d_pw_backward_workspace_size(const dsa3d_desc* desc) {
  dsa3d::Geometry g;
  uint64_t rows, io_bytes, f32_bytes, off_bytes, logit_bytes;
  if (check_pw(desc, &g, &rows, &io_bytes, &f32_bytes, &off_bytes, &logit_bytes) != DSA3D_OK)
    return 0;
  if (dsa3d::check_backward_range(g, rows) != DSA3D_OK) return 0;
  return dsa3d::backward_workspace_bytes(g);
}

dsa3d_status dsa3d_pw_backward(const dsa3d_desc* desc, const float* logits, const void* v,
                               const float* offsets, const float* lse, const void* dout,
                               float* dlogits, float* dv, float* d_offsets, void* workspace,
                               size_t workspace_bytes, hipStream_t stream,
                               const hipEvent_t* events) {
  dsa3d::Geometry g;
  uint64_t rows, io_bytes, f32_bytes, off_bytes, logit_bytes;
  dsa3d_status st = check_pw(desc, &g, &rows, &io_bytes, &f32_bytes, &off_bytes, &logit_bytes);
  if (st != DSA3D_OK) return st;
  if (!logits || !v || !offsets || !lse || !dout || !dlogits || !dv || !d_offsets)
    return DSA3D_ERR_NULL_POINTER;
  st = dsa3d::check_backward_range(g, rows);
  if (st != DSA3D_OK) return st;
  const size_t ws_need = dsa3d::backward_workspace_bytes(g);
  if (workspace == nullptr || workspace_bytes < ws_need) return DSA3D_ERR_WORKSPACE;
  if (!aligned(workspace, 256)) return DSA3D_ERR_MISALIGNED;
  if (!aligned(v, 16) || !aligned(dout, 16) || !aligned(dv, 16) || !aligned(logits, 4) ||
      !aligned(offsets, 4) || !aligned(lse, 4) || !aligned(dlogits, 4) || !aligned(d_offsets, 4))
    return DSA3D_ERR_MISALIGNED;
  const Span in[] = {span_of(logits, logit_bytes), span_of(v, io_bytes),
                     span_of(offsets, off_bytes),  span_of(lse, rows * 4),
                     span_of(dout, io_bytes)};
  const Span outs[] = {span_of(dlogits, logit_bytes), span_of(dv, f32_bytes),
                       span_of(d_offsets, off_bytes)};
  const Span sw = span_of(workspace, ws_need);
  for (int a = 0; a < 3; ++a) {
    for (const Span& s : in)
      if (overlaps(outs[a], s)) return DSA3D_ERR_ALIAS;
    for (int b = a + 1; b < 3; ++b)
      if (overlaps(outs[a], outs[b])) return DSA3D_ERR_ALIAS;
    if (overlaps(outs[a], sw)) return DSA3D_ERR_ALIAS;
  }
  for (const Span& s : in)
    if (overlaps(sw, s)) return DSA3D_ERR_ALIAS;
  // q, k, dq and dk are not used: valid pointers stand in for them
  const hipError_t e = dsa3d::launch_backward(
      g, desc->dtype == DSA3D_BF16, dout, v, v, logits, offsets, lse, dout, dv, dv, dv, d_offsets,
      dlogits, workspace, stream, events);
  return e == hipSuccess ? DSA3D_OK : DSA3D_ERR_DEVICE;
}

}  // extern "C"
