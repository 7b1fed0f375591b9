// C-ABI entry points of the depthwise 3D convolution: argument validation and dispatch.
// The operation and the conventions are described in include/dsa3d_dwconv.h.
#include "dsa3d_dwconv.h"

#include <hip/hip_runtime.h>

#include <cstdint>

#include "api_util.h"
#include "dsa3d_internal.h"

namespace {

using dsa3d::api::aligned;
using dsa3d::api::overlaps;
using dsa3d::api::Span;
using dsa3d::api::span_of;

bool kernel_width_ok(int32_t k) { return k == 1 || k == 3 || k == 5 || k == 7; }

// Checks the descriptor, fills the geometry and the byte size of x (= y = dy) and of dx.
dsa3d_status check_conv(const dsa3d_dwconv_desc* d, dsa3d::ConvGeometry* g, uint64_t* io_bytes,
                        uint64_t* f32_bytes) {
  if (d == nullptr) return DSA3D_ERR_NULL_POINTER;
  const int32_t dims[] = {d->batch, d->frames, d->height, d->width, d->channels, d->kt, d->kh,
                          d->kw};
  for (int32_t v : dims)
    if (v < 1) return DSA3D_ERR_INVALID_SHAPE;
  if (d->kt % 2 == 0 || d->kh % 2 == 0 || d->kw % 2 == 0 || d->channels % 2 != 0)
    return DSA3D_ERR_INVALID_SHAPE;
  const uint64_t tokens = (uint64_t)d->batch * d->frames * d->height * d->width;
  if (tokens >= (1ull << 31) || d->channels >= (1 << 24)) return DSA3D_ERR_INVALID_SHAPE;
  // tiles of 4 rows x 8 tokens, bricks of up to 5 tiles along x, per 128-channel chunk
  const uint64_t chunks = ((uint64_t)d->channels + 127) / 128;
  const uint64_t strips = ((uint64_t)d->width + 7) / 8, sg = strips < 5 ? strips : 5;
  const uint64_t tiles = chunks * d->batch * ((strips + sg - 1) / sg) * sg * d->frames *
                         (((uint64_t)d->height + 3) / 4);
  if (tiles >= (1ull << 31)) return DSA3D_ERR_INVALID_SHAPE;
  if (d->dtype != DSA3D_F32 && d->dtype != DSA3D_BF16) return DSA3D_ERR_UNSUPPORTED;
  if (!kernel_width_ok(d->kh) || !kernel_width_ok(d->kw)) return DSA3D_ERR_UNSUPPORTED;
  if ((uint64_t)d->kt * d->kh * d->kw > DSA3D_DWCONV_MAX_TAPS) return DSA3D_ERR_UNSUPPORTED;
  g->B = d->batch;
  g->T = d->frames;
  g->H = d->height;
  g->W = d->width;
  g->C = d->channels;
  g->kt = d->kt;
  g->kh = d->kh;
  g->kw = d->kw;
  g->bf16 = d->dtype == DSA3D_BF16;
  dsa3d::conv_plan(*g);
  *io_bytes = tokens * d->channels * (d->dtype == DSA3D_BF16 ? 2 : 4);
  *f32_bytes = tokens * d->channels * 4;
  return DSA3D_OK;
}

}  // namespace

extern "C" {

dsa3d_status dsa3d_dwconv3d_forward(const dsa3d_dwconv_desc* desc, const void* x,
                                    const float* weight, const float* bias, void* y,
                                    int accumulate, hipStream_t stream) {
  dsa3d::ConvGeometry g;
  uint64_t io_bytes, f32_bytes;
  const dsa3d_status st = check_conv(desc, &g, &io_bytes, &f32_bytes);
  if (st != DSA3D_OK) return st;
  if (!x || !weight || !y) return DSA3D_ERR_NULL_POINTER;
  const uintptr_t pair = desc->dtype == DSA3D_BF16 ? 4 : 8;
  if (!aligned(x, pair) || !aligned(y, pair) || !aligned(weight, 4) || (bias && !aligned(bias, 4)))
    return DSA3D_ERR_MISALIGNED;
  const Span sy = span_of(y, io_bytes);
  if (overlaps(sy, span_of(x, io_bytes)) ||
      overlaps(sy, span_of(weight, (uint64_t)g.C * g.taps * 4)) ||
      (bias && overlaps(sy, span_of(bias, (uint64_t)g.C * 4))))
    return DSA3D_ERR_ALIAS;
  const hipError_t e = dsa3d::launch_conv_forward(g, desc->dtype == DSA3D_BF16, x, weight, bias, y,
                                                  accumulate != 0, stream);
  return e == hipSuccess ? DSA3D_OK : DSA3D_ERR_DEVICE;
}

size_t dsa3d_dwconv3d_backward_workspace_size(const dsa3d_dwconv_desc* desc) {
  dsa3d::ConvGeometry g;
  uint64_t io_bytes, f32_bytes;
  if (check_conv(desc, &g, &io_bytes, &f32_bytes) != DSA3D_OK) return 0;
  return dsa3d::conv_workspace_bytes(g);
}

dsa3d_status dsa3d_dwconv3d_backward(const dsa3d_dwconv_desc* desc, const void* x,
                                     const float* weight, const void* dy, float* dx,
                                     int accumulate_dx, float* dweight, float* dbias,
                                     void* workspace, size_t workspace_bytes, hipStream_t stream) {
  dsa3d::ConvGeometry g;
  uint64_t io_bytes, f32_bytes;
  const dsa3d_status st = check_conv(desc, &g, &io_bytes, &f32_bytes);
  if (st != DSA3D_OK) return st;
  if (!x || !weight || !dy) return DSA3D_ERR_NULL_POINTER;
  if (!dx && !dweight && !dbias) return DSA3D_ERR_NULL_POINTER;
  const bool wgrad = dweight != nullptr || dbias != nullptr;
  const size_t ws_need = dsa3d::conv_workspace_bytes(g);
  if (wgrad && (workspace == nullptr || workspace_bytes < ws_need)) return DSA3D_ERR_WORKSPACE;
  const uintptr_t pair = desc->dtype == DSA3D_BF16 ? 4 : 8;
  if (!aligned(x, pair) || !aligned(dy, pair) || !aligned(weight, 4) || (dx && !aligned(dx, 8)) ||
      (dweight && !aligned(dweight, 4)) || (dbias && !aligned(dbias, 4)) ||
      (wgrad && !aligned(workspace, 256)))
    return DSA3D_ERR_MISALIGNED;
  const uint64_t wbytes = (uint64_t)g.C * g.taps * 4, bbytes = (uint64_t)g.C * 4;
  const Span in[] = {span_of(x, io_bytes), span_of(weight, wbytes), span_of(dy, io_bytes)};
  Span outs[4];
  int n = 0;
  if (dx) outs[n++] = span_of(dx, f32_bytes);
  if (dweight) outs[n++] = span_of(dweight, wbytes);
  if (dbias) outs[n++] = span_of(dbias, bbytes);
  if (wgrad) outs[n++] = span_of(workspace, ws_need);
  for (int a = 0; a < n; ++a) {
    for (const Span& s : in)
      if (overlaps(outs[a], s)) return DSA3D_ERR_ALIAS;
    for (int b = a + 1; b < n; ++b)
      if (overlaps(outs[a], outs[b])) return DSA3D_ERR_ALIAS;
  }
  const hipError_t e = dsa3d::launch_conv_backward(
      g, desc->dtype == DSA3D_BF16, x, weight, dy, dx, accumulate_dx != 0, dweight, dbias,
      workspace, stream);
  return e == hipSuccess ? DSA3D_OK : DSA3D_ERR_DEVICE;
}

}  // extern "C"
