/*
 * Depthwise 3D convolution of 3D Deformable Slide Attention, C ABI (gfx950 HIP kernels).
 *
 * The first term of MegaSlide-DiT's Eq. (1) (Section 5.2) adds a depthwise 3D convolution of
 * the activation to the attention output, and the offset network that predicts the sampling
 * offsets starts with depthwise 3D convolutions (Section 5.3: nn.Conv3d with groups equal to
 * the channel count).  This is that operation, forward and backward:
 *
 *   y[b,t,i,j,c] = bias[c] + sum_(a,e,f) w[c][a][e][f] * x[b, t+a-rt, i+e-rh, j+f-rw, c]
 *
 * (a cross-correlation over the kt x kh x kw neighbourhood, rt = (kt-1)/2 and so on, with x
 * read as zero outside the grid: nn.Conv3d with padding (rt, rh, rw) and groups = C).
 *
 * Conventions are those of dsa3d.h: plain device pointers, work enqueued on `stream`, host
 * validation first (on any error nothing is enqueued and no output is touched), no
 * allocation, no synchronisation.
 *
 * Layouts (contiguous, row-major):
 *   x, y, dy      [B][T][H][W][C]   descriptor dtype (fp32, or bf16 bit patterns)
 *   weight, dw    [C][kt][kh][kw]   float32 (nn.Conv3d's [C][1][kt][kh][kw] without the 1)
 *   bias, dbias   [C]               float32
 *   dx            [B][T][H][W][C]   float32
 * With C the full channel count (heads x head_dim of the attention), y is laid out like the
 * attention output, so the Eq. (1) sum is dsa3d_forward followed by this call with
 * accumulate = 1 on the same buffer.
 */
#ifndef DSA3D_DWCONV_H
#define DSA3D_DWCONV_H

#include <stddef.h>
#include <stdint.h>

#include "dsa3d.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Largest kt * kh * kw supported (the filter taps of a 128-channel chunk live in 64 KB of
 * LDS); kh and kw must each be 1, 3, 5 or 7, kt any odd value. */
#define DSA3D_DWCONV_MAX_TAPS 128

typedef struct {
  int32_t batch, frames, height, width; /* B, T, H', W' */
  int32_t channels;                     /* C, even */
  int32_t kt, kh, kw;                   /* odd filter size */
  dsa3d_dtype dtype;                    /* storage of x, y and dy */
} dsa3d_dwconv_desc;

/* y = conv(x) + bias (bias may be NULL), or y += conv(x) + bias when accumulate != 0 (y is
 * read first; with bf16 storage the sum is rounded once to bf16).  fp32 accumulation, the
 * bf16 output rounded to nearest even.  Errors: NULL x, weight or y -> DSA3D_ERR_NULL_POINTER;
 * a dimension < 1, an even filter size, odd C, B*T*H*W of 2^31 or more, C of 2^24 or more,
 * or 2^31 or more work tiles (tiles of 4 rows x 8 tokens x 128 channels, about
 * B*T*H*W*C/4096) -> DSA3D_ERR_INVALID_SHAPE; kh or kw not in {1,3,5,7}, more than DSA3D_DWCONV_MAX_TAPS taps
 * or an unknown dtype -> DSA3D_ERR_UNSUPPORTED; x or y not aligned to one channel pair
 * (4 bytes bf16, 8 fp32), weight or bias not 4-byte aligned -> DSA3D_ERR_MISALIGNED; y
 * overlapping x, weight or bias -> DSA3D_ERR_ALIAS. */
dsa3d_status dsa3d_dwconv3d_forward(const dsa3d_dwconv_desc* desc, const void* x,
                                    const float* weight, const float* bias, void* y,
                                    int accumulate, hipStream_t stream);

/* Bytes of device workspace dsa3d_dwconv3d_backward needs for the weight and bias gradients
 * (partial sums of the grid sweep: 4 bytes per channel and tap, and per channel, for each of
 * about 3072 / (ceil(C/128) kt) wave slots, a few MB); 0 for a descriptor the backward would
 * reject. */
size_t dsa3d_dwconv3d_backward_workspace_size(const dsa3d_dwconv_desc* desc);

/* Backward of dsa3d_dwconv3d_forward for upstream gradient dy:
 *   dx[b,t,i,j,c]  = sum_(a,e,f) w[c][a][e][f] * dy[b, t-a+rt, i-e+rh, j-f+rw, c]
 *   dw[c][a][e][f] = sum over the grid of dy[b,t,i,j,c] * x[b, t+a-rt, i+e-rh, j+f-rw, c]
 *   dbias[c]       = sum over the grid of dy[b,t,i,j,c]
 * Each of dx, dweight and dbias may be NULL (not computed); dx is overwritten, or added to
 * when accumulate_dx != 0 (so the other uses of x can be summed into one buffer); dweight and
 * dbias are overwritten, summed in a fixed order (bitwise repeatable).  The workspace (at
 * least dsa3d_dwconv3d_backward_workspace_size bytes, 256-byte aligned) is needed only when
 * dweight or dbias is requested.  Errors as for the forward, plus: dy NULL or all three
 * outputs NULL -> DSA3D_ERR_NULL_POINTER; workspace missing or too small ->
 * DSA3D_ERR_WORKSPACE; outputs overlapping each other, an input or the workspace ->
 * DSA3D_ERR_ALIAS. */
dsa3d_status dsa3d_dwconv3d_backward(const dsa3d_dwconv_desc* desc, const void* x,
                                     const float* weight, const void* dy, float* dx,
                                     int accumulate_dx, float* dweight, float* dbias,
                                     void* workspace, size_t workspace_bytes, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* DSA3D_DWCONV_H */
