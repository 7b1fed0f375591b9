/*
 * Fixed / shifted 3D window attention, C ABI (gfx950 HIP kernels, MFMA).
 *
 * The Swin-DiT baseline of MegaSlide-DiT (Section 6.2) replaces 3D-DSA by attention inside
 * static windows of wt x wh x ww tokens (3 x 16 x 16 there), alternating plain and shifted
 * windows between blocks as in the Swin Transformer; Section 5.1 contrasts these static
 * partitions with 3D-DSA's learned offsets.  This library computes that attention, forward
 * and backward, for projected q, k, v:
 *
 *   The grid is padded to multiples of the window, cyclically rolled by -(st, sh, sw) and cut
 *   into windows.  A query attends to the keys of its window that came from the same side of
 *   every wrap-around seam of the roll and that are real tokens (padding positions are
 *   neither keys nor queries):
 *     s = scale <q, k>,  alpha = softmax over those keys,  out = sum alpha v,
 *     lse = logsumexp of s over those keys.
 *   Equivalently, along each axis the cut points are st + n wt for integers n (plus the grid
 *   ends), and every box of the resulting partition of the T x H' x W' grid attends densely
 *   within itself.  A zero shift gives plain windows; a shift of half the window gives
 *   Swin's shifted windows.  No causal mask.
 *
 * Conventions are those of dsa3d.h (plain device pointers, work enqueued on `stream`, host
 * validation first, no allocation, no synchronisation).  Built for bf16 storage (the MFMA
 * path) with fp32 accumulation.
 *
 * Layouts (contiguous, row-major, 16-byte aligned):
 *   q, k, v, out, dout   [B][T][H][W][heads][head_dim]   bf16 bit patterns
 *   out_res              [B][T][H][W][heads][head_dim]   bf16 bit patterns
 *   lse                  [B][T][H][W][heads]             float32 (4-byte aligned)
 *   dq, dk, dv           [B][T][H][W][heads][head_dim]   float32
 */
#ifndef DSA3D_WIN_H
#define DSA3D_WIN_H

#include <stddef.h>
#include <stdint.h>

#include "dsa3d.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Largest window volume wt * wh * ww accepted. */
#define DSA3D_WIN_MAX_TOKENS 65536

typedef struct {
  int32_t batch, frames, height, width; /* B, T, H', W'                                   */
  int32_t heads, head_dim;              /* head_dim 64 or 128                             */
  int32_t wt, wh, ww;                   /* window (the paper's Swin-DiT: 3 x 16 x 16)     */
  int32_t st, sh, sw;                   /* cyclic shift, 0 <= shift < window on each axis */
  float scale;                          /* logit scale > 0; 0 selects 1/sqrt(head_dim)   */
  dsa3d_dtype dtype;                    /* DSA3D_BF16                                     */
} dsa3d_win_desc;

/* out (bf16, round-to-nearest-even of the fp32 result O) and, when not NULL, lse and out_res,
 * the rounding residual bf16(O - out): out + out_res carries O to about 16 significant bits,
 * which the backward uses for an exact Delta.
 * Errors: NULL desc, q, k, v or out -> DSA3D_ERR_NULL_POINTER; a dimension or window < 1, a
 * shift outside [0, window), a negative or non-finite scale, B*T*H*W*heads of 2^31 or more, a
 * grid side of 2^24 or more, or a window volume above DSA3D_WIN_MAX_TOKENS ->
 * DSA3D_ERR_INVALID_SHAPE; a dtype other than bf16 or a head_dim other than 64 and 128 ->
 * DSA3D_ERR_UNSUPPORTED; q, k, v, out, out_res not 16-byte or lse not 4-byte aligned ->
 * DSA3D_ERR_MISALIGNED; out, out_res or lse overlapping an input or each other ->
 * DSA3D_ERR_ALIAS. */
dsa3d_status dsa3d_win_forward(const dsa3d_win_desc* desc, const void* q, const void* k,
                               const void* v, void* out, void* out_res, float* lse,
                               hipStream_t stream);

/* Workspace bytes dsa3d_win_backward needs: 4 per query row (Delta = <dout, out>), rounded up
 * to 256; 0 for a descriptor it would reject. */
size_t dsa3d_win_backward_workspace_size(const dsa3d_win_desc* desc);

/* Phases of dsa3d_win_backward, in launch order: 0 the pass over query tiles (dq and Delta),
 * 1 the pass over key tiles (dk, dv). */
#define DSA3D_WIN_BACKWARD_PHASES 2

/* Backward for upstream gradient dout, with alpha recomputed from lse:
 *   dP = <dout, v_key>,  Delta = <dout, O> (= sum alpha dP),  dS = alpha (dP - Delta)
 *   dq = scale sum dS k_key,   dk_key = scale sum over its queries of dS q,
 *   dv_key = sum over its queries of alpha dout
 * out, out_res and lse are the forward's for the same inputs; O is taken as out + out_res, or
 * as out alone when out_res is NULL (then Delta carries the bf16 rounding of the output,
 * about 2^-9 |dout| |out| per row, into dq and dk, as in flash attention; dv is unaffected).
 * dq, dk and dv are fully overwritten,
 * each element written once, with no atomics (bitwise repeatable).  The workspace (at least
 * dsa3d_win_backward_workspace_size bytes, 256-byte aligned) must not overlap any argument.
 * `events` is NULL or DSA3D_WIN_BACKWARD_PHASES + 1 HIP events created by the caller on the
 * current device: event i is recorded on `stream` right before phase i and the last one after
 * the last phase (a failed record returns DSA3D_ERR_DEVICE).
 * Errors as for the forward (out_res 16-byte aligned), plus: lse, dout, dq, dk or dv NULL ->
 * DSA3D_ERR_NULL_POINTER;
 * workspace missing or too small -> DSA3D_ERR_WORKSPACE; dq, dk, dv not 16-byte aligned ->
 * DSA3D_ERR_MISALIGNED; outputs overlapping an input, the workspace or each other ->
 * DSA3D_ERR_ALIAS. */
dsa3d_status dsa3d_win_backward(const dsa3d_win_desc* desc, const void* q, const void* k,
                                const void* v, const void* out, const void* out_res,
                                const float* lse, const void* dout, float* dq, float* dk, float* dv,
                                void* workspace, size_t workspace_bytes, hipStream_t stream,
                                const hipEvent_t* events);

#ifdef __cplusplus
}
#endif

#endif /* DSA3D_WIN_H */
