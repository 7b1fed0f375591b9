/*
 * Predicted-weights variant of 3D Deformable Slide Attention, C ABI (gfx950 HIP kernels).
 *
 * MegaSlide-DiT's Section 5.2 says the module learns, per token and head, a set of offsets and
 * attention weights.  Eq. (1) (dsa3d.h) takes the weights from a softmax over q.k at the
 * sampled positions.  In this variant, as in Deformable DETR, a linear layer predicts one
 * logit a_p per (token, head, point) and
 *
 *   alpha = softmax_p(a),   out = sum_p alpha_p TrilinearSample(V, pos_p),   LSE = logsumexp_p(a)
 *
 * with pos_p and the zero-padded trilinear sampling exactly as in dsa3d_forward.  There is no q
 * and no K, so the corner gather halves.  The logits are used as given: the descriptor's scale
 * must be 0 or 1 (other values return DSA3D_ERR_INVALID_SHAPE); heads, head_dim, dtype and the
 * kernel size follow dsa3d.h, as do the conventions (plain device pointers, host validation
 * first, no allocation, no synchronisation, work enqueued on `stream`).
 *
 * Layouts: logits and dlogits [B][T][H][W][heads][P] float32 (P = kt kh kw, points in the
 * order of dsa3d.h); v, out, dout, dv, offsets, d_offsets and lse as in dsa3d.h.
 */
#ifndef DSA3D_PW_H
#define DSA3D_PW_H

#include <stddef.h>
#include <stdint.h>

#include "dsa3d.h"

#ifdef __cplusplus
extern "C" {
#endif

/* out and (when not NULL) lse = logsumexp of the logits; the errors of dsa3d_forward, with
 * logits taking the place of q and k (4-byte aligned). */
dsa3d_status dsa3d_pw_forward(const dsa3d_desc* desc, const float* logits, const void* v,
                              const float* offsets, void* out, float* lse, hipStream_t stream);

/* Workspace bytes dsa3d_pw_backward needs (the same binning as dsa3d_backward: about 56 bytes
 * per (row, point) and 12 per cell); 0 for a descriptor it would reject. */
size_t dsa3d_pw_backward_workspace_size(const dsa3d_desc* desc);

/* Backward for upstream gradient dout, with alpha_p recomputed from the logits and lse:
 *   da_p = <dout, v_p>,  Delta = sum_p alpha_p da_p
 *   dlogits[p]   = alpha_p (da_p - Delta)
 *   dV[c]        = sum over the points with corner c of alpha_p w_c dout
 *   d_offsets[p] = alpha_p sum_c (d w_c / d pos) <dout, V[c]>
 * dlogits, dv and d_offsets are fully overwritten (dv by the same atomic-free binned gather
 * as dsa3d_backward, whose order inside a bin can vary between calls); errors as for
 * dsa3d_backward.  `events` is NULL or DSA3D_BACKWARD_PHASES + 1 caller-owned HIP events,
 * recorded around the phases as by dsa3d_backward_timed. */
dsa3d_status dsa3d_pw_backward(const dsa3d_desc* desc, const float* logits, const void* v,
                               const float* offsets, const float* lse, const void* dout,
                               float* dlogits, float* dv, float* d_offsets, void* workspace,
                               size_t workspace_bytes, hipStream_t stream, const hipEvent_t* events);

#ifdef __cplusplus
}
#endif

#endif /* DSA3D_PW_H */
