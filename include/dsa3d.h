/*
 * dsa3d.h -- C ABI of the MI355X (gfx950) 3D Deformable Slide Attention library.
 *
 * The operator is the attention term of Eq. (1) in Section 5.2 of the
 * MegaSlide-DiT paper: for every token (t, i, j) of a T x H' x W' latent video
 * grid and every head m, the k_t x k_h x k_w neighbourhood of sampling points
 * is moved by learned per-point offsets, K and V are sampled there by
 * trilinear interpolation (Section 5.3: F.grid_sample on 5D tensors, zero
 * padding), the scaled dot products q . k_p are soft-maxed over the points and
 * the weights average the sampled values:
 *
 *   pos_p   = (j, i, t) + g_p + offset_p            (x = w, y = h, z = t)
 *   k_p     = TrilinearSample(K_m, pos_p),   v_p = TrilinearSample(V_m, pos_p)
 *   alpha_p = softmax_p(scale * <q, k_p>)
 *   out     = sum_p alpha_p v_p,             lse = logsumexp_p(scale * <q, k_p>)
 *
 * g_p is the query-centred base grid of the kernel (the zero-offset ablation
 * of Section 9.1 reduces the operator to fixed local attention over it);
 * points are numbered p = (it * k_h + ih) * k_w + iw and
 * g_p = (iw - (k_w-1)/2, ih - (k_h-1)/2, it - (k_t-1)/2).  pos is formed in
 * fp32 as (float)(integer base) + offset.  A corner outside the grid
 * contributes zero; a point with all 8 corners outside still takes part in the
 * softmax with logit 0.  No causal mask (Section 5.3).  The depthwise-conv
 * term of Eq. (1), the projections W_q/W_k/W_v and the offset network are not
 * part of this library: it takes projected q, k, v and the offsets.
 *
 * Conventions shared by every entry point
 *  - Every data pointer is a DEVICE pointer on the current HIP device, owned
 *    by the caller.  The library never allocates, frees, synchronises or
 *    prints, and keeps no mutable global state; calls are thread-safe.
 *  - Work is enqueued on `stream` (NULL = the null stream).
 *    DSA3D_OK means "validated and enqueued"; a fault during execution shows
 *    up at the caller's next synchronisation.
 *  - All arguments are validated on the host before anything is enqueued.  On
 *    any error nothing is enqueued and no output is touched.
 *  - Tensors are contiguous and row-major:
 *      q, k, v, out, dout   [B][T][H][W][heads][head_dim]   dtype of the descriptor
 *      offsets, d_offsets   [B][T][H][W][heads][P][3]       float32, (x, y, z) in token units
 *      lse                  [B][T][H][W][heads]             float32
 *      dq, dk, dv           [B][T][H][W][heads][head_dim]   float32
 *  - Alignment: q, k, v, out, dout, dq, dk, dv must be 16-byte aligned;
 *    offsets, d_offsets and lse 4-byte aligned.
 *  - Outputs must not overlap inputs or each other.
 */
#ifndef DSA3D_H
#define DSA3D_H

#include <hip/hip_runtime_api.h> /* hipStream_t, hipEvent_t */
#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  DSA3D_OK = 0,
  DSA3D_ERR_NULL_POINTER = 1,  /* a required pointer (or the descriptor) is NULL           */
  DSA3D_ERR_INVALID_SHAPE = 2, /* a dim < 1, an even kernel size, a non-finite scale, or a
                                  size beyond the library's index range (see below)        */
  DSA3D_ERR_UNSUPPORTED = 3,   /* dtype or head_dim not built in, or P > DSA3D_MAX_POINTS  */
  DSA3D_ERR_MISALIGNED = 4,    /* a pointer breaks the alignment rule above               */
  DSA3D_ERR_WORKSPACE = 5,     /* workspace NULL or smaller than the required size        */
  DSA3D_ERR_DEVICE = 6,        /* a HIP launch failed (the HIP error is not cleared)      */
  DSA3D_ERR_ALIAS = 7,         /* an output overlaps an input or another output           */
  DSA3D_ERR_SCRATCH = 8        /* dsa3d_backward_noalloc: the problem needs more workspace
                                  than DSA3D_NOALLOC_SCRATCH_BYTES                          */
} dsa3d_status;

typedef enum { DSA3D_F32 = 0, DSA3D_BF16 = 1 } dsa3d_dtype;

/* Largest neighbourhood size P = kt * kh * kw accepted (the paper's 3x7x7 is 147). */
#define DSA3D_MAX_POINTS 1024

/* Problem descriptor.  Index range: B*T*H*W*heads (the number of query rows)
 * must be below 2^31; grid sizes below 2^24 so token coordinates are exact in
 * fp32. */
typedef struct {
  int32_t batch;      /* B                                              */
  int32_t frames;     /* T  (Section 5.2: T frames)                     */
  int32_t height;     /* H' (latent grid height)                        */
  int32_t width;      /* W' (latent grid width)                         */
  int32_t heads;      /* attention heads (offsets are per head)         */
  int32_t head_dim;   /* channels per head: 32, 64 or 128               */
  int32_t kt, kh, kw; /* odd base neighbourhood (the paper uses 3x7x7)  */
  float scale;        /* logit scale; 0 selects 1/sqrt(head_dim)        */
  dsa3d_dtype dtype;  /* storage type of q, k, v, out, dout             */
} dsa3d_desc;

/* Forward (Section 5.2, Eq. (1) attention term).
 *   q, k, v : inputs; offsets: learned offsets.
 *   out     : output, written in the descriptor's dtype (bf16 by round-to-nearest-even
 *             of the fp32 accumulator).
 *   lse     : per-row log-sum-exp of the logits, needed by dsa3d_backward; may be NULL
 *             for inference.
 * Accumulation is fp32 for both dtypes. */
dsa3d_status dsa3d_forward(const dsa3d_desc* desc, const void* q, const void* k, const void* v,
                           const float* offsets, void* out, float* lse, hipStream_t stream);

/* Bytes of device workspace dsa3d_backward needs for `desc`: about 60 bytes per
 * (query row, point) pair plus 12 bytes per trilinear cell.  Returns 0 for a descriptor that
 * dsa3d_backward would reject. */
size_t dsa3d_backward_workspace_size(const dsa3d_desc* desc);

/* Backward: the exact gradient of the forward (for full-parameter fine-tuning the offsets,
 * q, k and v all need gradients), with the standard softmax calculus
 *   da_p = <dout, v_p>,  Delta = sum_p alpha_p da_p,  ds_p = alpha_p (da_p - Delta)
 *   dq = scale sum_p ds_p k_p,   dK[c] += scale ds_p w_c q,   dV[c] += alpha_p w_c dout
 *   d_offsets[p] = sum_c (d w_c / d pos) (scale ds_p <q, K[c]> + alpha_p <dout, V[c]>)
 * summed over the trilinear corners c of every point (w_c its weight, zero-padded corners
 * skipped).  At an exact integer coordinate the floor-based (upper one-sided) derivative is
 * used.  alpha_p is recomputed from `lse`.
 *   out      : the forward's output for the same inputs, or NULL.  It is not read: Delta is
 *              formed exactly from the recomputed alpha_p and da_p while the points are swept
 *              (it equals <dout, out> up to the rounding of out to its storage type, which
 *              for bf16 would cost about 2^-9 of Delta).  When given it must be 16-byte
 *              aligned and must not overlap an output or the workspace.
 *   lse      : the forward's LSE for the same inputs.
 *   dout     : upstream gradient of out (descriptor dtype).
 *   dq, d_offsets : fully overwritten.
 *   dk, dv   : fully overwritten.  No floating-point atomics are used: every (row, point)
 *              pair is binned by its trilinear cell and each voxel gathers its gradient
 *              rows from the 8 bins it is a corner of.  The order of the pairs inside a bin
 *              follows the order in which they claimed their slots, which can change from
 *              call to call, so dk and dv can differ between calls in the last bits
 *              (dq and d_offsets are bitwise repeatable).
 *   workspace: device memory of at least dsa3d_backward_workspace_size(desc) bytes, 256-byte
 *              aligned, not overlapping any argument; contents on entry do not matter.
 * Additional limit: rows * P and the number of cells, B*heads*(T+1)*(H+1)*(W+1), must be
 * below 2^31 (DSA3D_ERR_INVALID_SHAPE otherwise).
 * Accumulation is fp32. */
dsa3d_status dsa3d_backward(const dsa3d_desc* desc, const void* q, const void* k, const void* v,
                            const float* offsets, const void* out, const float* lse,
                            const void* dout, float* dq, float* dk, float* dv, float* d_offsets,
                            void* workspace, size_t workspace_bytes, hipStream_t stream);

/* Phases of dsa3d_backward, in launch order: 0 the pass over the V corners of every query row
 * (da_p, per-point records, bin counts and ranks), 1 the exclusive scan of the bin counts, 2 the
 * pass over the K corners (alpha_p, dq, and once a row's Delta is known its d_offsets and
 * binned dK/dV coefficients), 3 the dK/dV gather over voxels. */
#define DSA3D_BACKWARD_PHASES 4

/* dsa3d_backward with phase timing, for benchmarks and profilers.  `events` is NULL or
 * points to DSA3D_BACKWARD_PHASES + 1 HIP events (created by the caller on the current
 * device and owned by it); event i is recorded on `stream` right before phase i is launched
 * and the last one after the last phase, so the time between events i and i + 1 is phase i
 * alone.  Arguments, checks and results are those of dsa3d_backward; a failed event record
 * returns DSA3D_ERR_DEVICE. */
dsa3d_status dsa3d_backward_timed(const dsa3d_desc* desc, const void* q, const void* k,
                                  const void* v, const float* offsets, const void* out,
                                  const float* lse, const void* dout, float* dq, float* dk,
                                  float* dv, float* d_offsets, void* workspace,
                                  size_t workspace_bytes, hipStream_t stream,
                                  const hipEvent_t* events);

/* Bytes of the fixed device scratch buffer of dsa3d_backward_noalloc (128 MiB). */
#define DSA3D_NOALLOC_SCRATCH_BYTES (128u << 20)

/* dsa3d_backward without a caller workspace and without any allocation, for callers that
 * cannot allocate device memory (code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc).  The workspace is a file-scope device array of the library,
 * DSA3D_NOALLOC_SCRATCH_BYTES bytes on each GPU the library runs on, held until the process
 * ends; its device address is looked up once per device on the first call there.  Arguments,
 * results and checks are those of dsa3d_backward minus the workspace; a problem whose
 * dsa3d_backward_workspace_size exceeds the scratch returns DSA3D_ERR_SCRATCH (that is about
 * 2.2 million (row, point) pairs, e.g. 80,000 query rows with a 3x3x3 kernel) and enqueues
 * nothing.  Every call on a GPU uses that GPU's one scratch array: calls that can overlap on
 * one GPU (two streams, two host threads) race and must be serialised by the caller.  The
 * library clears what must start at zero on `stream` itself (with a kernel, not a memset),
 * so nothing from an earlier call carries over. */
dsa3d_status dsa3d_backward_noalloc(const dsa3d_desc* desc, const void* q, const void* k,
                                    const void* v, const float* offsets, const void* out,
                                    const float* lse, const void* dout, float* dq, float* dk,
                                    float* dv, float* d_offsets, hipStream_t stream);

/* Static description of a status code (never NULL). */
const char* dsa3d_status_string(dsa3d_status status);

/* ABI version of this header: 1. */
int dsa3d_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* DSA3D_H */
