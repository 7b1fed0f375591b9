/*
 * CPU oracle for 3D Deformable Slide Attention (3D-DSA).
 *
 * TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the bench's
 * CPU-baseline leg may load this library.  It shares no source, header,
 * table or helper with the GPU library and must never be used as a fallback
 * for it.
 *
 * What it computes (MegaSlide-DiT, Section 5.2, Eq. (1) attention term; the
 * DWConv3D term and the projections are outside the operator):
 *
 *   For batch b, token (t, i, j) on the T x H' x W' latent grid and head m,
 *   each point p of the k_t x k_h x k_w neighbourhood has the sampling
 *   position   pos_p = (j, i, t) + g_p + dp_p                      (x, y, z)
 *   where g_p is the query-centred base offset of the kernel cell and dp_p the
 *   learned offset.  (Section 5.2 writes the position as the token index plus
 *   the offset; the zero-offset ablation of Section 9.1, which turns the
 *   operator into fixed local attention over the whole kernel, fixes the
 *   base grid g_p.)
 *
 *   k_p = TrilinearSample(K_m, pos_p),  v_p = TrilinearSample(V_m, pos_p)
 *   s_p = scale * <q, k_p>,   alpha = softmax_p(s),   LSE = logsumexp_p(s)
 *   out = sum_p alpha_p v_p
 *
 *   TrilinearSample is grid_sample-style trilinear interpolation (Section 5.3
 *   names F.grid_sample in bilinear mode on 5D tensors) with zero padding:
 *   each of the 8 corners that lies outside the grid contributes zero and the
 *   others keep their weights.
 *
 * Readings of points the paper leaves open (each is documented with the
 * tests that pin it):
 *   - positions are in token-grid units; offsets are stored (x=w, y=h, z=t);
 *   - points are enumerated row-major over (it, ih, iw), iw fastest;
 *   - pos is formed in fp32 with one rounding, (float)(integer base) + dp;
 *     its floor and fractional part are then exact, and everything after
 *     that is fp64 here;
 *   - a point whose 8 corners are all outside still takes part in the
 *     softmax with k_p = v_p = 0 (logit 0);
 *   - at an exact integer coordinate the derivative is the one-sided one of
 *     the floor-based formula (upper corner weight 0);
 *   - no causal mask (Section 5.3).
 *
 * Backward: the exact derivative of the above, written with the standard
 * softmax calculus:
 *   da_p = <dout, v_p>,  Delta = sum_p alpha_p da_p,  ds_p = alpha_p (da_p - Delta)
 *   dq   = scale * sum_p ds_p k_p
 *   dK[corner c of p] += scale * ds_p * w_c * q      (zero-padded corners skipped)
 *   dV[corner c of p] += alpha_p * w_c * dout
 *   d dp_p[axis] = sum_c (d w_c / d pos[axis]) * (scale ds_p <q,K[c]> + alpha_p <dout,V[c]>)
 *
 * Build: gcc -O2 -fopenmp -shared -fPIC dsa3d_oracle.c -o liboracle.so -lm
 */
#include <math.h>
#include <omp.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

typedef struct {
  int64_t B, T, H, W; /* batch, frames, grid height H', grid width W' */
  int64_t heads, D;   /* heads, head dim */
  int64_t kt, kh, kw; /* base neighbourhood (odd) */
  double scale;       /* logit scale */
  int32_t bf16;       /* q, k, v, dout hold bf16 bit patterns (1) or fp32 (0) */
  int32_t pad_;
} orc_problem;

/* element of an io tensor as a double (bf16 -> fp32 is exact) */
static double ld(const void* base, int bf16, int64_t idx) {
  if (!bf16) return (double)((const float*)base)[idx];
  uint32_t bits = ((uint32_t)((const uint16_t*)base)[idx]) << 16;
  float f;
  memcpy(&f, &bits, 4);
  return (double)f;
}

/* flat row index of (b, t, i, j, head) in a [B][T][H][W][heads] row space */
static int64_t row_of(const orc_problem* pr, int64_t b, int64_t t, int64_t i, int64_t j, int64_t m) {
  return (((b * pr->T + t) * pr->H + i) * pr->W + j) * pr->heads + m;
}

/* One sampling point: its position and its 8 trilinear corners. */
typedef struct {
  float pos[3];      /* x, y, z in token-grid units (fp32, one rounding) */
  int64_t cell[3];   /* floor(pos) */
  double frac[3];    /* pos - floor(pos), in [0, 1) */
  int valid[8];      /* corner inside the grid */
  int64_t crow[8];   /* row index of the corner (when valid) */
  double w[8];       /* trilinear weight of the corner */
} orc_point;

/* Corner c = (cz, cy, cx) bits: c = cz*4 + cy*2 + cx. */
static void sample_point(const orc_problem* pr, int64_t b, int64_t t, int64_t i, int64_t j, int64_t m,
                         int64_t p, const float* dp, orc_point* s) {
  const int64_t it = p / (pr->kh * pr->kw);
  const int64_t ih = (p / pr->kw) % pr->kh;
  const int64_t iw = p % pr->kw;
  /* base grid: query-centred kernel cell */
  const int64_t gx = iw - (pr->kw - 1) / 2;
  const int64_t gy = ih - (pr->kh - 1) / 2;
  const int64_t gz = it - (pr->kt - 1) / 2;
  s->pos[0] = (float)(j + gx) + dp[0];
  s->pos[1] = (float)(i + gy) + dp[1];
  s->pos[2] = (float)(t + gz) + dp[2];
  const int64_t size[3] = {pr->W, pr->H, pr->T};
  int far_out = 0;
  for (int a = 0; a < 3; ++a) {
    float f = floorf(s->pos[a]);
    double fr = (double)s->pos[a] - (double)f; /* exact in fp64 (not always in fp32) */
    /* A position more than one cell outside the grid has no corner inside;
     * keep the integer conversion in range for such (or non-finite) values. */
    if (!(f >= -2.0f && f <= (float)size[a] + 1.0f)) {
      far_out = 1;
      f = -2.0f;
      fr = 0.0;
    }
    s->cell[a] = (int64_t)f;
    s->frac[a] = fr;
  }
  for (int c = 0; c < 8; ++c) {
    const int cx = c & 1, cy = (c >> 1) & 1, cz = (c >> 2) & 1;
    const int64_t x = s->cell[0] + cx, y = s->cell[1] + cy, z = s->cell[2] + cz;
    const double wx = cx ? s->frac[0] : 1.0 - s->frac[0];
    const double wy = cy ? s->frac[1] : 1.0 - s->frac[1];
    const double wz = cz ? s->frac[2] : 1.0 - s->frac[2];
    s->w[c] = wx * wy * wz;
    s->valid[c] = !far_out && x >= 0 && x < pr->W && y >= 0 && y < pr->H && z >= 0 && z < pr->T;
    s->crow[c] = s->valid[c] ? row_of(pr, b, z, y, x, m) : -1;
  }
}

/* k_p or v_p: zero-padded trilinear sample of one head's rows, fp64. */
static void trilinear(const orc_problem* pr, const void* F, const orc_point* s, double* acc) {
  for (int64_t d = 0; d < pr->D; ++d) acc[d] = 0.0;
  for (int c = 0; c < 8; ++c) {
    if (!s->valid[c]) continue;
    for (int64_t d = 0; d < pr->D; ++d) acc[d] += s->w[c] * ld(F, pr->bf16, s->crow[c] * pr->D + d);
  }
}

int orc_num_points(const orc_problem* pr) { return (int)(pr->kt * pr->kh * pr->kw); }

/* Threads an OpenMP parallel region of this library uses. */
int orc_max_threads(void) {
  int n = 1;
#pragma omp parallel
  {
#pragma omp single
    n = omp_get_num_threads();
  }
  return n;
}

/*
 * Forward for a list of query rows.
 *   rows[r] = flat index of (b, t, i, j, head), row-major over [B][T][H][W][heads].
 *   out[r][D] = attention output, lse[r] = logsumexp of the logits (may be NULL).
 *   q, k, v : [B][T][H][W][heads][D] (bf16 bits or fp32); off: [..][heads][P][3] fp32.
 * Returns 0, or -1 on a malformed problem.
 */
int orc_forward(const orc_problem* pr, const void* q, const void* k, const void* v, const float* off,
                const int64_t* rows, int64_t nrows, double* out, double* lse) {
  const int64_t P = pr->kt * pr->kh * pr->kw, D = pr->D;
  if (P <= 0 || D <= 0 || pr->kt % 2 == 0 || pr->kh % 2 == 0 || pr->kw % 2 == 0) return -1;
#pragma omp parallel
  {
    double* kp = (double*)malloc(sizeof(double) * D);
    double* vp = (double*)malloc(sizeof(double) * D * P);
    double* sp = (double*)malloc(sizeof(double) * P);
    double* al = (double*)malloc(sizeof(double) * P);
#pragma omp for schedule(dynamic, 16)
    for (int64_t r = 0; r < nrows; ++r) {
      const int64_t row = rows[r];
      const int64_t m = row % pr->heads;
      const int64_t tok = row / pr->heads;
      const int64_t j = tok % pr->W, i = (tok / pr->W) % pr->H, t = (tok / (pr->W * pr->H)) % pr->T;
      const int64_t b = tok / (pr->W * pr->H * pr->T);
      for (int64_t p = 0; p < P; ++p) {
        orc_point s;
        sample_point(pr, b, t, i, j, m, p, off + (row * P + p) * 3, &s);
        trilinear(pr, k, &s, kp);
        trilinear(pr, v, &s, vp + p * D);
        double dot = 0.0;
        for (int64_t d = 0; d < D; ++d) dot += ld(q, pr->bf16, row * D + d) * kp[d];
        sp[p] = pr->scale * dot;
      }
      double mx = -INFINITY;
      for (int64_t p = 0; p < P; ++p) mx = sp[p] > mx ? sp[p] : mx;
      double l = 0.0;
      for (int64_t p = 0; p < P; ++p) l += exp(sp[p] - mx);
      for (int64_t p = 0; p < P; ++p) al[p] = exp(sp[p] - mx) / l;
      for (int64_t d = 0; d < D; ++d) {
        double o = 0.0;
        for (int64_t p = 0; p < P; ++p) o += al[p] * vp[p * D + d];
        out[r * D + d] = o;
      }
      if (lse) lse[r] = mx + log(l);
    }
    free(kp);
    free(vp);
    free(sp);
    free(al);
  }
  return 0;
}

/* Scratch of one query's backward, sized for P points and D channels. */
typedef struct {
  orc_point* pts;
  double *kp, *vp, *qv, *gv, *sp, *al, *da;
} orc_scratch;

static void scratch_alloc(orc_scratch* w, int64_t P, int64_t D) {
  w->pts = (orc_point*)malloc(sizeof(orc_point) * P);
  w->kp = (double*)malloc(sizeof(double) * D * P);
  w->vp = (double*)malloc(sizeof(double) * D * P);
  w->qv = (double*)malloc(sizeof(double) * D);
  w->gv = (double*)malloc(sizeof(double) * D);
  w->sp = (double*)malloc(sizeof(double) * P);
  w->al = (double*)malloc(sizeof(double) * P);
  w->da = (double*)malloc(sizeof(double) * P);
}

static void scratch_free(orc_scratch* w) {
  free(w->pts);
  free(w->kp);
  free(w->vp);
  free(w->qv);
  free(w->gv);
  free(w->sp);
  free(w->al);
  free(w->da);
}

/* Backward of one query (b, t, i, j, head m).  Writes dq_out[D] and doff_out[P][3];
 * when dk/dv are given ([T*H*W][D] of (b, m)) the query's contributions are added there. */
static void backward_query(const orc_problem* pr, const void* q, const void* k, const void* v,
                           const float* off, const void* dout, int64_t b, int64_t t, int64_t i,
                           int64_t j, int64_t m, double* dq_out, double* doff_out, double* dk,
                           double* dv, orc_scratch* w) {
  const int64_t P = pr->kt * pr->kh * pr->kw, D = pr->D;
  const int64_t HW = pr->H * pr->W;
  const int64_t row = row_of(pr, b, t, i, j, m);
  for (int64_t d = 0; d < D; ++d) {
    w->qv[d] = ld(q, pr->bf16, row * D + d);
    w->gv[d] = ld(dout, pr->bf16, row * D + d);
  }
  /* forward recompute */
  for (int64_t p = 0; p < P; ++p) {
    sample_point(pr, b, t, i, j, m, p, off + (row * P + p) * 3, &w->pts[p]);
    trilinear(pr, k, &w->pts[p], w->kp + p * D);
    trilinear(pr, v, &w->pts[p], w->vp + p * D);
    double dot = 0.0, dd = 0.0;
    for (int64_t d = 0; d < D; ++d) {
      dot += w->qv[d] * w->kp[p * D + d];
      dd += w->gv[d] * w->vp[p * D + d];
    }
    w->sp[p] = pr->scale * dot;
    w->da[p] = dd;
  }
  double mx = -INFINITY;
  for (int64_t p = 0; p < P; ++p) mx = w->sp[p] > mx ? w->sp[p] : mx;
  double l = 0.0;
  for (int64_t p = 0; p < P; ++p) l += exp(w->sp[p] - mx);
  double delta = 0.0;
  for (int64_t p = 0; p < P; ++p) {
    w->al[p] = exp(w->sp[p] - mx) / l;
    delta += w->al[p] * w->da[p];
  }
  /* dq */
  for (int64_t d = 0; d < D; ++d) {
    double acc = 0.0;
    for (int64_t p = 0; p < P; ++p) acc += w->al[p] * (w->da[p] - delta) * w->kp[p * D + d];
    dq_out[d] = pr->scale * acc;
  }
  /* dK, dV scatter and offset gradients */
  for (int64_t p = 0; p < P; ++p) {
    const orc_point* s = &w->pts[p];
    const double al = w->al[p];
    const double ds = al * (w->da[p] - delta);
    double g[3] = {0.0, 0.0, 0.0};
    for (int c = 0; c < 8; ++c) {
      if (!s->valid[c]) continue;
      const int cx = c & 1, cy = (c >> 1) & 1, cz = (c >> 2) & 1;
      const int64_t dst = ((s->crow[c] / pr->heads) % (pr->T * HW)) * D; /* (z,y,x) of batch b */
      double qk = 0.0, dvv = 0.0;
      for (int64_t d = 0; d < D; ++d) {
        const double kc = ld(k, pr->bf16, s->crow[c] * D + d);
        const double vc = ld(v, pr->bf16, s->crow[c] * D + d);
        qk += w->qv[d] * kc;
        dvv += w->gv[d] * vc;
        if (dk) {
          const double addk = pr->scale * ds * s->w[c] * w->qv[d];
          const double addv = al * s->w[c] * w->gv[d];
#pragma omp atomic
          dk[dst + d] += addk;
#pragma omp atomic
          dv[dst + d] += addv;
        }
      }
      const double G = pr->scale * ds * qk + al * dvv;
      const double ax[2] = {1.0 - s->frac[0], s->frac[0]};
      const double ay[2] = {1.0 - s->frac[1], s->frac[1]};
      const double az[2] = {1.0 - s->frac[2], s->frac[2]};
      g[0] += G * (cx ? 1.0 : -1.0) * ay[cy] * az[cz];
      g[1] += G * (cy ? 1.0 : -1.0) * ax[cx] * az[cz];
      g[2] += G * (cz ? 1.0 : -1.0) * ax[cx] * ay[cy];
    }
    for (int a = 0; a < 3; ++a) doff_out[p * 3 + a] = g[a];
  }
}

/*
 * Backward for the queries of batch b, head m and frames [t0, t1).
 *   dq   [(t1-t0)*H*W][D]       gradient w.r.t. q of those queries (overwritten)
 *   doff [(t1-t0)*H*W][P][3]    gradient w.r.t. their offsets (overwritten)
 *   dk, dv [T*H*W][D]           gradient w.r.t. K, V of (b, m), ACCUMULATED (+=)
 *                               from these queries only; the caller zeroes them.
 * Recomputes the forward; does not need the stored output or LSE.
 */
int orc_backward(const orc_problem* pr, const void* q, const void* k, const void* v, const float* off,
                 const void* dout, int64_t b, int64_t m, int64_t t0, int64_t t1, double* dq,
                 double* doff, double* dk, double* dv) {
  const int64_t P = pr->kt * pr->kh * pr->kw, D = pr->D;
  const int64_t HW = pr->H * pr->W;
  if (P <= 0 || D <= 0 || t0 < 0 || t1 > pr->T || t0 > t1) return -1;
  const int64_t nq = (t1 - t0) * HW;
#pragma omp parallel
  {
    orc_scratch w;
    scratch_alloc(&w, P, D);
#pragma omp for schedule(dynamic, 16)
    for (int64_t n = 0; n < nq; ++n) {
      const int64_t t = t0 + n / HW, i = (n % HW) / pr->W, j = n % pr->W;
      backward_query(pr, q, k, v, off, dout, b, t, i, j, m, dq + n * D, doff + n * P * 3, dk, dv, &w);
    }
    scratch_free(&w);
  }
  return 0;
}

/*
 * dq [nrows][D] and doff [nrows][P][3] of a list of query rows (flat (b, t, i, j, head)
 * indices as in orc_forward).  No dK/dV: those gather contributions of many queries.
 */
int orc_backward_rows(const orc_problem* pr, const void* q, const void* k, const void* v,
                      const float* off, const void* dout, const int64_t* rows, int64_t nrows,
                      double* dq, double* doff) {
  const int64_t P = pr->kt * pr->kh * pr->kw, D = pr->D;
  if (P <= 0 || D <= 0) return -1;
#pragma omp parallel
  {
    orc_scratch w;
    scratch_alloc(&w, P, D);
#pragma omp for schedule(dynamic, 4)
    for (int64_t r = 0; r < nrows; ++r) {
      const int64_t row = rows[r];
      const int64_t m = row % pr->heads, tok = row / pr->heads;
      const int64_t j = tok % pr->W, i = (tok / pr->W) % pr->H, t = (tok / (pr->W * pr->H)) % pr->T;
      const int64_t b = tok / (pr->W * pr->H * pr->T);
      backward_query(pr, q, k, v, off, dout, b, t, i, j, m, dq + r * D, doff + r * P * 3, NULL, NULL,
                     &w);
    }
    scratch_free(&w);
  }
  return 0;
}

/*
 * Predicted-weights variant.  Section 5.2 says the module learns offsets "and attention
 * weights"; in this variant (as in Deformable DETR) the weights come from logits a_p that a
 * linear layer predicts per (token, head, point), instead of from q.k:
 *   alpha = softmax_p(a),  out = sum_p alpha_p v_p,  LSE = logsumexp_p(a)
 * with v_p the same zero-padded trilinear sample of V.  There is no q and no K.
 * Backward (same softmax calculus, no scale):
 *   da_p = <dout, v_p>,  Delta = sum_p alpha_p da_p
 *   d a_p          = alpha_p (da_p - Delta)
 *   dV[corner c]  += alpha_p w_c dout
 *   d dp_p[axis]   = alpha_p sum_c (d w_c / d pos[axis]) <dout, V[c]>
 * logits, dlogits: [B][T][H][W][heads][P] (fp32 in, fp64 out here).
 */
static void pw_query(const orc_problem* pr, const float* logits, const void* v, const float* off,
                     const void* dout, int64_t b, int64_t t, int64_t i, int64_t j, int64_t m,
                     double* out, double* lse, double* dlog, double* doff, double* dv,
                     orc_scratch* w) {
  const int64_t P = pr->kt * pr->kh * pr->kw, D = pr->D;
  const int64_t HW = pr->H * pr->W;
  const int64_t row = row_of(pr, b, t, i, j, m);
  double mx = -INFINITY;
  for (int64_t p = 0; p < P; ++p) {
    w->sp[p] = (double)logits[row * P + p];
    mx = w->sp[p] > mx ? w->sp[p] : mx;
  }
  double l = 0.0;
  for (int64_t p = 0; p < P; ++p) l += exp(w->sp[p] - mx);
  for (int64_t p = 0; p < P; ++p) {
    w->al[p] = exp(w->sp[p] - mx) / l;
    sample_point(pr, b, t, i, j, m, p, off + (row * P + p) * 3, &w->pts[p]);
    trilinear(pr, v, &w->pts[p], w->vp + p * D);
  }
  if (out) {
    for (int64_t d = 0; d < D; ++d) {
      double o = 0.0;
      for (int64_t p = 0; p < P; ++p) o += w->al[p] * w->vp[p * D + d];
      out[d] = o;
    }
  }
  if (lse) *lse = mx + log(l);
  if (!dlog && !doff && !dv) return;
  for (int64_t d = 0; d < D; ++d) w->gv[d] = ld(dout, pr->bf16, row * D + d);
  double delta = 0.0;
  for (int64_t p = 0; p < P; ++p) {
    double dd = 0.0;
    for (int64_t d = 0; d < D; ++d) dd += w->gv[d] * w->vp[p * D + d];
    w->da[p] = dd;
    delta += w->al[p] * dd;
  }
  for (int64_t p = 0; p < P; ++p) {
    const orc_point* s = &w->pts[p];
    const double al = w->al[p];
    if (dlog) dlog[p] = al * (w->da[p] - delta);
    double g[3] = {0.0, 0.0, 0.0};
    for (int c = 0; c < 8; ++c) {
      if (!s->valid[c]) continue;
      const int cx = c & 1, cy = (c >> 1) & 1, cz = (c >> 2) & 1;
      const int64_t dst = ((s->crow[c] / pr->heads) % (pr->T * HW)) * D; /* (z,y,x) of batch b */
      double dvv = 0.0;
      for (int64_t d = 0; d < D; ++d) {
        dvv += w->gv[d] * ld(v, pr->bf16, s->crow[c] * D + d);
        if (dv) {
          const double add = al * s->w[c] * w->gv[d];
#pragma omp atomic
          dv[dst + d] += add;
        }
      }
      const double ax[2] = {1.0 - s->frac[0], s->frac[0]};
      const double ay[2] = {1.0 - s->frac[1], s->frac[1]};
      const double az[2] = {1.0 - s->frac[2], s->frac[2]};
      g[0] += al * dvv * (cx ? 1.0 : -1.0) * ay[cy] * az[cz];
      g[1] += al * dvv * (cy ? 1.0 : -1.0) * ax[cx] * az[cz];
      g[2] += al * dvv * (cz ? 1.0 : -1.0) * ax[cx] * ay[cy];
    }
    if (doff)
      for (int a = 0; a < 3; ++a) doff[p * 3 + a] = g[a];
  }
}

/* Forward of the predicted-weights variant for a list of rows (as orc_forward). */
int orc_pw_forward(const orc_problem* pr, const float* logits, const void* v, const float* off,
                   const int64_t* rows, int64_t nrows, double* out, double* lse) {
  const int64_t P = pr->kt * pr->kh * pr->kw, D = pr->D;
  if (P <= 0 || D <= 0 || pr->kt % 2 == 0 || pr->kh % 2 == 0 || pr->kw % 2 == 0) return -1;
#pragma omp parallel
  {
    orc_scratch w;
    scratch_alloc(&w, P, D);
#pragma omp for schedule(dynamic, 16)
    for (int64_t r = 0; r < nrows; ++r) {
      const int64_t row = rows[r];
      const int64_t m = row % pr->heads, tok = row / pr->heads;
      const int64_t j = tok % pr->W, i = (tok / pr->W) % pr->H, t = (tok / (pr->W * pr->H)) % pr->T;
      const int64_t b = tok / (pr->W * pr->H * pr->T);
      pw_query(pr, logits, v, off, NULL, b, t, i, j, m, out + r * D, lse ? lse + r : NULL, NULL,
               NULL, NULL, &w);
    }
    scratch_free(&w);
  }
  return 0;
}

/* Backward of the predicted-weights variant for the queries of batch b, head m, frames
 * [t0, t1): dlogits [(t1-t0)*H*W][P] and doff [..][P][3] overwritten; dv [T*H*W][D] of
 * (b, m) ACCUMULATED from these queries. */
int orc_pw_backward(const orc_problem* pr, const float* logits, const void* v, const float* off,
                    const void* dout, int64_t b, int64_t m, int64_t t0, int64_t t1, double* dlog,
                    double* doff, double* dv) {
  const int64_t P = pr->kt * pr->kh * pr->kw, D = pr->D;
  const int64_t HW = pr->H * pr->W;
  if (P <= 0 || D <= 0 || t0 < 0 || t1 > pr->T || t0 > t1) return -1;
  const int64_t nq = (t1 - t0) * HW;
#pragma omp parallel
  {
    orc_scratch w;
    scratch_alloc(&w, P, D);
#pragma omp for schedule(dynamic, 16)
    for (int64_t n = 0; n < nq; ++n) {
      const int64_t t = t0 + n / HW, i = (n % HW) / pr->W, j = n % pr->W;
      pw_query(pr, logits, v, off, dout, b, t, i, j, m, NULL, NULL, dlog + n * P,
               doff + n * P * 3, dv, &w);
    }
    scratch_free(&w);
  }
  return 0;
}
