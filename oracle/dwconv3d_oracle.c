/*
 * CPU oracle for the depthwise 3D convolution of 3D-DSA.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the bench's
 * CPU-baseline leg may load this library.  It shares no source, header,
 * table or helper with the GPU library and must never be used as a fallback
 * for it.
 *
 * What it computes (MegaSlide-DiT, Section 5.2, Eq. (1): the DWConv3D term
 * added to the attention output; Section 5.3: the offset network's depthwise
 * nn.Conv3d with groups equal to the channel count):
 *
 *   x, y : [B][T][H][W][C]   (channels last, the layout of the activation X)
 *   w    : [C][kt][kh][kw]   (one filter per channel: depthwise)
 *   bias : [C] or none
 *
 *   y[b,t,i,j,c] = bias[c] + sum over (a, e, f) in [0,kt) x [0,kh) x [0,kw) of
 *                  w[c][a][e][f] * x[b, t + a - rt, i + e - rh, j + f - rw, c]
 *
 *   with rt = (kt-1)/2, rh = (kh-1)/2, rw = (kw-1)/2 and x read as zero
 *   outside the grid ("same" zero padding, nn.Conv3d's cross-correlation with
 *   padding (rt, rh, rw)).  Gradients, by the chain rule of that sum:
 *
 *   dx[b,t,i,j,c] = sum_(a,e,f) w[c][a][e][f] * dy[b, t - a + rt, i - e + rh, j - f + rw, c]
 *   dw[c][a][e][f] = sum_(b,t,i,j) dy[b,t,i,j,c] * x[b, t + a - rt, i + e - rh, j + f - rw, c]
 *   dbias[c]       = sum_(b,t,i,j) dy[b,t,i,j,c]
 *
 *   (dy read as zero outside the grid in dx).  Everything is accumulated in
 *   fp64; bf16 inputs are widened exactly.  Kernel sizes are odd (the "same"
 *   padding the formula assumes).
 */
#include <math.h>
#include <omp.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

typedef struct {
  int64_t B, T, H, W, C, kt, kh, kw;
  int32_t bf16, pad_;
} orc_conv;

static double cv_ld(const void* base, int bf16, int64_t idx) {
  if (bf16) {
    const uint16_t h = ((const uint16_t*)base)[idx];
    const uint32_t u = (uint32_t)h << 16;
    float f;
    memcpy(&f, &u, 4);
    return (double)f;
  }
  return (double)((const float*)base)[idx];
}

static int cv_bad(const orc_conv* p) {
  return p->B < 1 || p->T < 1 || p->H < 1 || p->W < 1 || p->C < 1 || p->kt < 1 || p->kh < 1 ||
         p->kw < 1 || p->kt % 2 == 0 || p->kh % 2 == 0 || p->kw % 2 == 0;
}

/* element index of (b, t, i, j, c), or -1 outside the grid */
static int64_t cv_at(const orc_conv* p, int64_t b, int64_t t, int64_t i, int64_t j, int64_t c) {
  if (t < 0 || t >= p->T || i < 0 || i >= p->H || j < 0 || j >= p->W) return -1;
  return (((b * p->T + t) * p->H + i) * p->W + j) * p->C + c;
}

/* y for frames [t0, t1) of every batch item: y[b][t - t0][i][j][c] (fp64). */
int orc_dwconv_forward(const orc_conv* p, const void* x, const float* w, const float* bias,
                       int64_t t0, int64_t t1, double* y) {
  if (cv_bad(p) || t0 < 0 || t1 > p->T || t0 > t1) return 1;
  const int64_t rt = (p->kt - 1) / 2, rh = (p->kh - 1) / 2, rw = (p->kw - 1) / 2;
  const int64_t taps = p->kt * p->kh * p->kw, nt = t1 - t0;
#pragma omp parallel for collapse(2) schedule(static)
  for (int64_t b = 0; b < p->B; ++b)
    for (int64_t t = t0; t < t1; ++t)
      for (int64_t i = 0; i < p->H; ++i)
        for (int64_t j = 0; j < p->W; ++j)
          for (int64_t c = 0; c < p->C; ++c) {
            double acc = bias ? (double)bias[c] : 0.0;
            for (int64_t a = 0; a < p->kt; ++a)
              for (int64_t e = 0; e < p->kh; ++e)
                for (int64_t f = 0; f < p->kw; ++f) {
                  const int64_t src = cv_at(p, b, t + a - rt, i + e - rh, j + f - rw, c);
                  if (src < 0) continue;
                  acc += (double)w[c * taps + (a * p->kh + e) * p->kw + f] * cv_ld(x, p->bf16, src);
                }
            y[(((b * nt + (t - t0)) * p->H + i) * p->W + j) * p->C + c] = acc;
          }
  return 0;
}

/* dx for frames [t0, t1) (dx[b][t - t0][i][j][c], may be NULL), and, when dw / db are not
 * NULL, dw[C][kt][kh][kw] and db[C] summed over the whole grid. */
int orc_dwconv_backward(const orc_conv* p, const void* x, const float* w, const void* dy,
                        int64_t t0, int64_t t1, double* dx, double* dw, double* db) {
  if (cv_bad(p) || t0 < 0 || t1 > p->T || t0 > t1) return 1;
  const int64_t rt = (p->kt - 1) / 2, rh = (p->kh - 1) / 2, rw = (p->kw - 1) / 2;
  const int64_t taps = p->kt * p->kh * p->kw, nt = t1 - t0;
  if (dx) {
#pragma omp parallel for collapse(2) schedule(static)
    for (int64_t b = 0; b < p->B; ++b)
      for (int64_t t = t0; t < t1; ++t)
        for (int64_t i = 0; i < p->H; ++i)
          for (int64_t j = 0; j < p->W; ++j)
            for (int64_t c = 0; c < p->C; ++c) {
              double acc = 0.0;
              for (int64_t a = 0; a < p->kt; ++a)
                for (int64_t e = 0; e < p->kh; ++e)
                  for (int64_t f = 0; f < p->kw; ++f) {
                    const int64_t src = cv_at(p, b, t - a + rt, i - e + rh, j - f + rw, c);
                    if (src < 0) continue;
                    acc += (double)w[c * taps + (a * p->kh + e) * p->kw + f] * cv_ld(dy, p->bf16, src);
                  }
              dx[(((b * nt + (t - t0)) * p->H + i) * p->W + j) * p->C + c] = acc;
            }
  }
  if (dw || db) {
    /* one channel per iteration: each (c, tap) sum is a plain loop over the grid */
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t c = 0; c < p->C; ++c) {
      if (db) {
        double s = 0.0;
        for (int64_t b = 0; b < p->B; ++b)
          for (int64_t t = 0; t < p->T; ++t)
            for (int64_t i = 0; i < p->H; ++i)
              for (int64_t j = 0; j < p->W; ++j) s += cv_ld(dy, p->bf16, cv_at(p, b, t, i, j, c));
        db[c] = s;
      }
      if (!dw) continue;
      for (int64_t a = 0; a < p->kt; ++a)
        for (int64_t e = 0; e < p->kh; ++e)
          for (int64_t f = 0; f < p->kw; ++f) {
            double s = 0.0;
            for (int64_t b = 0; b < p->B; ++b)
              for (int64_t t = 0; t < p->T; ++t)
                for (int64_t i = 0; i < p->H; ++i)
                  for (int64_t j = 0; j < p->W; ++j) {
                    const int64_t src = cv_at(p, b, t + a - rt, i + e - rh, j + f - rw, c);
                    if (src < 0) continue;
                    s += cv_ld(dy, p->bf16, cv_at(p, b, t, i, j, c)) * cv_ld(x, p->bf16, src);
                  }
            dw[c * taps + (a * p->kh + e) * p->kw + f] = s;
          }
    }
  }
  return 0;
}
