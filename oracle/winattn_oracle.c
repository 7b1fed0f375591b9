/*
 * CPU oracle for fixed / shifted window attention: the Swin-DiT baseline of MegaSlide-DiT
 * (Section 6.2: windows of 3 x 16 x 16 tokens with shifted-window attention; Section 5.1
 * contrasts such static partitions with 3D-DSA's learned offsets).
 *
 * TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the bench's CPU-baseline leg
 * may load this library.  It shares no source, header, table or helper with the GPU library
 * and must never be used as a fallback for it.
 *
 * What it computes, per batch item b and head m, on the T x H x W grid with windows of
 * wt x wh x ww tokens and a cyclic shift (st, sh, sw), each shift below its window size:
 *
 *   The grid is padded to Tp x Hp x Wp (the next multiples of the window).  A token at grid
 *   position p = (t, i, j) sits at rolled position r = (p - shift) mod (Tp, Hp, Wp), and the
 *   windows tile the rolled grid.  Along each axis a rolled coordinate has a region: 0 below
 *   size - window, 1 below size - shift, 2 above (shift 0: always 0).  Query p attends to the
 *   keys p' of its window whose rolled position carries the same region on all three axes
 *   and which lie inside the real grid (padding positions are neither keys nor queries):
 *
 *     s(p, p') = scale <q_p, k_p'>,  alpha = softmax over those p',
 *     out_p = sum alpha(p, p') v_p',  LSE_p = logsumexp over those p' of s(p, p')
 *
 *   (Swin Transformer's shifted-window attention: roll, partition, mask the pairs that the
 *   roll brought together from distant parts of the grid.)  Backward, for upstream dout:
 *     dP = dout . v_p',  Delta_p = sum alpha dP,  dS = alpha (dP - Delta_p)
 *     dq_p = scale sum_p' dS k_p',  dk_p' += scale dS q_p,  dv_p' += alpha dout_p
 *   All in fp64; bf16 inputs are widened exactly.
 */
#include <math.h>
#include <omp.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

typedef struct {
  int64_t B, T, H, W, heads, D;
  int64_t wt, wh, ww; /* window */
  int64_t st, sh, sw; /* cyclic shift */
  double scale;
  int32_t bf16, pad_;
} orc_win;

static double wa_ld(const void* base, int bf16, int64_t idx) {
  if (bf16) {
    const uint32_t u = (uint32_t)((const uint16_t*)base)[idx] << 16;
    float f;
    memcpy(&f, &u, 4);
    return (double)f;
  }
  return (double)((const float*)base)[idx];
}

static int64_t wa_ceil(int64_t a, int64_t b) { return (a + b - 1) / b * b; }

static int wa_region(int64_t r, int64_t size, int64_t win, int64_t shift) {
  if (shift == 0) return 0;
  return r < size - win ? 0 : (r < size - shift ? 1 : 2);
}

static int wa_bad(const orc_win* p) {
  return p->B < 1 || p->T < 1 || p->H < 1 || p->W < 1 || p->heads < 1 || p->D < 1 || p->wt < 1 ||
         p->wh < 1 || p->ww < 1 || p->st < 0 || p->sh < 0 || p->sw < 0 || p->st >= p->wt ||
         p->sh >= p->wh || p->sw >= p->ww;
}

/* The keys of query (t, i, j): their token indices (t*H + i)*W + j within the batch item. */
static int64_t wa_keys(const orc_win* p, int64_t t, int64_t i, int64_t j, int64_t* keys) {
  const int64_t Tp = wa_ceil(p->T, p->wt), Hp = wa_ceil(p->H, p->wh), Wp = wa_ceil(p->W, p->ww);
  const int64_t rt = ((t - p->st) % Tp + Tp) % Tp, ri = ((i - p->sh) % Hp + Hp) % Hp,
                rj = ((j - p->sw) % Wp + Wp) % Wp;
  const int g0 = wa_region(rt, Tp, p->wt, p->st), g1 = wa_region(ri, Hp, p->wh, p->sh),
            g2 = wa_region(rj, Wp, p->ww, p->sw);
  const int64_t t0 = rt / p->wt * p->wt, i0 = ri / p->wh * p->wh, j0 = rj / p->ww * p->ww;
  int64_t n = 0;
  for (int64_t a = 0; a < p->wt; ++a)
    for (int64_t e = 0; e < p->wh; ++e)
      for (int64_t f = 0; f < p->ww; ++f) {
        const int64_t xt = t0 + a, xi = i0 + e, xj = j0 + f; /* rolled position of the key */
        if (wa_region(xt, Tp, p->wt, p->st) != g0 || wa_region(xi, Hp, p->wh, p->sh) != g1 ||
            wa_region(xj, Wp, p->ww, p->sw) != g2)
          continue;
        const int64_t gt = (xt + p->st) % Tp, gi = (xi + p->sh) % Hp, gj = (xj + p->sw) % Wp;
        if (gt >= p->T || gi >= p->H || gj >= p->W) continue; /* padding */
        keys[n++] = (gt * p->H + gi) * p->W + gj;
      }
  return n;
}

/* Forward for the tokens of frames [t0, t1) of every batch item and head:
 * out[b][t - t0][i][j][m][D], lse[b][t - t0][i][j][m]. */
int orc_win_forward(const orc_win* p, const void* q, const void* k, const void* v, int64_t t0,
                    int64_t t1, double* out, double* lse) {
  if (wa_bad(p) || t0 < 0 || t1 > p->T || t0 > t1) return 1;
  const int64_t N = p->T * p->H * p->W, D = p->D, M = p->heads, nw = p->wt * p->wh * p->ww;
  const int64_t HW = p->H * p->W, nt = t1 - t0;
#pragma omp parallel
  {
    int64_t* keys = (int64_t*)malloc(sizeof(int64_t) * nw);
    double* s = (double*)malloc(sizeof(double) * nw);
#pragma omp for collapse(2) schedule(dynamic, 16)
    for (int64_t b = 0; b < p->B; ++b)
      for (int64_t n = t0 * HW; n < t1 * HW; ++n) {
        const int64_t t = n / HW, i = (n / p->W) % p->H, j = n % p->W;
        const int64_t nk = wa_keys(p, t, i, j, keys);
        for (int64_t m = 0; m < M; ++m) {
          const int64_t qrow = ((b * N + n) * M + m) * D;
          double mx = -INFINITY;
          for (int64_t c = 0; c < nk; ++c) {
            const int64_t krow = ((b * N + keys[c]) * M + m) * D;
            double dot = 0.0;
            for (int64_t d = 0; d < D; ++d) dot += wa_ld(q, p->bf16, qrow + d) * wa_ld(k, p->bf16, krow + d);
            s[c] = p->scale * dot;
            mx = s[c] > mx ? s[c] : mx;
          }
          double l = 0.0;
          for (int64_t c = 0; c < nk; ++c) l += exp(s[c] - mx);
          const int64_t o = ((b * nt * HW + (n - t0 * HW)) * M + m);
          for (int64_t d = 0; d < D; ++d) {
            double acc = 0.0;
            for (int64_t c = 0; c < nk; ++c)
              acc += exp(s[c] - mx) / l * wa_ld(v, p->bf16, ((b * N + keys[c]) * M + m) * D + d);
            out[o * D + d] = acc;
          }
          if (lse) lse[o] = mx + log(l);
        }
      }
    free(keys);
    free(s);
  }
  return 0;
}

/* Backward over the queries of frames [t0, t1): dq, dk, dv [B][t1 - t0][H][W][heads][D]
 * (overwritten, fp64) for the tokens of those frames.  dq is complete; dk and dv receive the
 * contributions of the queries in the range, so they are complete for keys whose window
 * region lies inside the range (all of them for the full range). */
int orc_win_backward(const orc_win* p, const void* q, const void* k, const void* v,
                     const void* dout, int64_t t0, int64_t t1, double* dq, double* dk,
                     double* dv) {
  if (wa_bad(p) || t0 < 0 || t1 > p->T || t0 > t1) return 1;
  const int64_t N = p->T * p->H * p->W, D = p->D, M = p->heads, nw = p->wt * p->wh * p->ww;
  const int64_t HW = p->H * p->W, NR = (t1 - t0) * HW; /* tokens per batch item in the range */
  const int64_t total = p->B * NR * M * D;
  memset(dq, 0, sizeof(double) * total);
  memset(dk, 0, sizeof(double) * total);
  memset(dv, 0, sizeof(double) * total);
#pragma omp parallel
  {
    int64_t* keys = (int64_t*)malloc(sizeof(int64_t) * nw);
    double* s = (double*)malloc(sizeof(double) * nw);
    double* dp = (double*)malloc(sizeof(double) * nw);
#pragma omp for collapse(2) schedule(dynamic, 16)
    for (int64_t b = 0; b < p->B; ++b)
      for (int64_t n = t0 * p->H * p->W; n < t1 * p->H * p->W; ++n) {
        const int64_t t = n / (p->H * p->W), i = (n / p->W) % p->H, j = n % p->W;
        const int64_t nk = wa_keys(p, t, i, j, keys);
        for (int64_t m = 0; m < M; ++m) {
          const int64_t qrow = ((b * N + n) * M + m) * D;
          double mx = -INFINITY;
          for (int64_t c = 0; c < nk; ++c) {
            const int64_t krow = ((b * N + keys[c]) * M + m) * D;
            double dot = 0.0, g = 0.0;
            for (int64_t d = 0; d < D; ++d) {
              dot += wa_ld(q, p->bf16, qrow + d) * wa_ld(k, p->bf16, krow + d);
              g += wa_ld(dout, p->bf16, qrow + d) * wa_ld(v, p->bf16, krow + d);
            }
            s[c] = p->scale * dot;
            dp[c] = g;
            mx = s[c] > mx ? s[c] : mx;
          }
          double l = 0.0;
          for (int64_t c = 0; c < nk; ++c) l += exp(s[c] - mx);
          double delta = 0.0;
          for (int64_t c = 0; c < nk; ++c) delta += exp(s[c] - mx) / l * dp[c];
          const int64_t orow = ((b * NR + n - t0 * HW) * M + m) * D; /* this query's output row */
          for (int64_t c = 0; c < nk; ++c) {
            const double al = exp(s[c] - mx) / l;
            const double ds = al * (dp[c] - delta);
            const int64_t krow = ((b * N + keys[c]) * M + m) * D;
            const int64_t kt = keys[c] / HW;
            const int64_t okrow = ((b * NR + keys[c] - t0 * HW) * M + m) * D;
            for (int64_t d = 0; d < D; ++d) {
              dq[orow + d] += p->scale * ds * wa_ld(k, p->bf16, krow + d);
              if (kt < t0 || kt >= t1) continue;
              const double addk = p->scale * ds * wa_ld(q, p->bf16, qrow + d);
              const double addv = al * wa_ld(dout, p->bf16, qrow + d);
#pragma omp atomic
              dk[okrow + d] += addk;
#pragma omp atomic
              dv[okrow + d] += addv;
            }
          }
        }
      }
    free(keys);
    free(s);
    free(dp);
  }
  return 0;
}
