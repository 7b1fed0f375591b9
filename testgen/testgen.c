/*
 * Seeded synthetic-input generator for the 3D-DSA parity tests and bench.
 *
 * Test infrastructure: it produces inputs only and holds none of the
 * operator's arithmetic.  Both the CPU oracle and the GPU library receive
 * exactly the arrays this file writes; neither side links it.
 *
 * Counter-based generation: element e of tensor `tid` under `seed` is a pure
 * function of (seed, tid, e), so any slab of a tensor can be regenerated on
 * its own (the full-scale grids do not fit in host memory all at once).
 *
 *   bits    = Philox4x32-10(counter = (lo32(e), hi32(e), tid, 0x44534133),
 *                           key     = (lo32(seed), hi32(seed)))
 *             as defined by Salmon, Moraes, Dror and Shaw, "Parallel random
 *             numbers: as easy as 1, 2, 3", SC'11 (round multipliers
 *             0xD2511F53 / 0xCD9E8D57, Weyl key increments 0x9E3779B9 /
 *             0xBB67AE85, ten rounds).
 *   u1, u2  = 53-bit uniforms in (0,1) from (bits0,bits1) and (bits2,bits3).
 *   normal  = mean + std * sqrt(-2 ln u1) * cos(2 pi u2)   (Box-Muller, fp64),
 *             then clipped to [lo, hi] and rounded to fp32.
 *   uniform = lo + (hi - lo) * u1, rounded to fp32.
 *   bf16    = round-to-nearest-even of the fp32 value.
 *
 * Build: gcc -O3 -fopenmp -shared -fPIC testgen.c -o libtestgen.so -lm
 */
#include <math.h>
#include <stdint.h>
#include <string.h>

#define PHILOX_M0 0xD2511F53u
#define PHILOX_M1 0xCD9E8D57u
#define PHILOX_W0 0x9E3779B9u
#define PHILOX_W1 0xBB67AE85u

static inline void philox_round(uint32_t c[4], const uint32_t k[2]) {
  uint64_t p0 = (uint64_t)PHILOX_M0 * c[0];
  uint64_t p1 = (uint64_t)PHILOX_M1 * c[2];
  uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
  uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
  uint32_t n0 = hi1 ^ c[1] ^ k[0];
  uint32_t n2 = hi0 ^ c[3] ^ k[1];
  c[0] = n0;
  c[1] = lo1;
  c[2] = n2;
  c[3] = lo0;
}

/* Philox4x32-10: ten rounds, key bumped between rounds. */
static inline void philox10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4]) {
  uint32_t c[4] = {ctr[0], ctr[1], ctr[2], ctr[3]};
  uint32_t k[2] = {key[0], key[1]};
  for (int r = 0; r < 10; ++r) {
    if (r) {
      k[0] += PHILOX_W0;
      k[1] += PHILOX_W1;
    }
    philox_round(c, k);
  }
  memcpy(out, c, sizeof(c));
}

void tg_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4]) {
  philox10(ctr, key, out);
}

#define TG_STREAM_TAG 0x44534133u

static inline void element_bits(uint64_t seed, uint32_t tid, uint64_t e, uint32_t r[4]) {
  uint32_t ctr[4] = {(uint32_t)e, (uint32_t)(e >> 32), tid, TG_STREAM_TAG};
  uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
  philox10(ctr, key, r);
}

static inline double unit_open(uint32_t a, uint32_t b) {
  uint64_t x = (((uint64_t)a << 32) | b) >> 11; /* 53 bits */
  return ((double)x + 0.5) * (1.0 / 9007199254740992.0);
}

static inline uint16_t f32_to_bf16_rne(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  if ((u & 0x7f800000u) == 0x7f800000u && (u & 0x007fffffu)) return (uint16_t)((u >> 16) | 0x40u);
  uint32_t lsb = (u >> 16) & 1u;
  u += 0x7fffu + lsb;
  return (uint16_t)(u >> 16);
}

static inline void store(void* out, int bf16, uint64_t i, float f) {
  if (bf16)
    ((uint16_t*)out)[i] = f32_to_bf16_rne(f);
  else
    ((float*)out)[i] = f;
}

/* dist: 0 = normal(a = mean, b = std), 1 = uniform[a, b).
 * Values are clipped to [lo, hi] (pass +-INFINITY for none).
 * out_bf16: 0 = write fp32, 1 = write bf16 (RNE of the fp32 value).
 * Writes out[i] = element (start + i) for i in [0, count). */
void tg_fill(uint64_t seed, uint32_t tid, uint64_t start, uint64_t count, int dist, double a, double b,
             double lo, double hi, int out_bf16, void* out) {
  const double two_pi = 6.283185307179586476925286766559;
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < (int64_t)count; ++i) {
    uint32_t r[4];
    element_bits(seed, tid, start + (uint64_t)i, r);
    double u1 = unit_open(r[0], r[1]);
    double x;
    if (dist == 0) {
      double u2 = unit_open(r[2], r[3]);
      x = a + b * (sqrt(-2.0 * log(u1)) * cos(two_pi * u2));
    } else {
      x = a + (b - a) * u1;
    }
    if (x < lo) x = lo;
    if (x > hi) x = hi;
    store(out, out_bf16, (uint64_t)i, (float)x);
  }
}

/* Round an fp32 array to bf16 (RNE); used to build bf16 copies of test data. */
void tg_f32_to_bf16(const float* in, uint16_t* out, uint64_t count) {
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < (int64_t)count; ++i) out[i] = f32_to_bf16_rne(in[i]);
}
