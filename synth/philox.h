/*
 * Seeded synthetic-input generator shared by the host (gcc) and the device
 * (hipcc) builds.  Test and benchmark infrastructure only: it produces the
 * base weights and expert deltas, and holds none of the merge arithmetic.
 *
 * Counter-based: the value of element i of a tensor depends only on
 * (seed, stream, i), so any element can be regenerated on its own.  Every
 * floating-point step is an IEEE-754 binary64 add, multiply or divide in a
 * fixed order (both builds use -ffp-contract=off), so the host and device
 * builds produce identical bits.
 *
 * Bit source: Philox4x32-10 (Salmon, Moraes, Dror, Shaw, "Parallel random
 * numbers: as easy as 1, 2, 3", SC'11): round function
 *   (c0,c1,c2,c3) -> (hi(M1*c2)^c1^k0, lo(M1*c2), hi(M0*c0)^c3^k1, lo(M0*c0))
 * with M0=0xD2511F53, M1=0xCD9E8D57, Weyl key increments 0x9E3779B9 and
 * 0xBB67AE85 between the ten rounds.
 *
 * Transforms:
 *  - normal: the classic sum-of-twelve-uniforms approximation (Irwin-Hall,
 *    n=12, unit variance, support [-6,6]) built from 24-bit uniforms; the sum
 *    is formed exactly in integers and rescaled exactly, one rounding at the
 *    final multiply by sigma.
 *  - laplace: random sign times an exponential magnitude -b*ln(U); ln is the
 *    module's own (exponent split plus the atanh series), so no libm enters.
 *  - exact zeros: element is zero when an independent 32-bit word falls below
 *    zero_thresh (probability zero_thresh/2^32).
 * The value is then rounded to the storage type (fp32 by the IEEE cast,
 * bf16 by round-to-nearest-even of that fp32).
 */
#ifndef SYNTH_PHILOX_H
#define SYNTH_PHILOX_H

#include <stdint.h>
#include <string.h>

/* One header, compiled by both the host C compiler and hipcc. */
#if defined(__HIPCC__)
#define SYNTH_FN __host__ __device__ static inline
#else
#define SYNTH_FN static inline
#endif

enum { SYNTH_DIST_NORMAL = 0, SYNTH_DIST_LAPLACE = 1, SYNTH_DIST_ZERO = 2 };
enum { SYNTH_F32 = 0, SYNTH_BF16 = 1 };

typedef struct synth_recipe {
  uint32_t seed;        /* Philox key word 0 */
  uint32_t stream;      /* Philox key word 1: one value per (tensor, role) */
  uint32_t dist;        /* SYNTH_DIST_* */
  uint32_t zero_thresh; /* P(exact zero) = zero_thresh / 2^32 */
  double scale;         /* sigma (normal) or b (laplace) */
} synth_recipe;

typedef struct { uint32_t v[4]; } synth_u32x4;

SYNTH_FN synth_u32x4 synth_philox4x32_10(synth_u32x4 c, uint32_t k0, uint32_t k1) {
  for (int r = 0; r < 10; ++r) {
    if (r > 0) { k0 += 0x9E3779B9u; k1 += 0xBB67AE85u; }
    uint64_t p0 = (uint64_t)0xD2511F53u * (uint64_t)c.v[0];
    uint64_t p1 = (uint64_t)0xCD9E8D57u * (uint64_t)c.v[2];
    synth_u32x4 n;
    n.v[0] = (uint32_t)(p1 >> 32) ^ c.v[1] ^ k0;
    n.v[1] = (uint32_t)p1;
    n.v[2] = (uint32_t)(p0 >> 32) ^ c.v[3] ^ k1;
    n.v[3] = (uint32_t)p0;
    c = n;
  }
  return c;
}

SYNTH_FN synth_u32x4 synth_draw(const synth_recipe* r, uint64_t i, uint32_t j) {
  synth_u32x4 c;
  c.v[0] = (uint32_t)i; c.v[1] = (uint32_t)(i >> 32); c.v[2] = j; c.v[3] = 0u;
  return synth_philox4x32_10(c, r->seed, r->stream);
}

SYNTH_FN uint64_t synth_bits_f64(double x) { uint64_t b; memcpy(&b, &x, 8); return b; }
SYNTH_FN double synth_f64_bits(uint64_t b) { double x; memcpy(&x, &b, 8); return x; }

/* Natural log of a positive normal double: x = m*2^e with m in [sqrt(1/2), sqrt(2)),
 * ln m = 2*atanh(s), s = (m-1)/(m+1), |s| < 0.1716; the series is cut after s^23,
 * whose truncation error is below 1e-19.  Deterministic, not correctly rounded. */
SYNTH_FN double synth_log(double x) {
  uint64_t b = synth_bits_f64(x);
  int e = (int)((b >> 52) & 0x7FF) - 1023;
  double m = synth_f64_bits((b & 0x000FFFFFFFFFFFFFull) | 0x3FF0000000000000ull);
  if (m > 1.4142135623730951) { m = m * 0.5; e = e + 1; }
  double s = (m - 1.0) / (m + 1.0);
  double z = s * s;
  double p = 2.0 / 23.0;
  p = 2.0 / 21.0 + z * p;
  p = 2.0 / 19.0 + z * p;
  p = 2.0 / 17.0 + z * p;
  p = 2.0 / 15.0 + z * p;
  p = 2.0 / 13.0 + z * p;
  p = 2.0 / 11.0 + z * p;
  p = 2.0 / 9.0 + z * p;
  p = 2.0 / 7.0 + z * p;
  p = 2.0 / 5.0 + z * p;
  p = 2.0 / 3.0 + z * p;
  p = 2.0 + z * p;
  return (double)e * 0.69314718055994530942 + s * p;
}

/* Value of element i before storage rounding. */
SYNTH_FN double synth_value(const synth_recipe* r, uint64_t i) {
  if (r->dist == SYNTH_DIST_ZERO) return 0.0;
  if (r->zero_thresh != 0u) {
    synth_u32x4 z = synth_draw(r, i, 3u);
    if (z.v[0] < r->zero_thresh) return 0.0;
  }
  if (r->dist == SYNTH_DIST_LAPLACE) {
    synth_u32x4 a = synth_draw(r, i, 0u);
    /* U in (0,1) from 53 bits, never 0 or 1 */
    uint64_t m53 = ((uint64_t)(a.v[1] >> 5) << 26) | (uint64_t)(a.v[2] >> 6);
    double u = ((double)m53 + 0.5) * 0x1p-53;
    double mag = -(r->scale * synth_log(u));
    return (a.v[0] & 1u) ? -mag : mag;
  }
  /* normal: twelve 24-bit uniforms (k+0.5)*2^-24, summed exactly */
  uint32_t s = 0u;
  for (uint32_t j = 0; j < 3u; ++j) {
    synth_u32x4 a = synth_draw(r, i, j);
    s += (a.v[0] >> 8) + (a.v[1] >> 8) + (a.v[2] >> 8) + (a.v[3] >> 8);
  }
  double z = (double)(s + 6u) * 0x1p-24 - 6.0;
  return z * r->scale;
}

SYNTH_FN uint32_t synth_f32_bits(float f) { uint32_t b; memcpy(&b, &f, 4); return b; }

SYNTH_FN uint16_t synth_bf16_from_f64(double x) {
  uint32_t b = synth_f32_bits((float)x);
  return (uint16_t)((b + 0x7FFFu + ((b >> 16) & 1u)) >> 16);
}

SYNTH_FN float synth_f32_from_f64(double x) { return (float)x; }

#endif /* SYNTH_PHILOX_H */
