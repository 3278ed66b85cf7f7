/* Counter-based synthetic gradient generator (input plumbing only).
 *
 * Every value is a pure function of (stream key, element index), so any slice
 * of any worker's gradient can be produced independently and in any order.
 * The arithmetic uses only integer operations and IEEE-754 double +, -, *, /
 * and sqrt (all correctly rounded), evaluated in a fixed order with no
 * contraction, so the same source compiled for another IEEE target gives the
 * same bits.  The includer defines GG_FN (e.g. "static inline").
 *
 *  - SplitMix64 (Steele, Lea, Flood, OOPSLA 2014) as a hash of a 64-bit counter.
 *  - uniform on (0,1): 53 random bits, offset by half a step.
 *  - normal: Marsaglia & Bray's polar method (1964); attempt a of element x uses
 *    counters 64 x + 2a and 64 x + 2a + 1.
 *  - natural log: exact binary exponent split, then 2 atanh((m-1)/(m+1)) by its
 *    odd power series (11 terms, |s| <= 0.1716, relative error < 1e-16).
 *  - Laplace(0, b): inverse CDF.
 *  - Student-t(3): Z / sqrt((Z1^2 + Z2^2 + Z3^2) / 3) from four normals.
 */
#ifndef GRADGEN_H
#define GRADGEN_H

#include <stdint.h>

#ifndef GG_FN
#define GG_FN static inline
#endif

#define GG_GOLDEN 0x9E3779B97F4A7C15ULL

enum { GG_NORMAL = 0, GG_LAPLACE = 1, GG_STUDENT_T3 = 2 };

GG_FN uint64_t gg_mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
  return z ^ (z >> 31);
}

/* i-th output of the SplitMix64 sequence seeded with `key` */
GG_FN uint64_t gg_hash(uint64_t key, uint64_t counter) {
  return gg_mix64(key + (counter + 1ULL) * GG_GOLDEN);
}

GG_FN double gg_uniform(uint64_t h) {
  return ((double)(h >> 11) + 0.5) * (1.0 / 9007199254740992.0); /* 2^-53 */
}

/* ln(x) for finite x > 0 (normal range) */
GG_FN double gg_log(double x) {
  union { double d; uint64_t u; } v;
  v.d = x;
  int64_t e = (int64_t)((v.u >> 52) & 0x7FF) - 1022;   /* x = m 2^e, m in [0.5, 1) */
  v.u = (v.u & 0x800FFFFFFFFFFFFFULL) | 0x3FE0000000000000ULL;
  double m = v.d;
  if (m < 0.70710678118654752) { m = m * 2.0; e = e - 1; }
  double s = (m - 1.0) / (m + 1.0);
  double s2 = s * s;
  double p = 1.0 / 21.0;
  p = p * s2 + 1.0 / 19.0;
  p = p * s2 + 1.0 / 17.0;
  p = p * s2 + 1.0 / 15.0;
  p = p * s2 + 1.0 / 13.0;
  p = p * s2 + 1.0 / 11.0;
  p = p * s2 + 1.0 / 9.0;
  p = p * s2 + 1.0 / 7.0;
  p = p * s2 + 1.0 / 5.0;
  p = p * s2 + 1.0 / 3.0;
  p = p * s2 + 1.0;
  double lnm = 2.0 * s * p;
  return (double)e * 0.69314718055994531 + lnm;
}

GG_FN double gg_normal(uint64_t key, uint64_t x) {
  for (uint64_t a = 0; a < 32; ++a) {
    double v1 = 2.0 * gg_uniform(gg_hash(key, 64ULL * x + 2ULL * a)) - 1.0;
    double v2 = 2.0 * gg_uniform(gg_hash(key, 64ULL * x + 2ULL * a + 1ULL)) - 1.0;
    double s = v1 * v1 + v2 * v2;
    if (s > 0.0 && s < 1.0) {
      double f = -2.0 * gg_log(s) / s;
      return v1 * __builtin_sqrt(f);
    }
  }
  return 0.0;
}

GG_FN double gg_laplace(uint64_t key, uint64_t x) {
  double t = gg_uniform(gg_hash(key, x)) - 0.5;
  double a = t < 0.0 ? -t : t;
  double mag = -gg_log(1.0 - 2.0 * a);
  return t < 0.0 ? -mag : mag;
}

GG_FN double gg_student_t3(uint64_t key, uint64_t x) {
  double z = gg_normal(gg_mix64(key + 1ULL), x);
  double z1 = gg_normal(gg_mix64(key + 2ULL), x);
  double z2 = gg_normal(gg_mix64(key + 3ULL), x);
  double z3 = gg_normal(gg_mix64(key + 4ULL), x);
  double chi = (z1 * z1 + z2 * z2 + z3 * z3) / 3.0;
  return z / __builtin_sqrt(chi);
}

/* One gradient value: scale * draw, zeroed with probability zero_prob. */
GG_FN float gg_value(uint64_t key, uint64_t x, int dist, double scale, double zero_prob) {
  if (zero_prob > 0.0) {
    double u = gg_uniform(gg_hash(gg_mix64(key + 101ULL), x));
    if (u < zero_prob) return 0.0f;
  }
  double d;
  if (dist == GG_LAPLACE) d = gg_laplace(key, x);
  else if (dist == GG_STUDENT_T3) d = gg_student_t3(key, x);
  else d = gg_normal(key, x);
  return (float)(scale * d);
}

#endif
