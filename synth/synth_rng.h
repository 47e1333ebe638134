/*
 * synth_rng.h -- counter-based generator for the synthetic workloads.
 *
 * This header holds input generation only: no step of the parameter-sync
 * method lives here.  It is compiled twice from this one source: by gcc for
 * the host library (libsynth_host.so, used to regenerate sampled inputs for
 * the oracle) and by hipcc for the device fill kernels (libsynth_dev.so, used
 * to fill multi-GB inputs in HBM).  Both builds must produce the same bits
 * for every (seed, stream, index).  To make that hold, every value is
 * computed from 64-bit integer hashing plus IEEE-754 double add, subtract,
 * multiply and divide only (each correctly rounded on both the x86-64 host
 * and gfx950), with floating-point contraction disabled on both compiles.
 * No libm call is made: log, cos and sqrt are evaluated below from their
 * series / Newton iterations.
 *
 * The includer defines SYNTH_FN before including this file
 * ("static inline" on the host, "__device__ static inline" on the device).
 *
 * Generator:
 *   mix64      -- the SplitMix64 output function (Steele, Lea, Flood,
 *                 "Fast splittable pseudorandom number generators",
 *                 OOPSLA 2014; constants as published by Vigna).
 *   stream key -- k = mix64(seed + GAMMA * (stream + 1))
 *   draw       -- h(i, sub) = mix64(k ^ (i * 8 + sub)), sub in 0..7
 *   uniform    -- (h >> 11) * 2^-53 in [0, 1)
 *   normal     -- Box-Muller, z = sqrt(-2 ln u1) * cos(2 pi u2),
 *                 u1 in (0, 1] from sub s, u2 in [0, 1) from sub s + 1.
 */
#ifndef SYNTH_RNG_H
#define SYNTH_RNG_H

#include <stdint.h>

#define SYNTH_GAMMA 0x9E3779B97F4A7C15ULL

SYNTH_FN uint64_t synth_mix64(uint64_t z) {
  z += SYNTH_GAMMA;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
  return z ^ (z >> 31);
}

SYNTH_FN uint64_t synth_stream_key(uint64_t seed, uint64_t stream) {
  return synth_mix64(seed + SYNTH_GAMMA * (stream + 1ULL));
}

SYNTH_FN uint64_t synth_draw(uint64_t key, uint64_t i, uint32_t sub) {
  return synth_mix64(key ^ ((i << 3) | (uint64_t)(sub & 7u)));
}

/* [0, 1) with 53 random bits */
SYNTH_FN double synth_u01(uint64_t h) {
  return (double)(h >> 11) * (1.0 / 9007199254740992.0);
}

/* (0, 1] with 53 random bits */
SYNTH_FN double synth_u01_open0(uint64_t h) {
  return (double)((h >> 11) + 1ULL) * (1.0 / 9007199254740992.0);
}

SYNTH_FN uint64_t synth_dbits(double x) {
  union { double d; uint64_t u; } c;
  c.d = x;
  return c.u;
}

SYNTH_FN double synth_bitsd(uint64_t u) {
  union { double d; uint64_t u; } c;
  c.u = u;
  return c.d;
}

/* Natural log for x in (0, 1], x normal.  x = m * 2^e with m in
 * [sqrt(1/2), sqrt(2)); ln m = 2 atanh(s), s = (m - 1) / (m + 1),
 * |s| <= 0.1716, series summed to s^27 (truncation < 1e-21 relative). */
SYNTH_FN double synth_log(double x) {
  uint64_t b = synth_dbits(x);
  int64_t e = (int64_t)((b >> 52) & 0x7FFULL) - 1023;
  double m = synth_bitsd((b & 0x000FFFFFFFFFFFFFULL) | 0x3FF0000000000000ULL);
  if (m > 1.4142135623730951) {
    m = m * 0.5;
    e = e + 1;
  }
  double s = (m - 1.0) / (m + 1.0);
  double s2 = s * s;
  double p = 0.037037037037037035;            /* 1/27 */
  p = p * s2 + 0.04;                          /* 1/25 */
  p = p * s2 + 0.043478260869565216;          /* 1/23 */
  p = p * s2 + 0.047619047619047616;          /* 1/21 */
  p = p * s2 + 0.05263157894736842;           /* 1/19 */
  p = p * s2 + 0.058823529411764705;          /* 1/17 */
  p = p * s2 + 0.06666666666666667;           /* 1/15 */
  p = p * s2 + 0.07692307692307693;           /* 1/13 */
  p = p * s2 + 0.09090909090909091;           /* 1/11 */
  p = p * s2 + 0.1111111111111111;            /* 1/9  */
  p = p * s2 + 0.14285714285714285;           /* 1/7  */
  p = p * s2 + 0.2;                           /* 1/5  */
  p = p * s2 + 0.3333333333333333;            /* 1/3  */
  p = p * s2 + 1.0;
  return (double)e * 0.6931471805599453 + 2.0 * s * p;
}

/* sin and cos of t for t in [0, pi/2], Taylor series to t^25 / t^24
 * (truncation below 1e-19). */
SYNTH_FN double synth_sin_q(double t) {
  double t2 = t * t;
  double p = -6.446950284384474e-26;          /* -1/25! */
  p = p * t2 + 3.8681701706306835e-23;        /*  1/23! */
  p = p * t2 - 1.9572941063391263e-20;        /* -1/21! */
  p = p * t2 + 8.22063524662433e-18;          /*  1/19! */
  p = p * t2 - 2.8114572543455206e-15;        /* -1/17! */
  p = p * t2 + 7.647163731819816e-13;         /*  1/15! */
  p = p * t2 - 1.6059043836821613e-10;        /* -1/13! */
  p = p * t2 + 2.505210838544172e-08;         /*  1/11! */
  p = p * t2 - 2.7557319223985893e-06;        /* -1/9!  */
  p = p * t2 + 0.0001984126984126984;         /*  1/7!  */
  p = p * t2 - 0.008333333333333333;          /* -1/5!  */
  p = p * t2 + 0.16666666666666666;           /*  1/3!  */
  p = p * t2 - 1.0;
  return -(t * p);
}

SYNTH_FN double synth_cos_q(double t) {
  double t2 = t * t;
  double p = 1.6117375710961184e-24;          /*  1/24! */
  p = p * t2 - 8.896791392450574e-22;         /* -1/22! */
  p = p * t2 + 4.110317623312165e-19;         /*  1/20! */
  p = p * t2 - 1.5619206968586225e-16;        /* -1/18! */
  p = p * t2 + 4.779477332387385e-14;         /*  1/16! */
  p = p * t2 - 1.1470745597729725e-11;        /* -1/14! */
  p = p * t2 + 2.08767569878681e-09;          /*  1/12! */
  p = p * t2 - 2.755731922398589e-07;         /* -1/10! */
  p = p * t2 + 2.48015873015873e-05;          /*  1/8!  */
  p = p * t2 - 0.001388888888888889;          /* -1/6!  */
  p = p * t2 + 0.041666666666666664;          /*  1/4!  */
  p = p * t2 - 0.5;                           /* -1/2!  */
  p = p * t2 + 1.0;
  return p;
}

/* cos(2 pi u) for u in [0, 1): quadrant from 4u, remainder angle in
 * [0, pi/2). */
SYNTH_FN double synth_cos2pi(double u) {
  double q = u * 4.0;              /* exact */
  int quad = (int)q;               /* 0..3 */
  double f = q - (double)quad;     /* exact */
  double t = f * 1.5707963267948966;
  switch (quad & 3) {
    case 0: return synth_cos_q(t);
    case 1: return -synth_sin_q(t);
    case 2: return -synth_cos_q(t);
    default: return synth_sin_q(t);
  }
}

/* sqrt for x >= 0 by Newton's iteration from a bit-level first guess
 * (relative error of the guess < 6.1 %, five iterations leave < 1e-30
 * truncation, so the result is within rounding of the true root). */
SYNTH_FN double synth_sqrt(double x) {
  if (!(x > 0.0)) return 0.0;
  double y = synth_bitsd((synth_dbits(x) >> 1) + 0x1FF8000000000000ULL);
  y = 0.5 * (y + x / y);
  y = 0.5 * (y + x / y);
  y = 0.5 * (y + x / y);
  y = 0.5 * (y + x / y);
  y = 0.5 * (y + x / y);
  return y;
}

/* Standard normal draw from subs (s, s + 1) at index i. */
SYNTH_FN double synth_normal(uint64_t key, uint64_t i, uint32_t s) {
  double u1 = synth_u01_open0(synth_draw(key, i, s));
  double u2 = synth_u01(synth_draw(key, i, s + 1u));
  double r = synth_sqrt(-2.0 * synth_log(u1));
  return r * synth_cos2pi(u2);
}

SYNTH_FN uint32_t synth_fbits(float x) {
  union { float f; uint32_t u; } c;
  c.f = x;
  return c.u;
}

/* fp32 -> bf16, round to nearest even (inputs here are finite). */
SYNTH_FN uint16_t synth_bf16(float x) {
  uint32_t u = synth_fbits(x);
  return (uint16_t)((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
}

/* ---- value kinds ------------------------------------------------------ */

enum {
  SYN_NORMAL_F32 = 1,   /* f32  = (float)(mean + std * z(stream))                   */
  SYN_NORMAL_BF16 = 2,  /* bf16 = rne((float)(mean + std * z(stream)))              */
  SYN_DRIFT_F32 = 3,    /* f32  = (float)((double)base + std2 * z(stream2)),
                           base = (float)(mean + std * z(stream))                   */
  SYN_DRIFT_BF16 = 4,   /* bf16 = rne(value of SYN_DRIFT_F32)                       */
  SYN_STUDENT3_BF16 = 5 /* bf16 = 0 when the uniform of sub 6 is below p_zero,
                           otherwise rne((float)(std * t3)), t3 = z0 /
                           sqrt((z1^2 + z2^2 + z3^2) / 3); z0..z2 from subs
                           (0,1), (2,3), (4,5); z3 from subs (0,1) of the key
                           mix64(key ^ 0xD1B54A32D192ED03)                      */
};

typedef struct {
  int32_t kind;
  int32_t pad_;
  uint64_t seed;
  uint64_t stream;
  uint64_t stream2;
  double mean;
  double std;
  double std2;
  double p_zero;
} synth_spec;

SYNTH_FN float synth_drift_f32(const synth_spec* sp, uint64_t k1, uint64_t k2,
                               uint64_t i) {
  float base = (float)(sp->mean + sp->std * synth_normal(k1, i, 0));
  return (float)((double)base + sp->std2 * synth_normal(k2, i, 0));
}

SYNTH_FN float synth_student3(const synth_spec* sp, uint64_t k1, uint64_t i) {
  double uz = synth_u01(synth_draw(k1, i, 6));
  if (uz < sp->p_zero) return 0.0f;
  uint64_t k3 = synth_mix64(k1 ^ 0xD1B54A32D192ED03ULL);
  double z0 = synth_normal(k1, i, 0);
  double z1 = synth_normal(k1, i, 2);
  double z2 = synth_normal(k1, i, 4);
  double z3 = synth_normal(k3, i, 0);
  double chi = (z1 * z1 + z2 * z2 + z3 * z3) / 3.0;
  return (float)(sp->std * (z0 / synth_sqrt(chi)));
}

#endif /* SYNTH_RNG_H */
