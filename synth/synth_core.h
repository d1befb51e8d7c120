/*
 * Seeded synthetic-input generator: the single definition that both the CPU
 * side (tests, the oracle's inputs) and the GPU side (full-size device
 * tensors) evaluate.  It holds none of the eviction method's arithmetic; it
 * only draws bf16 numbers.
 *
 * Every element is a pure function of (seed, tensor tag, sequence, layer,
 * head, token, dim), so any (layer, head, sequence) segment can be
 * regenerated on its own.  The definition uses only 64-bit integer ops and
 * IEEE-754 binary64 +, -, *, / and sqrt (all correctly rounded on both the
 * host and gfx950), with FP contraction disabled, so the host and device
 * builds produce bit-identical values.
 *
 * Building blocks (published definitions, re-implemented here):
 *  - SplitMix64 (Steele, Lea, Flood, "Fast splittable pseudorandom number
 *    generators", OOPSLA 2014): the n-th output of the stream seeded with s
 *    is mix(s + (n+1)*0x9E3779B97F4A7C15) with the Stafford "Mix13" finalizer.
 *  - Box-Muller transform (Box & Muller, 1958): z = sqrt(-2 ln u1) cos(2 pi u2).
 *    ln and cos are evaluated with fixed series (atanh series for ln, Taylor
 *    series for sin/cos after exact octant reduction), accurate to a few ulp,
 *    which is all a synthetic draw needs.
 *  - Student-t with nu = 3: z0 / sqrt((z1^2 + z2^2 + z3^2) / 3).
 *  - Outlier tokens: a keyed bijection of [0, 2^w) (odd multiply, add,
 *    xorshift rounds) restricted to [0, N) by cycle walking (Black & Rogaway,
 *    "Ciphers with arbitrary finite domains", CT-RSA 2002); token i is an
 *    outlier iff perm(i) < count, which marks exactly `count` tokens.
 *  - bf16 conversion: one round-to-nearest-even from binary64.
 */
#ifndef TP_SYNTH_CORE_H
#define TP_SYNTH_CORE_H

#include <stdint.h>

#if defined(__HIPCC__)
#define SYN_FN static inline __host__ __device__
#else
#define SYN_FN static inline
#endif

#if defined(__clang__)
#pragma clang fp contract(off)
#endif

#define SYN_GAMMA 0x9E3779B97F4A7C15ULL

enum { SYN_TAG_Q = 1, SYN_TAG_K = 2, SYN_TAG_V = 3, SYN_TAG_OUTLIER = 4, SYN_TAG_KG = 5, SYN_TAG_VG = 6 };
enum { SYN_DIST_NORMAL = 0, SYN_DIST_STUDENT_T3 = 1 };

SYN_FN uint64_t syn_mix(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
  return z ^ (z >> 31);
}

/* n-th output (n >= 0) of the SplitMix64 stream seeded with s. */
SYN_FN uint64_t syn_at(uint64_t s, uint64_t n) { return syn_mix(s + (n + 1) * SYN_GAMMA); }

/* Key of the (tag, seq, layer, head) stream. */
SYN_FN uint64_t syn_key(uint64_t seed, uint64_t tag, uint64_t seq, uint64_t layer, uint64_t head) {
  uint64_t k = syn_at(seed, tag);
  k = syn_at(k, seq);
  k = syn_at(k, layer);
  return syn_at(k, head);
}

SYN_FN double syn_bits_to_double(uint64_t b) {
  union { uint64_t u; double d; } c;
  c.u = b;
  return c.d;
}
SYN_FN uint64_t syn_double_to_bits(double d) {
  union { uint64_t u; double d; } c;
  c.d = d;
  return c.u;
}

/* Natural log of x in [2^-53, 1] (always a normal binary64 here). */
SYN_FN double syn_log(double x) {
  uint64_t b = syn_double_to_bits(x);
  int e = (int)((b >> 52) & 0x7FF) - 1023;
  double m = syn_bits_to_double((b & 0x000FFFFFFFFFFFFFULL) | 0x3FF0000000000000ULL); /* [1,2) */
  if (m > 1.4142135623730951) {
    m = m * 0.5;
    e = e + 1;
  }
  /* ln m = 2 atanh(t), t = (m-1)/(m+1), |t| <= 0.1716 */
  double t = (m - 1.0) / (m + 1.0);
  double t2 = t * t;
  double p = 1.0 / 27.0;
  p = p * t2 + 1.0 / 25.0;
  p = p * t2 + 1.0 / 23.0;
  p = p * t2 + 1.0 / 21.0;
  p = p * t2 + 1.0 / 19.0;
  p = p * t2 + 1.0 / 17.0;
  p = p * t2 + 1.0 / 15.0;
  p = p * t2 + 1.0 / 13.0;
  p = p * t2 + 1.0 / 11.0;
  p = p * t2 + 1.0 / 9.0;
  p = p * t2 + 1.0 / 7.0;
  p = p * t2 + 1.0 / 5.0;
  p = p * t2 + 1.0 / 3.0;
  p = p * t2 + 1.0;
  return (double)e * 0.6931471805599453 + 2.0 * t * p;
}

/* Taylor series on [0, pi/4]. */
SYN_FN double syn_cos_series(double x) {
  double x2 = x * x;
  double p = 1.0 / 6402373705728000.0; /* 1/18! */
  p = -p * x2 + 1.0 / 20922789888000.0; /* 1/16! */
  p = -p * x2 + 1.0 / 87178291200.0;    /* 1/14! */
  p = -p * x2 + 1.0 / 479001600.0;      /* 1/12! */
  p = -p * x2 + 1.0 / 3628800.0;        /* 1/10! */
  p = -p * x2 + 1.0 / 40320.0;          /* 1/8! */
  p = -p * x2 + 1.0 / 720.0;            /* 1/6! */
  p = -p * x2 + 1.0 / 24.0;             /* 1/4! */
  p = -p * x2 + 1.0 / 2.0;              /* 1/2! */
  p = -p * x2 + 1.0;
  return p;
}
SYN_FN double syn_sin_series(double x) {
  double x2 = x * x;
  double p = 1.0 / 355687428096000.0; /* 1/17! */
  p = -p * x2 + 1.0 / 1307674368000.0; /* 1/15! */
  p = -p * x2 + 1.0 / 6227020800.0;    /* 1/13! */
  p = -p * x2 + 1.0 / 39916800.0;      /* 1/11! */
  p = -p * x2 + 1.0 / 362880.0;        /* 1/9! */
  p = -p * x2 + 1.0 / 5040.0;          /* 1/7! */
  p = -p * x2 + 1.0 / 120.0;           /* 1/5! */
  p = -p * x2 + 1.0 / 6.0;             /* 1/3! */
  p = -p * x2 + 1.0;
  return x * p;
}

/* cos(2 pi w) for w in [0, 1), reduced exactly (Sterbenz) to [0, 1/8] turns. */
SYN_FN double syn_cos_turns(double w) {
  const double two_pi = 6.283185307179586;
  if (w >= 0.5) w = 1.0 - w;
  double sgn = 1.0;
  if (w > 0.25) {
    w = 0.5 - w;
    sgn = -1.0;
  }
  double r;
  if (w > 0.125)
    r = syn_sin_series(two_pi * (0.25 - w));
  else
    r = syn_cos_series(two_pi * w);
  return sgn * r;
}

SYN_FN double syn_sqrt(double x) {
#if defined(__HIP_DEVICE_COMPILE__)
  return __dsqrt_rn(x);
#else
  return __builtin_sqrt(x);
#endif
}

/* The m-th standard normal of a stream (Box-Muller on outputs 2m, 2m+1). */
SYN_FN double syn_normal(uint64_t key, uint64_t m) {
  uint64_t r1 = syn_at(key, 2 * m);
  uint64_t r2 = syn_at(key, 2 * m + 1);
  double u1 = (double)((r1 >> 11) + 1) * 0x1p-53; /* (0, 1] */
  double u2 = (double)(r2 >> 11) * 0x1p-53;       /* [0, 1) */
  return syn_sqrt(-2.0 * syn_log(u1)) * syn_cos_turns(u2);
}

/* Element e of a stream under the given distribution. */
SYN_FN double syn_draw(uint64_t key, int dist, uint64_t e) {
  if (dist == SYN_DIST_STUDENT_T3) {
    double z0 = syn_normal(key, 4 * e);
    double z1 = syn_normal(key, 4 * e + 1);
    double z2 = syn_normal(key, 4 * e + 2);
    double z3 = syn_normal(key, 4 * e + 3);
    double chi = z1 * z1 + z2 * z2 + z3 * z3;
    return z0 / syn_sqrt(chi / 3.0);
  }
  return syn_normal(key, e);
}

/* binary64 -> bf16 bits, one round-to-nearest-even (finite inputs). */
SYN_FN uint16_t syn_to_bf16(double x) {
  uint64_t b = syn_double_to_bits(x);
  uint16_t sign = (uint16_t)((b >> 48) & 0x8000);
  uint64_t a = b & 0x7FFFFFFFFFFFFFFFULL;
  double ax = syn_bits_to_double(a);
  if (ax < 0x1p-126) { /* below 2^-126: bf16 subnormal grid 2^-133 */
    double q = ax * 0x1p133; /* exact scaling */
    double fl = (double)(uint64_t)q;
    double fr = q - fl;
    uint64_t n = (uint64_t)fl;
    if (fr > 0.5 || (fr == 0.5 && (n & 1))) n += 1;
    return (uint16_t)(sign | (uint16_t)n);
  }
  a += 0x00000FFFFFFFFFFFULL + ((a >> 45) & 1);
  int e = (int)(a >> 52) - 1023 + 127;
  if (e >= 255) return (uint16_t)(sign | 0x7F80);
  return (uint16_t)(sign | ((uint16_t)e << 7) | (uint16_t)((a >> 45) & 0x7F));
}

/* Keyed bijection of [0, 2^w). */
SYN_FN uint64_t syn_perm_round(uint64_t x, uint64_t key, int w) {
  uint64_t mask = (w >= 64) ? ~0ULL : ((1ULL << w) - 1);
  int s = w / 2 + 1;
  for (int r = 0; r < 4; ++r) {
    uint64_t mul = syn_at(key, 2 * r) | 1ULL;
    uint64_t add = syn_at(key, 2 * r + 1);
    x = (x * mul + add) & mask;
    x ^= (x >> s);
  }
  return x;
}

/* Cycle-walking permutation of [0, n): perm(i) in [0, n). */
SYN_FN uint64_t syn_perm(uint64_t i, uint64_t n, uint64_t key) {
  int w = 0;
  while ((1ULL << w) < n) ++w;
  uint64_t x = syn_perm_round(i, key, w);
  while (x >= n) x = syn_perm_round(x, key, w);
  return x;
}

/* Number of outlier tokens in a sequence of n tokens: round-half-up(frac*n). */
SYN_FN uint64_t syn_outlier_count(double frac, uint64_t n) {
  if (!(frac > 0.0)) return 0;
  double c = frac * (double)n + 0.5;
  uint64_t r = (uint64_t)c;
  return r > n ? n : r;
}

typedef struct syn_spec {
  uint64_t seed;
  int32_t tag;       /* SYN_TAG_Q / K / V / KG / VG (the guide tokens' keys and values) */
  int32_t dist;      /* SYN_DIST_* */
  double out_frac;   /* fraction of tokens per (seq, layer, head) that are outliers; 0 = none */
  double out_scale;  /* factor applied to outlier rows before the bf16 rounding */
} syn_spec;

/* Multiplier of token t's row in the (seq, layer, head) row set of a sequence of n_seq tokens:
   out_scale for the round-half-up(out_frac * n_seq) outlier tokens, 1 otherwise. */
SYN_FN double syn_token_factor(const syn_spec* sp, uint64_t seq, uint64_t layer, uint64_t head,
                               uint64_t n_seq, uint64_t t) {
  if (!(sp->out_frac > 0.0)) return 1.0;
  uint64_t okey = syn_key(sp->seed, SYN_TAG_OUTLIER, seq, layer, head);
  uint64_t cnt = syn_outlier_count(sp->out_frac, n_seq);
  return syn_perm(t, n_seq, okey) < cnt ? sp->out_scale : 1.0;
}

/* bf16 bits of element (token t, dim c) of a row set with d elements per row, given the
   stream key syn_key(seed, tag, seq, layer, head) and the token's factor. */
SYN_FN uint16_t syn_element(uint64_t key, int dist, uint64_t t, uint64_t d, uint64_t c,
                            double factor) {
  double x = syn_draw(key, dist, t * d + c);
  if (factor != 1.0) x = x * factor;
  return syn_to_bf16(x);
}

#endif
