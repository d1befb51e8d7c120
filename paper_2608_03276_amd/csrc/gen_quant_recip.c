// Writes quant_recip_table.h: for every code format, the ulp adjustments of the reciprocal
// table that let the quantiser form each code without the correction step of the quotient.
//
// For an absmax A = m * 2^E with bf16 significand m = 1 + t/128, gamma = fl32(m/qmax) * 2^E
// and the code of a value v is clamp(RNE(fl32(v / gamma)), -qmax, qmax) for b-bit integers,
// or the OCP E4M3 code of fl32(v / gamma) (nearest, ties to even, saturating at 448) (Eq. 2).
// Power-of-two scalings are exact, so only the significands of A and v matter.  With a
// multiplier y'[t] near 1/fl32(m/qmax) the one-multiply forms are
//   qmax = 127 (int8):  fma(v, y' * 2^-E, 1.5 * 2^23), one rounding of the exact product onto
//                       the integer grid (the code sits in the low mantissa bits);
//   other integers:     fl32(v * y' * 2^-E) + 1.5 * 2^23, the product rounded to fp32, then to
//                       an integer (no clamp: the value must already be in range);
//   E4M3 (qmax = 448):  the E4M3 code of fl32(v * y' * 2^-E) clamped to +-448.
// y'[t] starts at fl32(1/fl32(m/qmax)) and moves by whole ulps (0, +1, -1) until the code
// equals the reference for every bf16 v with |v| <= A, both signs.  Where no such y' exists
// (a tie of the correctly rounded quotient that one rounding of v * y' cannot reproduce) the
// significand is marked, and the quantiser uses the corrected quotient for it.  The table is
// three 128-bit masks per format: up (+1 ulp), down (-1 ulp), none (no multiplier).
//
// --replay re-runs, on the CPU, the exact arithmetic of every path the quantiser can take
// for a row (quant_row.h), over every absmax A (every bf16 exponent field and significand)
// and every bf16 value v with |v| <= A, both signs, for every format, against the correctly
// rounded code; it prints the number of codes compared and of mismatches per path and exits
// 1 on any mismatch.  The paths: the one-multiply forms above (where the table holds a
// multiplier; absmax exponent field in [77, 240]); the corrected quotient of that range,
// q0 = v*y, q = fl(q0 + fma(-q0, gamma, v)*y), a residual correction of the reciprocal
// product in the manner of Markstein's division sequences ("IA-64 and elementary
// functions", 2000); the rescaled form of every row whose wave holds a row outside that
// range (the row scaled by 2^-e, the same correction against gamma*2^-e); and the IEEE
// division of rows with an absmax below 2^-100.  gamma itself is compared too.
//
//   gcc -O2 -fopenmp -ffp-contract=off -o gen gen_quant_recip.c -lm
//   ./gen > quant_recip_table.h       (write the table)
//   ./gen --check quant_recip_table.h (re-derive and compare with a written table; exit 1 on
//                                      any difference)
//   ./gen --replay [qmax]             (exhaustive replay of the kernel arithmetic, for every
//                                      format or the one with this qmax; exit 1 on any code
//                                      that differs)
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

static float from_bits(uint32_t b) {
  float f;
  memcpy(&f, &b, 4);
  return f;
}
static uint32_t to_bits(float f) {
  uint32_t b;
  memcpy(&b, &f, 4);
  return b;
}
static float bf16(uint32_t h) { return from_bits(h << 16); }

#define NFMT 8
static const float kQmax[NFMT] = {1, 3, 7, 15, 31, 63, 127, 448};
static const float kMagic = 12582912.0f;  // 1.5 * 2^23

// OCP E4M3 code of y clamped to +-448: nearest, ties to even, subnormals kept, sign kept.
static uint32_t e4m3(float y) {
  if (y > 448.0f) y = 448.0f;
  if (y < -448.0f) y = -448.0f;
  const uint32_t b = to_bits(y), sign = (b >> 24) & 0x80u, a = b & 0x7FFFFFFFu;
  const float af = from_bits(a);
  uint32_t code;
  if (af < 0.015625f) {
    code = (uint32_t)rintf(af * 512.0f);
  } else {
    const uint32_t r = a + 0x7FFFFu + ((a >> 20) & 1u);
    code = (((r >> 23) - 120u) << 3) | ((r >> 20) & 7u);
  }
  return sign | code;
}

static int reference_int(float v, float g, float qmax) {
  float c = rintf(v / g);  // IEEE single division, then round to nearest even
  if (c > qmax) c = qmax;
  if (c < -qmax) c = -qmax;
  return (int)c;
}

static int holds(int f, int t, float g, float y) {
  const float qmax = kQmax[f];
  const uint32_t top = (127u << 7) | (uint32_t)t;  // A = (1 + t/128) * 2^0
  for (uint32_t h = 0; h <= top; ++h)
    for (int s = 0; s < 2; ++s) {
      const float v = bf16(h | (s ? 0x8000u : 0u));
      if (qmax == 448.0f) {
        if (e4m3(v / g) != e4m3(v * y)) return 0;
      } else if (qmax == 127.0f) {
        const int code = (int)(int8_t)(to_bits(fmaf(v, y, kMagic)) & 0xFFu);
        if (code != reference_int(v, g, qmax)) return 0;
      } else {
        const float q = v * y;  // rounded to fp32 (no contraction: -ffp-contract=off)
        if ((int)rintf(q) != reference_int(v, g, qmax)) return 0;
      }
    }
  return 1;
}

// offs[f][t] in {-1, 0, 1}, or 2 where no multiplier within one ulp works
static void derive(int offs[NFMT][128]) {
  for (int f = 0; f < NFMT; ++f)
    for (int t = 0; t < 128; ++t) {
      const float g = (1.0f + (float)t * 0.0078125f) / kQmax[f];
      const uint32_t y0 = to_bits(1.0f / g);
      offs[f][t] = 2;
      const int cand[3] = {0, 1, -1};
      for (int k = 0; k < 3; ++k)
        if (holds(f, t, g, from_bits(y0 + (uint32_t)cand[k]))) {
          offs[f][t] = cand[k];
          break;
        }
    }
}

// ------------------------------------------------------------------ replay of the kernels
// Exponent fields of the absmax whose rows take the table paths, and below which a row is
// divided directly (quant_row.h: kFastExpLo, kFastExpHi; ef <= 27).
#define FAST_LO 77
#define FAST_HI 240
#define DIVIDE_MAX 27
enum { P_MUL, P_CORR, P_SCALED, P_DIV, P_GAMMA, NPATH };
static const char* kPathName[NPATH] = {"one-multiply", "corrected quotient", "rescaled row", "divided row",
                                       "gamma of the table"};

static float clampf(float x, float lo, float hi) { return x < lo ? lo : (x > hi ? hi : x); }

// integer code held in the low mantissa bits of y + 1.5 * 2^23, as a full integer
static int magic_int(float y_plus_magic) { return (int)(to_bits(y_plus_magic) - to_bits(kMagic)); }

// Per-(format, absmax) constants of the paths, as the kernels form them.
struct RowConsts {
  int fast, has_mul, divided;
  float gamma_c, ys_c, ysm_c;  // table paths: gamma, 1/gamma and the one-multiply multiplier, scaled
  float sc, gs, ys_s;          // rescaled row: 2^-e, gamma * 2^-e and its reciprocal
  float gamma;                 // fl32(absmax / qmax)
};

// The codes of every path the row takes for one value v, compared with the correctly rounded
// code ref: bit p of the result is set when path p differs.
static inline unsigned replay_one(int e4, float qmax, const struct RowConsts* r, float v, int ref) {
  unsigned bad = 0;
  if (r->fast) {
    const float q0 = v * r->ys_c;
#ifdef REPLAY_PLANT_UNCORRECTED
    const float q = q0;  // a planted mistake (tests only): the correction step dropped
#else
    const float q = fmaf(fmaf(-q0, r->gamma_c, v), r->ys_c, q0);
#endif
    const int c = e4 ? (int)e4m3(copysignf(clampf(q, -448.0f, 448.0f), v)) : magic_int(q + kMagic);
    bad |= (unsigned)(c != ref) << P_CORR;
    if (r->has_mul) {
      int cm;
      if (e4)
        cm = (int)e4m3(copysignf(clampf(v * r->ysm_c, -448.0f, 448.0f), v));
      else if (qmax == 127.0f)
        cm = magic_int(fmaf(v, r->ysm_c, kMagic));
      else
        cm = magic_int((v * r->ysm_c) + kMagic);  // two roundings (no contraction)
      bad |= (unsigned)(cm != ref) << P_MUL;
    }
  }
  if (!r->divided) {
    const float vs = v * r->sc;
    const float q0 = vs * r->ys_s;
    const float y = fmaf(fmaf(-q0, r->gs, vs), r->ys_s, q0);
    const int c = e4 ? (int)e4m3(copysignf(y, v)) : (int)clampf(rintf(y), -qmax, qmax);
    bad |= (unsigned)(c != ref) << P_SCALED;
  } else {
    int c;
    if (r->gamma == 0.0f)
      c = 0;  // an all-zero row: every code 0 (+0 for E4M3, whatever the sign of v)
    else
      c = e4 ? (int)e4m3(copysignf(v / r->gamma, v)) : (int)clampf(rintf(v / r->gamma), -qmax, qmax);
    bad |= (unsigned)(c != ref) << P_DIV;
  }
  return bad;
}

// only_qmax > 0 restricts the replay to that format
static int replay(int offs[NFMT][128], float only_qmax) {
  long long cnt[NFMT][NPATH], bad[NFMT][NPATH];
  memset(cnt, 0, sizeof cnt);
  memset(bad, 0, sizeof bad);
  for (int f = 0; f < NFMT; ++f) {
    if (only_qmax > 0.0f && kQmax[f] != only_qmax) continue;
    const float qmax = kQmax[f];
    const int e4 = qmax == 448.0f;
    long long c_f[NPATH] = {0}, b_f[NPATH] = {0};
#pragma omp parallel for schedule(dynamic, 1) reduction(+ : c_f[:NPATH], b_f[:NPATH])
    for (int ef = 0; ef < 255; ++ef) {
      for (int t = 0; t < 128; ++t) {
        const uint32_t abits = ((uint32_t)ef << 7) | (uint32_t)t;
        const float g_t = (1.0f + (float)t * 0.0078125f) / qmax;
        const float y_t = 1.0f / g_t;
        struct RowConsts r;
        r.fast = ef >= FAST_LO && ef <= FAST_HI;
        r.has_mul = offs[f][t] != 2;
        r.divided = ef <= DIVIDE_MAX;
        r.gamma_c = ldexpf(g_t, ef - 127);
        r.ys_c = ldexpf(y_t, 127 - ef);
        r.ysm_c = r.has_mul ? ldexpf(from_bits(to_bits(y_t) + (uint32_t)offs[f][t]), 127 - ef) : 0.0f;
        r.gamma = bf16(abits) / qmax;  // Eq. 2: fl32(absmax / qmax)
        r.sc = ldexpf(1.0f, 127 - ef);
        r.gs = r.gamma * r.sc;
        r.ys_s = 1.0f / r.gs;
        if (r.fast) {
          ++c_f[P_GAMMA];
          b_f[P_GAMMA] += to_bits(r.gamma_c) != to_bits(r.gamma);
        }
        long long nbad[NPATH] = {0};
        for (uint32_t h = 0; h <= abits; ++h)
          for (int sgn = 0; sgn < 2; ++sgn) {
            const float v = bf16(h | (sgn ? 0x8000u : 0u));
            int ref;
            if (r.gamma == 0.0f)
              ref = 0;  // Eq. 2 with gamma = 0: code 0 (the all-zero row's reading)
            else
              ref = e4 ? (int)e4m3(v / r.gamma) : reference_int(v, r.gamma, qmax);
            const unsigned b = replay_one(e4, qmax, &r, v, ref);
            if (b) {
              for (int p = 0; p < NPATH; ++p) nbad[p] += (b >> p) & 1u;
            }
          }
        const long long nv = 2 * ((long long)abits + 1);  // values of the row, both signs
        if (r.fast) c_f[P_CORR] += nv;
        if (r.fast && r.has_mul) c_f[P_MUL] += nv;
        c_f[r.divided ? P_DIV : P_SCALED] += nv;
        for (int p = 0; p < NPATH; ++p) b_f[p] += nbad[p];
      }
    }
    for (int p = 0; p < NPATH; ++p) {
      cnt[f][p] = c_f[p];
      bad[f][p] = b_f[p];
    }
  }
  int fail = 0;
  for (int f = 0; f < NFMT; ++f)
    for (int p = 0; p < NPATH; ++p) {
      if (only_qmax > 0.0f && kQmax[f] != only_qmax) continue;
      printf("qmax %g, %s: %lld compared, %lld differ\n", kQmax[f], kPathName[p], cnt[f][p], bad[f][p]);
      fail |= bad[f][p] != 0;
    }
  printf(fail ? "MISMATCH\n" : "ok\n");
  return fail;
}

// The encoder used above, against the OCP E4M3 value set: every bf16 magnitude up to 2^10
// goes to the nearest of the 127 finite non-negative E4M3 values, ties to the even code, and
// magnitudes at or above 448 to 448.
static int check_e4m3_encoder(void) {
  double val[127];
  for (int c = 0; c < 127; ++c) {
    const int e = c >> 3, m = c & 7;
    val[c] = e == 0 ? ldexp(m / 8.0, -6) : ldexp(1.0 + m / 8.0, e - 7);
  }
  for (uint32_t h = 0; h < 0x4480; ++h) {  // bf16 magnitudes [0, 1024)
    const double a = (double)bf16(h);
    int best = 0;
    for (int c = 1; c < 127; ++c) {
      const double d0 = fabs(a - val[best]), d1 = fabs(a - val[c]);
      if (d1 < d0 || (d1 == d0 && (c & 1) == 0)) best = c;
    }
    if (a >= 448.0) best = 126;
    if ((int)e4m3(bf16(h)) != best || (int)e4m3(bf16(h | 0x8000u)) != (best | 0x80)) {
      printf("E4M3 encoder differs at bf16 0x%04x\n", h);
      return 1;
    }
  }
  return 0;
}

int main(int argc, char** argv) {
  static int offs[NFMT][128];
  derive(offs);
  if (argc >= 2 && strcmp(argv[1], "--replay") == 0) {
    if (check_e4m3_encoder() != 0) return 1;
    return replay(offs, argc >= 3 ? (float)atof(argv[2]) : 0.0f);
  }
  uint64_t m[NFMT][3][2];
  int counts[NFMT][3];
  memset(m, 0, sizeof m);
  memset(counts, 0, sizeof counts);
  for (int f = 0; f < NFMT; ++f)
    for (int t = 0; t < 128; ++t) {
      const int o = offs[f][t];
      const int k = o == 1 ? 0 : o == -1 ? 1 : o == 2 ? 2 : -1;
      if (k >= 0) {
        m[f][k][t >> 6] |= 1ull << (t & 63);
        ++counts[f][k];
      }
    }
  if (counts[6][2] != 0) {
    fprintf(stderr, "int8 needs a multiplier for every significand\n");
    return 1;
  }
  if (argc == 3 && strcmp(argv[1], "--check") == 0) {
    FILE* fp = fopen(argv[2], "r");
    if (!fp) return 1;
    char line[512];
    uint64_t got[NFMT * 6];
    int n = 0;
    while (fgets(line, sizeof line, fp)) {
      char* p = line;
      while ((p = strstr(p, "0x")) != NULL) {
        const uint64_t b = strtoull(p, &p, 16);
        if (n < NFMT * 6) got[n] = b;
        ++n;
      }
    }
    fclose(fp);
    int bad = n != NFMT * 6;
    for (int f = 0; f < NFMT && !bad; ++f)
      for (int k = 0; k < 3; ++k)
        for (int h = 0; h < 2; ++h) bad |= got[f * 6 + k * 2 + h] != m[f][k][h];
    if (bad) {
      fprintf(stderr, "table differs (%d values read)\n", n);
      return 1;
    }
    for (int f = 0; f < NFMT; ++f)
      printf("qmax %g: %d up, %d down, %d without a multiplier\n", kQmax[f], counts[f][0], counts[f][1],
             counts[f][2]);
    printf("ok\n");
    return 0;
  }
  printf("// Generated by gen_quant_recip.c; do not edit.  Per code format (qmax), the significands\n");
  printf("// t of the absmax (m = 1 + t/128) whose one-multiply multiplier is fl32(1/fl32(m/qmax))\n");
  printf("// plus one ulp (up), minus one ulp (down), or does not exist (none: the corrected quotient\n");
  printf("// is used); bit t of word t/64.  qmax = 127 is the single-fma int8 form.\n");
  printf("#pragma once\n\n#include <stdint.h>\n\nnamespace tp {\n\n");
  printf("struct RecipMasks {\n  uint64_t up[2], down[2], none[2];\n};\n\n");
  printf("constexpr float kRecipQmax[%d] = {", NFMT);
  for (int f = 0; f < NFMT; ++f) printf("%s%g.0f", f ? ", " : "", kQmax[f]);
  printf("};\n");
  printf("constexpr RecipMasks kRecipMasks[%d] = {\n", NFMT);
  for (int f = 0; f < NFMT; ++f) {
    printf("    {{0x%016llxull, 0x%016llxull}, {0x%016llxull, 0x%016llxull}, {0x%016llxull, 0x%016llxull}},",
           (unsigned long long)m[f][0][0], (unsigned long long)m[f][0][1], (unsigned long long)m[f][1][0],
           (unsigned long long)m[f][1][1], (unsigned long long)m[f][2][0], (unsigned long long)m[f][2][1]);
    printf("  // qmax %g: %d up, %d down, %d none\n", kQmax[f], counts[f][0], counts[f][1], counts[f][2]);
  }
  printf("};\n\n}  // namespace tp\n");
  return 0;
}
