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
//   gcc -O2 -ffp-contract=off -o gen gen_quant_recip.c -lm
//   ./gen > quant_recip_table.h       (write the table)
//   ./gen --check quant_recip_table.h (re-derive and compare with a written table; exit 1 on
//                                      any difference)
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

int main(int argc, char** argv) {
  static int offs[NFMT][128];
  derive(offs);
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
