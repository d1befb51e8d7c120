// Per-token V quantisation of Eq. 2 (Sec. 3.3), shared by the quantisation kernel and the
// compaction kernel that quantises only the kept rows:
//   gamma_t = fl32(max_c |v_tc| / qmax)
//   q_tc    = clamp(RNE(fl32(v_tc / gamma_t)), -qmax, qmax)    (b-bit integers), or the OCP
//             E4M3 code of fl32(v_tc / gamma_t), RNE, saturating at 448; gamma_t = 0 gives 0.
//
// A token row of d bf16 values is held by LPT = d/8 consecutive lanes, 16 bytes each.  The
// absmax is an integer max of the bf16 magnitude bits (exact), reduced across those lanes
// with DPP row operations.
//
// Common path (every row of the wave has an absmax A in [2^-50, 2^114)): with A = m * 2^E,
// m the bf16 significand, gamma = fl32(m/qmax) * 2^E and y = fl32(1/fl32(m/qmax)) * 2^-E
// exactly (power-of-two scalings of normal numbers), both read from 128-entry tables per
// significand that the workgroup computes with IEEE divisions.
//  - One multiply, where the significand has a checked multiplier: quant_recip_table.h
//    marks, per format, a y'' within one ulp of 1/fl32(m/qmax) for which one multiply gives
//    every code of that significand (its generator checks every bf16 v, both signs).  int8:
//    fma(v, y'', 1.5 * 2^23), a single rounding of the exact product onto the integer grid,
//    whose two's complement sits in the low mantissa bits (every int8 significand has one);
//    other integers: fl32(v * y'') + 1.5 * 2^23; E4M3: the value fl32(v * y'').  A wave
//    takes this path when every row in it has such a multiplier.
//  - Corrected quotient otherwise: q0 = v * y, then fl(q0 + fma(-q0, gamma, v) * y), plus
//    1.5 * 2^23 for an integer code.  This is the residual correction of a reciprocal
//    product used in Markstein's division sequences (P. Markstein, "IA-64 and Elementary
//    Functions", 2000): the exact remainder v - q0*gamma comes from one fma, and one more
//    fma adds its scaled value back.  gen_quant_recip.c --replay re-runs this arithmetic
//    (and every other path below) over every (A, v) pair of bf16 values, both signs, for
//    every qmax of the supported formats: it gives the codes of the correctly rounded
//    quotient.
// No clamp is needed for integer codes since |v/gamma| < qmax + 1/2.  An E4M3 code is the
// hardware conversion of the value clamped to +-448 (it can exceed 448 by an ulp), with the
// sign of v.  Every intermediate that can decide a code is a normal number in this range.
// Other rows (tiny, zero or huge absmax) take the general path: the row is rescaled by
// 2^-e (e = exponent of the absmax), the same corrected quotient is formed against
// gamma' = gamma * 2^-e with one division per row, and the code is rounded and clamped
// explicitly; rows whose absmax is below 2^-100 use the IEEE division directly.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "taskpress.h"
#include "tp_internal.h"

namespace tp {

struct QuantFmt {
  bool int_fmt;  // b-bit integers (else fp8-e4m3)
  bool nibbles;  // int with b <= 4: two codes per byte, even element in the low nibble
  float qmax;
};

// Code formats, fixed per kernel instance: one integer code per byte (b in [5, 7]; int8 has
// its own instance for its single-rounding path), two per byte (b <= 4), or E4M3.
enum QKind { kQByte = 0, kQNibble = 1, kQE4M3 = 2, kQInt8 = 3 };

__host__ __device__ inline int qkind_of(int32_t qfmt, int32_t bits) {
  if (qfmt != TP_QFMT_INT) return kQE4M3;
  return bits <= 4 ? kQNibble : (bits == 8 ? kQInt8 : kQByte);
}

// gamma and 1/gamma of the significand m = 1 + t/128 of an absmax, for the common path.
struct QuantTables {
  float g[128];   // fl32(m / qmax)
  float y[128];   // fl32(1 / g)
  float ym[128];  // the one-multiply multiplier y'', or -1 where the significand has none
};

// All threads of the block call this, followed by a barrier before the first quant_piece.
// off: the ulp offsets of the one-multiply multipliers (recip_offsets_for(qmax)).
__device__ inline void build_tables(QuantTables& tab, float qmax, const int8_t* off) {
  for (int t = threadIdx.x; t < 128; t += blockDim.x) {
    const float g = (1.0f + (float)t * 0.0078125f) / qmax;
    const uint32_t y = __float_as_uint(1.0f / g);
    const int o = off[t];
    tab.g[t] = g;
    tab.y[t] = __uint_as_float(y);
    tab.ym[t] = o == kNoMultiplier ? -1.0f : __uint_as_float(y + (uint32_t)o);
  }
}

// Absmax exponent fields (bf16 = fp32 exponent field) of the common path: A in [2^-50, 2^114).
constexpr int kFastExpLo = 77;
constexpr int kFastExpHi = 240;
constexpr float kRoundMagic = 12582912.0f;  // 1.5 * 2^23

// max over the LPT (8 or 16) consecutive lanes of a DPP row segment.
template <int LPT>
__device__ inline uint32_t group_max(uint32_t x) {
  // quad_perm [1,0,3,2] and [2,3,0,1]: lanes xor 1, xor 2
  x = max(x, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0xB1, 0xF, 0xF, false));
  x = max(x, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x4E, 0xF, 0xF, false));
  // row_half_mirror: lane i <-> 7-i within each 8 (pairs the two quads of a half-row)
  x = max(x, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x141, 0xF, 0xF, false));
  if (LPT == 16) {
    // row_mirror: lane i <-> 15-i within each row of 16 (pairs the two half-rows)
    x = max(x, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x140, 0xF, 0xF, false));
  }
  return x;
}

// OCP E4M3 code of y: nearest value, ties to the even mantissa, |y| >= 448 -> 448, sign kept.
__device__ inline uint32_t e4m3_code(float y) {
  const uint32_t b = __float_as_uint(y);
  const uint32_t sign = (b >> 24) & 0x80u;
  const uint32_t a = b & 0x7FFFFFFFu;
  const float af = __uint_as_float(a);
  uint32_t code;
  if (af >= 448.0f) {
    code = 0x7Eu;
  } else if (af < 0.015625f) {  // below 2^-6: subnormal codes, step 2^-9 (8 = 2^-6)
    code = (uint32_t)__builtin_rintf(af * 512.0f);
  } else {  // round the 23-bit mantissa to 3 bits (RNE); a carry bumps the exponent
    const uint32_t r = a + 0x7FFFFu + ((a >> 20) & 1u);
    code = (((r >> 23) - 120u) << 3) | ((r >> 20) & 7u);
  }
  return sign | code;
}

// Codes of 8 values in the normalised domain (the quotient y of each, then the format's code).
// ys = 1/gs, sc = 2^-e; valid when the absmax exponent field exceeds 27.
__device__ inline void codes_scaled(const uint32_t (&w)[4], float sc, float gs, float ys, const QuantFmt& f,
                                    uint32_t (&code)[8]) {
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const uint32_t h = (i & 1) ? (w[i >> 1] & 0xFFFF0000u) : (w[i >> 1] << 16);
    const float v = __uint_as_float(h);
    const float vs = v * sc;
    const float q0 = vs * ys;
    const float y = fmaf(fmaf(-q0, gs, vs), ys, q0);
    if (f.int_fmt)
      code[i] = (uint32_t)(int32_t)__builtin_amdgcn_fmed3f(__builtin_rintf(y), -f.qmax, f.qmax);
    else
      code[i] = e4m3_code(__builtin_copysignf(y, v));
  }
}

// Codes by IEEE division (rows with a tiny or zero absmax).
__device__ inline void codes_divided(const uint32_t (&w)[4], float gamma, const QuantFmt& f, uint32_t (&code)[8]) {
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const uint32_t h = (i & 1) ? (w[i >> 1] & 0xFFFF0000u) : (w[i >> 1] << 16);
    const float v = __uint_as_float(h);
    const float y = v / gamma;
    if (gamma == 0.0f)
      code[i] = 0;
    else if (f.int_fmt)
      code[i] = (uint32_t)(int32_t)__builtin_amdgcn_fmed3f(__builtin_rintf(y), -f.qmax, f.qmax);
    else
      code[i] = e4m3_code(__builtin_copysignf(y, v));
  }
}

// Magnitude bits of the absmax of the row whose LPT pieces sit in LPT consecutive lanes (all
// lanes call together): an integer max of the bf16 magnitudes, reduced across the lanes.
// PACKED: two magnitudes per packed 16-bit max (fewer vector instructions beside the codes'
// arithmetic); the scales-only kernel keeps the 32-bit form, which measured faster there.
template <int LPT, bool PACKED = true>
__device__ inline uint32_t row_absmax_bits(const uint32_t (&w)[4]) {
  if (PACKED) {
    typedef unsigned short u16x2 __attribute__((ext_vector_type(2)));
    u16x2 m2 = {0, 0};
#pragma unroll
    for (int i = 0; i < 4; ++i) m2 = __builtin_elementwise_max(m2, __builtin_bit_cast(u16x2, w[i] & 0x7FFF7FFFu));
    return group_max<LPT>(max((uint32_t)m2.x, (uint32_t)m2.y));
  }
  uint32_t mx = 0;
#pragma unroll
  for (int i = 0; i < 4; ++i) mx = max(mx, max(w[i] & 0x7FFFu, (w[i] >> 16) & 0x7FFFu));
  return group_max<LPT>(mx);
}

// gamma alone (no codes).
template <int LPT>
__device__ inline float scale_piece(const uint4& x, const QuantFmt& f) {
  const uint32_t w[4] = {x.x, x.y, x.z, x.w};
  return __uint_as_float(row_absmax_bits<LPT, false>(w) << 16) / f.qmax;
}

// Codes of 8 values on the common path: y = v / gamma corrected as above; an integer code is
// the low bits of y + 1.5 * 2^23.
template <int K>
__device__ inline void codes_fast(const uint32_t (&w)[4], float gamma, float ys, uint32_t (&code)[8]) {
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const uint32_t h = (i & 1) ? (w[i >> 1] & 0xFFFF0000u) : (w[i >> 1] << 16);
    const float v = __uint_as_float(h);
    const float q0 = v * ys;
    const float y = fmaf(fmaf(-q0, gamma, v), ys, q0);
    code[i] = __float_as_uint(y + kRoundMagic);
  }
}

// int8 codes of 8 values on the common path: one rounding of the exact v * y'' to the integer
// grid, whose two's complement sits in the low bits of the result.
__device__ inline void codes_fast_int8(const uint32_t (&w)[4], float ys, uint32_t (&code)[8]) {
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const uint32_t h = (i & 1) ? (w[i >> 1] & 0xFFFF0000u) : (w[i >> 1] << 16);
    code[i] = __float_as_uint(fmaf(__uint_as_float(h), ys, kRoundMagic));
  }
}

// Other integer codes with a one-multiply multiplier: the product rounded to fp32, then to an
// integer by the add (two roundings, exactly as the table was checked; the multiply and the
// add must not be fused).
__device__ inline void codes_mul(const uint32_t (&w)[4], float ys, uint32_t (&code)[8]) {
#pragma clang fp contract(off)
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const uint32_t h = (i & 1) ? (w[i >> 1] & 0xFFFF0000u) : (w[i >> 1] << 16);
    const float q = __uint_as_float(h) * ys;
    code[i] = __float_as_uint(q + kRoundMagic);
  }
}

// E4M3 codes of 8 values on the common path, packed: the corrected quotient, clamped to
// +-448 (it can exceed 448 by an ulp), with the sign of v (so -0 keeps its sign), converted
// two at a time by the hardware fp32 -> OCP E4M3 conversion (nearest, ties to even,
// subnormals kept); element 2i in byte 2i.
__device__ inline uint2 codes_fast_e4m3(const uint32_t (&w)[4], float gamma, float ys) {
  float y[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const uint32_t h = (i & 1) ? (w[i >> 1] & 0xFFFF0000u) : (w[i >> 1] << 16);
    const float v = __uint_as_float(h);
    const float q0 = v * ys;
    const float q = fmaf(fmaf(-q0, gamma, v), ys, q0);
    y[i] = __builtin_copysignf(__builtin_amdgcn_fmed3f(q, -448.0f, 448.0f), v);
  }
  uint32_t lo = (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(y[0], y[1], 0, false);
  lo = (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(y[2], y[3], (int)lo, true);
  uint32_t hi = (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(y[4], y[5], 0, false);
  hi = (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(y[6], y[7], (int)hi, true);
  return make_uint2(lo, hi);
}

// E4M3 codes of 8 values with a one-multiply multiplier, packed as codes_fast_e4m3.
__device__ inline uint2 codes_mul_e4m3(const uint32_t (&w)[4], float ys) {
  float y[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const uint32_t h = (i & 1) ? (w[i >> 1] & 0xFFFF0000u) : (w[i >> 1] << 16);
    const float v = __uint_as_float(h);
    y[i] = __builtin_copysignf(__builtin_amdgcn_fmed3f(v * ys, -448.0f, 448.0f), v);
  }
  uint32_t lo = (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(y[0], y[1], 0, false);
  lo = (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(y[2], y[3], (int)lo, true);
  uint32_t hi = (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(y[4], y[5], 0, false);
  hi = (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(y[6], y[7], (int)hi, true);
  return make_uint2(lo, hi);
}

// Quantise the lane's 16-byte piece `x` (8 bf16 values) of a row whose LPT pieces sit in
// LPT consecutive lanes; every lane of the wave must call this together (the absmax is
// reduced across lanes, and the path is chosen per wave).  Returns gamma (the same on all
// LPT lanes of the row) and the piece's codes: 8 bytes in out.x, out.y, or 8 nibbles in out.x.
template <int LPT, int K>
__device__ inline float quant_piece(const uint4& x, const QuantTables& tab, const QuantFmt& f, uint2& out) {
  const uint32_t w[4] = {x.x, x.y, x.z, x.w};
  const uint32_t mx = row_absmax_bits<LPT>(w);
  const int ef = (int)(mx >> 7);
  uint32_t code[8];
  float gamma;
  if (__builtin_amdgcn_ballot_w64(ef < kFastExpLo || ef > kFastExpHi) == 0) {
    const int t = (int)(mx & 0x7Fu);
    gamma = __builtin_amdgcn_ldexpf(tab.g[t], ef - 127);
    const float ym = tab.ym[t];
    if (K == kQInt8) {  // every int8 significand has a multiplier
      codes_fast_int8(w, __builtin_amdgcn_ldexpf(ym, 127 - ef), code);
    } else if (__builtin_amdgcn_ballot_w64(!(ym > 0.0f)) == 0) {
      const float ys = __builtin_amdgcn_ldexpf(ym, 127 - ef);
      if (K == kQE4M3) {
        out = codes_mul_e4m3(w, ys);
        return gamma;
      }
      codes_mul(w, ys, code);
    } else {
      const float ys = __builtin_amdgcn_ldexpf(tab.y[t], 127 - ef);
      if (K == kQE4M3) {
        out = codes_fast_e4m3(w, gamma, ys);
        return gamma;
      }
      codes_fast<K>(w, gamma, ys, code);
    }
  } else {
    const float amax = __uint_as_float(mx << 16);
    gamma = amax / f.qmax;
    // below 2^-100 (zero rows included) the division path is taken, for the whole wave
    // when any lane needs it
    if (__builtin_amdgcn_ballot_w64(ef <= 27) == 0) {
      const float sc = __builtin_amdgcn_ldexpf(1.0f, 127 - ef);
      const float gs = gamma * sc;
      codes_scaled(w, sc, gs, 1.0f / gs, f, code);
    } else if (ef <= 27) {
      codes_divided(w, gamma, f, code);
    } else {
      const float sc = __builtin_amdgcn_ldexpf(1.0f, 127 - ef);
      const float gs = gamma * sc;
      codes_scaled(w, sc, gs, 1.0f / gs, f, code);
    }
  }
  if (K == kQNibble) {
    uint32_t p = 0;
#pragma unroll
    for (int i = 0; i < 8; ++i) p |= (code[i] & 0xFu) << (4 * i);
    out.x = p;
    out.y = 0;
  } else {
    // bytes 0 of (c0, c1, c2, c3) -> one dword, via two byte permutes and a word merge
    const uint32_t lo01 = __builtin_amdgcn_perm(code[1], code[0], 0x0c0c0400u);
    const uint32_t lo23 = __builtin_amdgcn_perm(code[3], code[2], 0x0c0c0400u);
    const uint32_t hi01 = __builtin_amdgcn_perm(code[5], code[4], 0x0c0c0400u);
    const uint32_t hi23 = __builtin_amdgcn_perm(code[7], code[6], 0x0c0c0400u);
    out.x = __builtin_amdgcn_perm(lo23, lo01, 0x05040100u);
    out.y = __builtin_amdgcn_perm(hi23, hi01, 0x05040100u);
  }
  return gamma;
}

// quant_piece for NP consecutive 16-byte pieces per lane (8 NP bf16 values; a row's D/8
// pieces in LPT = D/(8 NP) consecutive lanes): the same arithmetic and the same per-wave path
// choice, with the row's per-lane work (absmax reduction, table lookup, path tests) shared by
// the NP pieces.  Returns gamma and each piece's codes in out[n], as quant_piece.  The
// quantisation kernels keep quant_piece's own one-piece form: the lean kernel's register
// count, on which its fit beside the score passes depends, is that form's.
template <int LPT, int K, int NP>
__device__ inline float quant_pieces(const uint4 (&x)[NP], const QuantTables& tab, const QuantFmt& f,
                                     uint2 (&out)[NP]) {
  uint32_t w[NP][4];
  typedef unsigned short u16x2 __attribute__((ext_vector_type(2)));
  u16x2 m2 = {0, 0};  // the lane's largest magnitude, two per packed max
#pragma unroll
  for (int n = 0; n < NP; ++n) {
    w[n][0] = x[n].x;
    w[n][1] = x[n].y;
    w[n][2] = x[n].z;
    w[n][3] = x[n].w;
#pragma unroll
    for (int i = 0; i < 4; ++i) m2 = __builtin_elementwise_max(m2, __builtin_bit_cast(u16x2, w[n][i] & 0x7FFF7FFFu));
  }
  const uint32_t mx = group_max<LPT>(max((uint32_t)m2.x, (uint32_t)m2.y));
  const int ef = (int)(mx >> 7);
  uint32_t code[NP][8];
  float gamma;
  if (__builtin_amdgcn_ballot_w64(ef < kFastExpLo || ef > kFastExpHi) == 0) {
    const int t = (int)(mx & 0x7Fu);
    gamma = __builtin_amdgcn_ldexpf(tab.g[t], ef - 127);
    const float ym = tab.ym[t];
    if (K == kQInt8) {  // every int8 significand has a multiplier
      const float ys = __builtin_amdgcn_ldexpf(ym, 127 - ef);
#pragma unroll
      for (int n = 0; n < NP; ++n) codes_fast_int8(w[n], ys, code[n]);
    } else if (__builtin_amdgcn_ballot_w64(!(ym > 0.0f)) == 0) {
      const float ys = __builtin_amdgcn_ldexpf(ym, 127 - ef);
      if (K == kQE4M3) {
#pragma unroll
        for (int n = 0; n < NP; ++n) out[n] = codes_mul_e4m3(w[n], ys);
        return gamma;
      }
#pragma unroll
      for (int n = 0; n < NP; ++n) codes_mul(w[n], ys, code[n]);
    } else {
      const float ys = __builtin_amdgcn_ldexpf(tab.y[t], 127 - ef);
      if (K == kQE4M3) {
#pragma unroll
        for (int n = 0; n < NP; ++n) out[n] = codes_fast_e4m3(w[n], gamma, ys);
        return gamma;
      }
#pragma unroll
      for (int n = 0; n < NP; ++n) codes_fast<K>(w[n], gamma, ys, code[n]);
    }
  } else {
    const float amax = __uint_as_float(mx << 16);
    gamma = amax / f.qmax;
    // below 2^-100 (zero rows included) the division path is taken, for the whole wave
    // when any lane needs it
    if (__builtin_amdgcn_ballot_w64(ef <= 27) == 0) {
      const float sc = __builtin_amdgcn_ldexpf(1.0f, 127 - ef);
      const float gs = gamma * sc;
      const float ys = 1.0f / gs;
#pragma unroll
      for (int n = 0; n < NP; ++n) codes_scaled(w[n], sc, gs, ys, f, code[n]);
    } else if (ef <= 27) {
#pragma unroll
      for (int n = 0; n < NP; ++n) codes_divided(w[n], gamma, f, code[n]);
    } else {
      const float sc = __builtin_amdgcn_ldexpf(1.0f, 127 - ef);
      const float gs = gamma * sc;
      const float ys = 1.0f / gs;
#pragma unroll
      for (int n = 0; n < NP; ++n) codes_scaled(w[n], sc, gs, ys, f, code[n]);
    }
  }
#pragma unroll
  for (int n = 0; n < NP; ++n) {
    if (K == kQNibble) {
      uint32_t p = 0;
#pragma unroll
      for (int i = 0; i < 8; ++i) p |= (code[n][i] & 0xFu) << (4 * i);
      out[n].x = p;
      out[n].y = 0;
    } else {
      // bytes 0 of (c0, c1, c2, c3) -> one dword, via two byte permutes and a word merge
      const uint32_t lo01 = __builtin_amdgcn_perm(code[n][1], code[n][0], 0x0c0c0400u);
      const uint32_t lo23 = __builtin_amdgcn_perm(code[n][3], code[n][2], 0x0c0c0400u);
      const uint32_t hi01 = __builtin_amdgcn_perm(code[n][5], code[n][4], 0x0c0c0400u);
      const uint32_t hi23 = __builtin_amdgcn_perm(code[n][7], code[n][6], 0x0c0c0400u);
      out[n].x = __builtin_amdgcn_perm(lo23, lo01, 0x05040100u);
      out[n].y = __builtin_amdgcn_perm(hi23, hi01, 0x05040100u);
    }
  }
  return gamma;
}

// Store the codes of one piece: row `row` of a code tensor with `row_bytes` per row, piece
// `sub` (D/8 pieces per row).  Nontemporal: the codes are streamed out, not re-read here.
template <int D, int K>
__device__ inline void store_codes(uint8_t* vq, int64_t row, int sub, const uint2& c) {
  typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
  if (K == kQNibble) {
    __builtin_nontemporal_store(c.x, (uint32_t*)(vq + row * (D / 2)) + sub);
  } else {
    u32x2 t;
    t.x = c.x;
    t.y = c.y;
    __builtin_nontemporal_store(t, (u32x2*)(vq + row * D) + sub);
  }
}

// Store the codes of NP adjacent pieces, the lane's j-th group of NP in row `row`, at once.
template <int D, int K, int NP>
__device__ inline void store_code_pieces(uint8_t* vq, int64_t row, int j, const uint2 (&c)[NP]) {
  typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
  typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
  static_assert(NP == 1 || NP == 2, "one or two pieces");
  if (NP == 1) {
    store_codes<D, K>(vq, row, j, c[0]);
  } else if (K == kQNibble) {
    u32x2 t;
    t.x = c[0].x;
    t.y = c[NP - 1].x;
    __builtin_nontemporal_store(t, (u32x2*)(vq + row * (D / 2)) + j);
  } else {
    u32x4 t;
    t.x = c[0].x;
    t.y = c[0].y;
    t.z = c[NP - 1].x;
    t.w = c[NP - 1].y;
    __builtin_nontemporal_store(t, (u32x4*)(vq + row * D) + j);
  }
}

}  // namespace tp
