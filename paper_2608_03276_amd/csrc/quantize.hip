// Step 2 of the eviction path: the per-token V quantisation scale of Eq. 2 (Sec. 3.3),
//   gamma_t = fl32(max_c |v_tc| / qmax),
// which is the value score, fused with the per-token quantisation of V it belongs to:
//   q_tc = clamp(RNE(fl32(v_tc / gamma_t)), -qmax, qmax)   (b-bit integers), or
//   the OCP E4M3 code of fl32(v_tc / gamma_t), RNE, saturating at 448.
//
// Pure streaming work bound by HBM: each token row (d bf16) is read once by d/8 lanes
// (16 B each, fully coalesced), the absmax is an integer max of the bf16 magnitude bits
// (exact) reduced across those lanes with DPP row operations, and every lane writes its
// quantised bytes.
//
// The per-element quotient avoids a full IEEE division: the row is rescaled by 2^-e
// (e = exponent of its absmax, an exact power-of-two scaling that keeps every product and
// residual in the normal range), the quotient is v' * y with y = 1/gamma' (one correctly
// rounded division per token), and one residual step fl(q0 + fma(-q0, gamma', v') * y)
// corrects it.  An exhaustive check over every (absmax, v) pair of bf16 values, for every
// supported qmax, shows the resulting integer / E4M3 codes equal those of the correctly
// rounded quotient; rows whose absmax is below 2^-100 use the IEEE division directly.
#include "tp_internal.h"

namespace tp {
namespace {

constexpr int kQuantThreads = 256;
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
constexpr int kUnroll = 4;

// max over the `lanes` (8 or 16) consecutive lanes of a DPP row segment.
template <int LANES>
__device__ inline uint32_t group_max(uint32_t x) {
  // quad_perm [1,0,3,2] and [2,3,0,1]: lanes xor 1, xor 2
  x = max(x, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0xB1, 0xF, 0xF, false));
  x = max(x, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x4E, 0xF, 0xF, false));
  // row_half_mirror: lane i <-> 7-i within each 8 (pairs the two quads of a half-row)
  x = max(x, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x141, 0xF, 0xF, false));
  if (LANES == 16) {
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

template <int D>
__global__ __launch_bounds__(kQuantThreads) void k_quantize(QuantArgs a) {
  constexpr int LPT = D / 8;                 // lanes per token row
  constexpr int TPW = 64 / LPT;              // token rows per wave per load
  constexpr int TPB = kQuantThreads / LPT;   // token rows per block per load
  const int lane = threadIdx.x & 63;
  const int sub = lane % LPT;                // 16-byte piece within the row
  const int row_in_block = threadIdx.x / LPT;
  const bool int_fmt = a.qfmt == TP_QFMT_INT;
  const bool nibbles = int_fmt && a.bits <= 4;
  const float qmax = a.qmax;
  (void)TPW;

  for (int64_t base = (int64_t)blockIdx.x * TPB * kUnroll; base < a.rows;
       base += (int64_t)gridDim.x * TPB * kUnroll) {
    uint4 x[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int64_t row = base + u * TPB + row_in_block;
      if (row < a.rows) {
        const u32x4 t = __builtin_nontemporal_load((const u32x4*)(a.v + row * D) + sub);
        x[u] = make_uint4(t.x, t.y, t.z, t.w);
      } else {
        x[u] = make_uint4(0, 0, 0, 0);
      }
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int64_t row = base + u * TPB + row_in_block;
      const uint32_t w[4] = {x[u].x, x[u].y, x[u].z, x[u].w};
      uint32_t mx = 0;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        mx = max(mx, w[i] & 0x7FFFu);
        mx = max(mx, (w[i] >> 16) & 0x7FFFu);
      }
      mx = group_max<LPT>(mx);
      const float amax = __uint_as_float(mx << 16);
      const float gamma = amax / qmax;
      if (row >= a.rows) continue;
      if (sub == 0) a.scales[row] = gamma;
      if (a.vq == nullptr) continue;
      // exponent field of the absmax (bf16 and fp32 share it); below 2^-100 divide directly
      const int ef = (int)(mx >> 7);
      const bool direct = ef <= 27;
      const float sc = direct ? 1.0f : __builtin_amdgcn_ldexpf(1.0f, 127 - ef);
      const float gs = gamma * sc;
      const float ys = 1.0f / gs;
      uint32_t code[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const uint32_t h = (i & 1) ? (w[i >> 1] >> 16) : (w[i >> 1] & 0xFFFFu);
        const float v = __uint_as_float(h << 16);
        float y;
        if (direct) {
          y = v / gamma;
        } else {
          const float vs = v * sc;
          const float q0 = vs * ys;
          y = fmaf(fmaf(-q0, gs, vs), ys, q0);
        }
        if (gamma == 0.0f) {
          code[i] = 0;
        } else if (int_fmt) {
          const float r = __builtin_amdgcn_fmed3f(__builtin_rintf(y), -qmax, qmax);
          code[i] = (uint32_t)(int32_t)r;
        } else {
          code[i] = e4m3_code(__builtin_copysignf(y, v));
        }
      }
      if (nibbles) {
        uint32_t p = 0;
#pragma unroll
        for (int i = 0; i < 8; ++i) p |= (code[i] & 0xFu) << (4 * i);
        *((uint32_t*)(a.vq + row * (D / 2)) + sub) = p;
      } else {
        uint2 p;
        p.x = (code[0] & 0xFFu) | ((code[1] & 0xFFu) << 8) | ((code[2] & 0xFFu) << 16) | ((code[3] & 0xFFu) << 24);
        p.y = (code[4] & 0xFFu) | ((code[5] & 0xFFu) << 8) | ((code[6] & 0xFFu) << 16) | ((code[7] & 0xFFu) << 24);
        *((uint2*)(a.vq + row * D) + sub) = p;
      }
    }
  }
}

}  // namespace

hipError_t launch_quantize(const QuantArgs& a, int head_dim, hipStream_t stream) {
  const int lpt = head_dim / 8;
  const int64_t per_block = (int64_t)(kQuantThreads / lpt) * kUnroll;
  int64_t blocks = (a.rows + per_block - 1) / per_block;
  const int64_t cap = 256 * 32;  // 256 CUs x 32 resident blocks is plenty to saturate HBM
  if (blocks > cap) blocks = cap;
  if (blocks < 1) blocks = 1;
  if (head_dim == 128)
    hipLaunchKernelGGL(k_quantize<128>, dim3((unsigned)blocks), dim3(kQuantThreads), 0, stream, a);
  else
    hipLaunchKernelGGL(k_quantize<64>, dim3((unsigned)blocks), dim3(kQuantThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace tp
