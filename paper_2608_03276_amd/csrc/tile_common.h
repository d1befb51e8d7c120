// Tile definitions shared by the kernels that contract guide queries with context keys on
// v_mfma_f32_32x32x16_bf16 (the score passes and the guide rows' attention): operand
// fragments, the staged layout of a 32-token K sub-tile in LDS, and the (max, sum) merge.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace tp {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

union Frag {
  uint4 u;
  bf16x8 v;
};

template <int D>
struct Cfg {
  static constexpr int kSteps = D / 16;                  // MFMA k-steps over d
  static constexpr int kPieces = D / 8;                  // 16-byte pieces per row
  static constexpr int kRowBytes = D * 2;
  static constexpr int kStride = kRowBytes + 16;         // LDS bytes per staged query row
  static constexpr int kStageBytes = 32 * kRowBytes;     // one K sub-tile
  static constexpr int kTokPerKB = 1024 / kRowBytes;     // tokens per 1 KB copy instruction
};

__device__ inline int uniform(int x) { return __builtin_amdgcn_readfirstlane(x); }

// K sub-tiles in a wave's LDS staging buffer: token tl (0..31) of the sub-tile at
// tl * kRowBytes, its 16-byte piece p stored in slot p ^ swz(tl).  The swizzle puts the 16
// (D = 128) or 8 (D = 64, two rows per 256 bytes) tokens read by one group of lanes on
// different banks.
template <int D>
__device__ inline int swz(int tl) {
  return D == 128 ? (tl & 15) : ((tl >> 1) & 7);
}

// K fragment of the staged sub-tile for MFMA k-step s: token lane%32, the d-columns of this
// half-wave.
template <int D>
__device__ inline void read_kfrag_step(const char* kbuf, Frag& f, int s) {
  using C = Cfg<D>;
  const int lane = threadIdx.x & 63;
  const int tl = lane & 31;
  const int p = (lane >> 5) * (C::kPieces / 2) + s;
  f.u = *(const uint4*)(kbuf + tl * C::kRowBytes + ((p ^ swz<D>(tl)) * 16));
}

template <int D>
__device__ inline void read_kfrag(const char* kbuf, Frag (&kf)[Cfg<D>::kSteps]) {
#pragma unroll
  for (int s = 0; s < Cfg<D>::kSteps; ++s) read_kfrag_step<D>(kbuf, kf[s], s);
}

// The largest of the 16 accumulator values a lane holds.
__device__ inline float max16(const f32x16& x) {
  const float a0 = fmaxf(fmaxf(x[0], x[1]), x[2]), a1 = fmaxf(fmaxf(x[3], x[4]), x[5]);
  const float a2 = fmaxf(fmaxf(x[6], x[7]), x[8]), a3 = fmaxf(fmaxf(x[9], x[10]), x[11]);
  const float a4 = fmaxf(fmaxf(x[12], x[13]), x[14]);
  return fmaxf(fmaxf(fmaxf(a0, a1), x[15]), fmaxf(fmaxf(a2, a3), a4));
}

// Running (max, sum) statistics start at (-FLT_MAX, 0) rather than (-inf, 0): merging a
// unit whose logits are all -inf (masked tokens, or the empty pipeline slot before the
// first pair) is then an exact no-op, with no special case.
constexpr float kNoMax = -3.402823466e38f;

__device__ inline void merge_stats(float& m, float& s, float m2, float s2) {
  const float mn = fmaxf(m, m2);
  s = s * __builtin_amdgcn_exp2f(m - mn) + s2 * __builtin_amdgcn_exp2f(m2 - mn);
  m = mn;
}

}  // namespace
}  // namespace tp
