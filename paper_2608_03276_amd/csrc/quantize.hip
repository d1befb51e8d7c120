// Step 2 of the eviction path: the per-token V quantisation scale of Eq. 2 (Sec. 3.3), the
// value score, fused with the per-token quantisation of V it belongs to (the arithmetic is
// in quant_row.h).  Pure streaming work bound by HBM: each token row (d bf16) is read once by
// d/8 lanes (16 B each, fully coalesced, several rows in flight per lane) and every lane
// writes its quantised bytes.
#include "quant_row.h"
#include "tp_internal.h"

namespace tp {
namespace {

constexpr int kQuantThreads = 256;
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
constexpr int kUnroll = 8;  // rows in flight per lane group

// K = one of QKind (codes of that format), or kScalesOnly (no code tensor, which needs only the
// row absmax).
constexpr int kScalesOnly = -1;

template <int D, int K>
__global__ __launch_bounds__(kQuantThreads) void k_quantize(QuantArgs a) {
  constexpr int LPT = D / 8;                 // lanes per token row
  constexpr int TPB = kQuantThreads / LPT;   // token rows per block per load
  const int sub = threadIdx.x % LPT;         // 16-byte piece within the row
  const int row_in_block = threadIdx.x / LPT;
  const QuantFmt f{a.qfmt == TP_QFMT_INT, a.qfmt == TP_QFMT_INT && a.bits <= 4, a.qmax};
  __shared__ QuantTables tab;
  if (K != kScalesOnly) {
    build_tables(tab, a.qmax, a.ro.off);
    __syncthreads();
  }

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
      if (K != kScalesOnly) {
        uint2 c;
        const float gamma = quant_piece<LPT, (K < 0 ? 0 : K)>(x[u], tab, f, c);
        if (row >= a.rows) continue;
        if (sub == 0) a.scales[row] = gamma;
        store_codes<D, (K < 0 ? 0 : K)>(a.vq, row, sub, c);
      } else {
        const float gamma = scale_piece<LPT>(x[u], f);
        if (row < a.rows && sub == 0) a.scales[row] = gamma;
      }
    }
  }
}

template <int D>
void launch_d(const QuantArgs& a, unsigned blocks, hipStream_t stream) {
  if (a.vq == nullptr) {
    hipLaunchKernelGGL((k_quantize<D, kScalesOnly>), dim3(blocks), dim3(kQuantThreads), 0, stream, a);
    return;
  }
  switch (qkind_of(a.qfmt, a.bits)) {
    case kQInt8:
      hipLaunchKernelGGL((k_quantize<D, kQInt8>), dim3(blocks), dim3(kQuantThreads), 0, stream, a);
      break;
    case kQByte:
      hipLaunchKernelGGL((k_quantize<D, kQByte>), dim3(blocks), dim3(kQuantThreads), 0, stream, a);
      break;
    case kQNibble:
      hipLaunchKernelGGL((k_quantize<D, kQNibble>), dim3(blocks), dim3(kQuantThreads), 0, stream, a);
      break;
    default:
      hipLaunchKernelGGL((k_quantize<D, kQE4M3>), dim3(blocks), dim3(kQuantThreads), 0, stream, a);
  }
}

// ------------------------------------------------------------------ lean variant
// The same quantisation with one workgroup per CU (one wave per SIMD) and at most 48 VGPRs,
// so that it stays resident beside a score-pass workgroup (which leaves one wave slot and 48
// VGPRs per SIMD free): each wave quantises kLeanLoads loads of RPW = 64/LPT consecutive rows
// (1 KB each, coalesced), all loads issued before any row is quantised, then strides on.
// No launch attribute can cap a kernel below the 64 VGPRs of eight waves per SIMD (and the
// compiler ignores a plain VGPR-count request), so the budget holds by construction (four
// loads in flight: 42 VGPRs) and a build test checks that the two kernels fit together.
constexpr int kLeanLoads = 4;
constexpr int kLeanBlocks = 256;

template <int D, int K>
__global__ __launch_bounds__(kQuantThreads) void k_quantize_lean(QuantArgs a) {
  constexpr int LPT = D / 8;
  constexpr int RPW = 64 / LPT;
  constexpr int kWaves = kQuantThreads / 64;
  const int lane = threadIdx.x & 63;
  const int sub = lane % LPT;
  const QuantFmt f{a.qfmt == TP_QFMT_INT, a.qfmt == TP_QFMT_INT && a.bits <= 4, a.qmax};
  __shared__ QuantTables tab;
  if (K != kScalesOnly) {
    build_tables(tab, a.qmax, a.ro.off);
    __syncthreads();
  }
  const int64_t stride = (int64_t)gridDim.x * kWaves * kLeanLoads * RPW;
  for (int64_t row0 = ((int64_t)blockIdx.x * kWaves + threadIdx.x / 64) * kLeanLoads * RPW; row0 < a.rows;
       row0 += stride) {
    uint4 x[kLeanLoads];
#pragma unroll
    for (int u = 0; u < kLeanLoads; ++u) {
      const int64_t row = row0 + u * RPW + lane / LPT;
      if (row < a.rows) {
        const u32x4 t = __builtin_nontemporal_load((const u32x4*)(a.v + row * D) + sub);
        x[u] = make_uint4(t.x, t.y, t.z, t.w);
      } else {
        x[u] = make_uint4(0, 0, 0, 0);
      }
    }
#pragma unroll
    for (int u = 0; u < kLeanLoads; ++u) {
      const int64_t row = row0 + u * RPW + lane / LPT;
      if (K != kScalesOnly) {
        uint2 c;
        const float gamma = quant_piece<LPT, (K < 0 ? 0 : K)>(x[u], tab, f, c);
        if (row >= a.rows) continue;
        if (sub == 0) a.scales[row] = gamma;
        store_codes<D, (K < 0 ? 0 : K)>(a.vq, row, sub, c);
      } else {
        const float gamma = scale_piece<LPT>(x[u], f);
        if (row < a.rows && sub == 0) a.scales[row] = gamma;
      }
    }
  }
}

template <int D>
void launch_lean_d(const QuantArgs& a, hipStream_t stream) {
  const dim3 grid(kLeanBlocks), block(kQuantThreads);
  if (a.vq == nullptr) {
    hipLaunchKernelGGL((k_quantize_lean<D, kScalesOnly>), grid, block, 0, stream, a);
    return;
  }
  switch (qkind_of(a.qfmt, a.bits)) {
    case kQInt8:
      hipLaunchKernelGGL((k_quantize_lean<D, kQInt8>), grid, block, 0, stream, a);
      break;
    case kQByte:
      hipLaunchKernelGGL((k_quantize_lean<D, kQByte>), grid, block, 0, stream, a);
      break;
    case kQNibble:
      hipLaunchKernelGGL((k_quantize_lean<D, kQNibble>), grid, block, 0, stream, a);
      break;
    default:
      hipLaunchKernelGGL((k_quantize_lean<D, kQE4M3>), grid, block, 0, stream, a);
  }
}

}  // namespace

hipError_t launch_quantize_lean(const QuantArgs& a, int head_dim, hipStream_t stream) {
  if (a.rows <= 0) return hipSuccess;
  if (head_dim == 128)
    launch_lean_d<128>(a, stream);
  else
    launch_lean_d<64>(a, stream);
  return hipGetLastError();
}

hipError_t launch_quantize(const QuantArgs& a, int head_dim, hipStream_t stream) {
  const int lpt = head_dim / 8;
  const int64_t per_block = (int64_t)(kQuantThreads / lpt) * kUnroll;
  int64_t blocks = (a.rows + per_block - 1) / per_block;
  const int64_t cap = 256 * 32;  // 256 CUs x 32 resident blocks is plenty to saturate HBM
  if (blocks > cap) blocks = cap;
  if (blocks < 1) blocks = 1;
  if (head_dim == 128)
    launch_d<128>(a, (unsigned)blocks, stream);
  else
    launch_d<64>(a, (unsigned)blocks, stream);
  return hipGetLastError();
}

}  // namespace tp
