// Step 4 of the eviction path: compaction of the kept rows (Sec. 3.1: only the index set I
// of each KV head is kept; Sec. 4 setup: eviction right after prefill).
//
// A row gather bound by HBM: d/8 lanes move one bf16 K row (16 B each), the first
// row_bytes/16 of them the quantised V row, lane 0 the scale; each lane group handles four
// kept rows so their index loads and row loads are in flight together.  Reads of the source
// rows are 16-byte aligned and each row's bytes are contiguous, so every wave touches whole
// cache lines.  Indices outside [0, N_b) produce a zero row (no out-of-bounds access).
//
// k_compact_quant is the same gather fused with step 2 for the kept rows only: it reads the
// kept bf16 V rows and quantises them with the arithmetic of the standalone quantisation
// (quant_row.h), so its codes and scales are bit-identical to quantising every row and then
// gathering, without writing the codes of the evicted rows.
#include "quant_row.h"
#include "tp_internal.h"

namespace tp {
namespace {

constexpr int kCompactThreads = 256;
constexpr int kRowsPerLane = 4;  // kept rows per lane group: their index and row loads overlap

template <int D>
__global__ __launch_bounds__(kCompactThreads) void k_compact(CompactArgs a) {
  constexpr int LPR = D / 8;  // lanes per row
  constexpr int RPB = kCompactThreads / LPR;
  const int seg = blockIdx.y;
  const int sub = threadIdx.x % LPR;
  const int64_t r0 = (int64_t)blockIdx.x * RPB * kRowsPerLane + threadIdx.x / LPR;
  int64_t src[kRowsPerLane];
  bool ok[kRowsPerLane];
#pragma unroll
  for (int u = 0; u < kRowsPerLane; ++u) {  // kept row r in [0, K_tot): its source row
    const int64_t r = r0 + u * RPB;
    ok[u] = false;
    src[u] = 0;
    if (r < a.k_tot) {
      int b = 0;
      while (b + 1 < a.bt.batch && a.kept_off[b + 1] <= r) ++b;
      const int64_t n0 = a.bt.ctx_off[b];
      const int64_t nb = a.bt.ctx_off[b + 1] - n0;
      const int64_t idx = a.kept[(int64_t)seg * a.k_tot + r];
      ok[u] = idx >= 0 && idx < nb;
      src[u] = (int64_t)seg * a.n_tot + n0 + (ok[u] ? idx : 0);
    }
  }
  uint4 kv[kRowsPerLane], qv[kRowsPerLane];
  const bool has_q = a.vq != nullptr && sub * 16 < a.row_bytes;
#pragma unroll
  for (int u = 0; u < kRowsPerLane; ++u) {
    kv[u] = ok[u] ? *((const uint4*)(a.k + src[u] * D) + sub) : make_uint4(0, 0, 0, 0);
    qv[u] = ok[u] && has_q ? *((const uint4*)(a.vq + src[u] * a.row_bytes) + sub) : make_uint4(0, 0, 0, 0);
  }
#pragma unroll
  for (int u = 0; u < kRowsPerLane; ++u) {
    const int64_t r = r0 + u * RPB;
    if (r >= a.k_tot) break;
    const int64_t dst = (int64_t)seg * a.k_tot + r;
    *((uint4*)(a.k_out + dst * D) + sub) = kv[u];
    if (has_q) *((uint4*)(a.vq_out + dst * a.row_bytes) + sub) = qv[u];
    if (a.scales != nullptr && sub == 0) a.scales_out[dst] = ok[u] ? a.scales[src[u]] : 0.0f;
  }
}

// Source row of kept row r of segment seg, and whether its index is in range.
__device__ inline int64_t kept_source(const CompactArgs& a, int seg, int64_t r, bool& ok) {
  int b = 0;
  while (b + 1 < a.bt.batch && a.kept_off[b + 1] <= r) ++b;
  const int64_t n0 = a.bt.ctx_off[b];
  const int64_t nb = a.bt.ctx_off[b + 1] - n0;
  const int64_t idx = a.kept[(int64_t)seg * a.k_tot + r];
  ok = idx >= 0 && idx < nb;
  return (int64_t)seg * a.n_tot + n0 + (ok ? idx : 0);
}

template <int D, int K>
__global__ __launch_bounds__(kCompactThreads) void k_compact_quant(CompactArgs a) {
  constexpr int LPR = D / 8;
  constexpr int RPB = kCompactThreads / LPR;
  const int seg = blockIdx.y;
  const int sub = threadIdx.x % LPR;
  const int64_t r0 = (int64_t)blockIdx.x * RPB * kRowsPerLane + threadIdx.x / LPR;
  const QuantFmt f{a.qfmt == TP_QFMT_INT, a.qfmt == TP_QFMT_INT && a.bits <= 4, a.qmax};
  __shared__ QuantTables tab;
  build_tables(tab, a.qmax, a.ro.off);
  __syncthreads();
  int64_t src[kRowsPerLane];
  bool ok[kRowsPerLane];
#pragma unroll
  for (int u = 0; u < kRowsPerLane; ++u) {
    const int64_t r = r0 + u * RPB;
    ok[u] = false;
    src[u] = r < a.k_tot ? kept_source(a, seg, r, ok[u]) : 0;
  }
  uint4 kv[kRowsPerLane], vv[kRowsPerLane];
#pragma unroll
  for (int u = 0; u < kRowsPerLane; ++u) {
    kv[u] = ok[u] ? *((const uint4*)(a.k + src[u] * D) + sub) : make_uint4(0, 0, 0, 0);
    vv[u] = ok[u] ? *((const uint4*)(a.v + src[u] * D) + sub) : make_uint4(0, 0, 0, 0);
  }
#pragma unroll
  for (int u = 0; u < kRowsPerLane; ++u) {
    const int64_t r = r0 + u * RPB;
    uint2 c;
    const float gamma = quant_piece<LPR, K>(vv[u], tab, f, c);  // every lane of the wave takes part
    if (r >= a.k_tot) continue;
    const int64_t dst = (int64_t)seg * a.k_tot + r;
    *((uint4*)(a.k_out + dst * D) + sub) = kv[u];
    store_codes<D, K>(a.vq_out, dst, sub, c);
    if (sub == 0) a.scales_out[dst] = gamma;
  }
}

}  // namespace

hipError_t launch_compact(const CompactArgs& a, int segments, int head_dim, hipStream_t stream) {
  if (a.k_tot == 0) return hipSuccess;
  const int lpr = head_dim / 8;
  const int64_t rpb = (int64_t)(kCompactThreads / lpr) * kRowsPerLane;
  const dim3 grid((unsigned)((a.k_tot + rpb - 1) / rpb), (unsigned)segments);
  if (a.v != nullptr) {
    const int kind = qkind_of(a.qfmt, a.bits);
#define TP_COMPACT_QUANT(D_, K_) hipLaunchKernelGGL((k_compact_quant<D_, K_>), grid, dim3(kCompactThreads), 0, stream, a)
    if (head_dim == 128) {
      if (kind == kQInt8) TP_COMPACT_QUANT(128, kQInt8);
      else if (kind == kQByte) TP_COMPACT_QUANT(128, kQByte);
      else if (kind == kQNibble) TP_COMPACT_QUANT(128, kQNibble);
      else TP_COMPACT_QUANT(128, kQE4M3);
    } else {
      if (kind == kQInt8) TP_COMPACT_QUANT(64, kQInt8);
      else if (kind == kQByte) TP_COMPACT_QUANT(64, kQByte);
      else if (kind == kQNibble) TP_COMPACT_QUANT(64, kQNibble);
      else TP_COMPACT_QUANT(64, kQE4M3);
    }
#undef TP_COMPACT_QUANT
    return hipGetLastError();
  }
  if (head_dim == 128)
    hipLaunchKernelGGL(k_compact<128>, grid, dim3(kCompactThreads), 0, stream, a);
  else
    hipLaunchKernelGGL(k_compact<64>, grid, dim3(kCompactThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace tp
