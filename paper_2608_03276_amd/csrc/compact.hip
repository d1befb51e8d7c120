// Step 4 of the eviction path: compaction of the kept rows (Sec. 3.1: only the index set I
// of each KV head is kept; Sec. 4 setup: eviction right after prefill).
//
// A row gather bound by HBM: d/8 lanes move one bf16 K row (16 B each), the first
// row_bytes/16 of them the quantised V row, lane 0 the scale.  Reads of the source rows are
// 16-byte aligned and each row's bytes are contiguous, so every wave touches whole cache
// lines.  Indices outside [0, N_b) produce a zero row (no out-of-bounds access).
#include "tp_internal.h"

namespace tp {
namespace {

constexpr int kCompactThreads = 256;

template <int D>
__global__ __launch_bounds__(kCompactThreads) void k_compact(CompactArgs a) {
  constexpr int LPR = D / 8;  // lanes per row
  constexpr int RPB = kCompactThreads / LPR;
  const int seg = blockIdx.y;
  const int sub = threadIdx.x % LPR;
  const int64_t r = (int64_t)blockIdx.x * RPB + threadIdx.x / LPR;  // kept row in [0, K_tot)
  if (r >= a.k_tot) return;
  int b = 0;
  while (b + 1 < a.bt.batch && a.kept_off[b + 1] <= r) ++b;
  const int64_t n0 = a.bt.ctx_off[b];
  const int64_t nb = a.bt.ctx_off[b + 1] - n0;
  const int64_t idx = a.kept[(int64_t)seg * a.k_tot + r];
  const bool ok = idx >= 0 && idx < nb;
  const int64_t src = (int64_t)seg * a.n_tot + n0 + (ok ? idx : 0);
  const int64_t dst = (int64_t)seg * a.k_tot + r;

  const uint4 kv = ok ? *((const uint4*)(a.k + src * D) + sub) : make_uint4(0, 0, 0, 0);
  *((uint4*)(a.k_out + dst * D) + sub) = kv;
  if (a.vq != nullptr && sub * 16 < a.row_bytes) {
    const uint4 qv = ok ? *((const uint4*)(a.vq + src * a.row_bytes) + sub) : make_uint4(0, 0, 0, 0);
    *((uint4*)(a.vq_out + dst * a.row_bytes) + sub) = qv;
  }
  if (a.scales != nullptr && sub == 0) a.scales_out[dst] = ok ? a.scales[src] : 0.0f;
}

}  // namespace

hipError_t launch_compact(const CompactArgs& a, int segments, int head_dim, hipStream_t stream) {
  if (a.k_tot == 0) return hipSuccess;
  const int lpr = head_dim / 8;
  const int64_t rpb = kCompactThreads / lpr;
  const dim3 grid((unsigned)((a.k_tot + rpb - 1) / rpb), (unsigned)segments);
  if (head_dim == 128)
    hipLaunchKernelGGL(k_compact<128>, grid, dim3(kCompactThreads), 0, stream, a);
  else
    hipLaunchKernelGGL(k_compact<64>, grid, dim3(kCompactThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace tp
