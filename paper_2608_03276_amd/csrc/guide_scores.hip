// Step 1 of the eviction path: the task-guided key score of Eq. 1 (Sec. 3.2).
//
// For every (sequence b, layer l, KV head h) segment the guide rows are the R*G_b
// (query head, guide token) pairs of the GQA group; the score of context token i is
//   raw_i   = (1/R) sum_rows exp(scale*<q_row, k_i> - lse_row)        (softmax over context)
//   s_key_i = (1/K) sum_{|t|<=K/2} raw_{i+t}                           (zero-padded pooling)
// The exact per-row normaliser lse_row needs every logit of the row, so the logits are
// produced twice (never stored): pass 1 keeps an online (max, sum) per row and chunk,
// a small kernel merges the chunks into lse, and pass 2 recomputes the logits and sums the
// normalised weights per token.  Everything is kept in the log2 domain:
// x' = x * scale * log2(e), exp2(x' - lse2).
//
// The contraction over d runs on v_mfma_f32_32x32x16_bf16.  Pass 1 puts tokens on M and
// guide rows on N, so each lane owns one row and 16 tokens (row statistics reduce inside
// the lane); pass 2 swaps the operands, so each lane owns one token and 16 rows (the
// token's sum over rows reduces inside the lane).  The same register fragments serve both
// orientations because the A and B operand layouts of the instruction coincide.  K is
// streamed through LDS in 128-token tiles (double-buffered through registers); the guide
// queries of a wave stay in registers for its whole chunk.
#include "tp_internal.h"

namespace tp {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

union Frag {
  uint4 u;
  bf16x8 v;
};

template <int D>
struct Cfg {
  static constexpr int kSteps = D / 16;                     // MFMA k-steps over d
  static constexpr int kHalf = D / 2;                       // d columns per half-wave
  static constexpr int kStride = D + 8;                     // LDS row pitch (bf16), +16 B pad
  static constexpr int kPieces = D / 8;                     // 16-byte pieces per token row
  static constexpr int kLoads = kMacroTokens * kPieces / kGuideThreads;
  static_assert(kLoads * kGuideThreads == kMacroTokens * kPieces, "tile split");
};

struct Work {
  int b, seg, l, h, rg, chunk;
  int64_t n0, nb, c0, c1, g0;
  int gb, rows, row0, nrows;
};

// Workgroup -> (row group, chunk, segment, sequence).  Consecutive workgroup ids are dealt
// round-robin to the 8 XCDs; the row groups of one chunk are given ids 8 apart so they land
// on the same XCD and share the chunk's K through that XCD's L2.
__device__ inline bool decode(const GuideArgs& a, Work& w) {
  const int x = blockIdx.x;
  const int xcd = x & 7, slot = x >> 3;
  w.rg = slot % a.nrg_max;
  w.chunk = xcd + 8 * (slot / a.nrg_max);
  w.seg = blockIdx.y;
  w.l = w.seg / a.Hkv;
  w.h = w.seg % a.Hkv;
  w.b = blockIdx.z;
  w.n0 = a.bt.ctx_off[w.b];
  w.nb = a.bt.ctx_off[w.b + 1] - w.n0;
  w.c0 = (int64_t)w.chunk * kChunkTokens;
  if (w.c0 >= w.nb) return false;
  w.c1 = w.c0 + kChunkTokens < w.nb ? w.c0 + kChunkTokens : w.nb;
  w.g0 = a.bt.g_off[w.b];
  w.gb = (int)(a.bt.g_off[w.b + 1] - w.g0);
  w.rows = a.R * w.gb;
  w.row0 = w.rg * kRowsPerGroup;
  if (w.row0 >= w.rows) return false;
  w.nrows = w.rows - w.row0 < kRowsPerGroup ? w.rows - w.row0 : kRowsPerGroup;
  return true;
}

// Global row id (index into q_guide rows, stats and lse) of guide row rho of the segment.
__device__ inline int64_t grow_of(const GuideArgs& a, const Work& w, int rho) {
  const int r = rho / w.gb, j = rho - r * w.gb;
  const int64_t qh = (int64_t)w.h * a.R + r;
  return ((int64_t)w.l * a.Hq + qh) * a.g_tot + w.g0 + j;
}

// Wave layout: WR waves split the rows (64 each), WT = 4/WR teams split the 4 sub-tiles.
struct WaveRole {
  int wr, wt, WR, WT;
};
__device__ inline WaveRole wave_role(const Work& w) {
  WaveRole r;
  r.WR = w.nrows > 128 ? 4 : (w.nrows > 64 ? 2 : 1);
  r.WT = 4 / r.WR;
  const int wave = threadIdx.x >> 6;
  r.wr = wave % r.WR;
  r.wt = wave / r.WR;
  return r;
}

template <int D>
__device__ inline void load_q(const GuideArgs& a, const Work& w, int wrow0, Frag (&qf)[2][Cfg<D>::kSteps]) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int rb = 0; rb < 2; ++rb) {
    const int rho = wrow0 + rb * 32 + (lane & 31);
    if (rho < w.rows) {
      const uint16_t* src = a.q + grow_of(a, w, rho) * D + (lane >> 5) * Cfg<D>::kHalf;
#pragma unroll
      for (int s = 0; s < Cfg<D>::kSteps; ++s) qf[rb][s].u = *(const uint4*)(src + 8 * s);
    } else {
#pragma unroll
      for (int s = 0; s < Cfg<D>::kSteps; ++s) qf[rb][s].u = make_uint4(0, 0, 0, 0);
    }
  }
}

template <int D>
__device__ inline void load_tile(const uint16_t* kseg, int64_t t0, int64_t c1, uint4 (&st)[Cfg<D>::kLoads]) {
#pragma unroll
  for (int j = 0; j < Cfg<D>::kLoads; ++j) {
    const int p = threadIdx.x + j * kGuideThreads;
    const int tok = p / Cfg<D>::kPieces, pc = p % Cfg<D>::kPieces;
    const int64_t gt = t0 + tok;
    st[j] = gt < c1 ? *(const uint4*)(kseg + gt * D + pc * 8) : make_uint4(0, 0, 0, 0);
  }
}

template <int D>
__device__ inline void store_tile(uint16_t* buf, const uint4 (&st)[Cfg<D>::kLoads]) {
#pragma unroll
  for (int j = 0; j < Cfg<D>::kLoads; ++j) {
    const int p = threadIdx.x + j * kGuideThreads;
    const int tok = p / Cfg<D>::kPieces, pc = p % Cfg<D>::kPieces;
    *(uint4*)(buf + tok * Cfg<D>::kStride + pc * 8) = st[j];
  }
}

// K fragment of sub-tile `st` for this lane: token st*32 + lane%32, columns of its half.
template <int D>
__device__ inline void read_kfrag(const uint16_t* buf, int st, Frag (&kf)[Cfg<D>::kSteps]) {
  const int lane = threadIdx.x & 63;
  const uint16_t* src = buf + (st * 32 + (lane & 31)) * Cfg<D>::kStride + (lane >> 5) * Cfg<D>::kHalf;
#pragma unroll
  for (int s = 0; s < Cfg<D>::kSteps; ++s) kf[s].u = *(const uint4*)(src + 8 * s);
}

__device__ inline void merge_stats(float& m, float& s, float m2, float s2) {
  const float mn = fmaxf(m, m2);
  if (mn == -INFINITY) return;
  s = s * __builtin_amdgcn_exp2f(m - mn) + s2 * __builtin_amdgcn_exp2f(m2 - mn);
  m = mn;
}

// ---------------------------------------------------------------------------- pass 1
template <int D>
__global__ __launch_bounds__(kGuideThreads, 2) void k_guide_stats(GuideArgs a) {
  Work w;
  if (!decode(a, w)) return;
  using C = Cfg<D>;
  __shared__ __attribute__((aligned(16))) uint16_t kt[2][kMacroTokens * C::kStride];
  __shared__ float2 xch[4][kRowsPerGroup];

  const int lane = threadIdx.x & 63;
  const WaveRole role = wave_role(w);
  const int wrow0 = w.row0 + role.wr * kRowsPerWave;
  const bool blk_ok[2] = {wrow0 < w.rows, wrow0 + 32 < w.rows};

  Frag qf[2][C::kSteps];
  load_q<D>(a, w, wrow0, qf);
  float m[2] = {-INFINITY, -INFINITY}, s[2] = {0.f, 0.f};

  const uint16_t* kseg = a.k + ((int64_t)w.seg * a.n_tot + w.n0) * D;
  const int ntiles = (int)((w.c1 - w.c0 + kMacroTokens - 1) / kMacroTokens);
  uint4 stage[C::kLoads];
  load_tile<D>(kseg, w.c0, w.c1, stage);
  store_tile<D>(kt[0], stage);
  __syncthreads();

  for (int it = 0; it < ntiles; ++it) {
    const int64_t t0 = w.c0 + (int64_t)it * kMacroTokens;
    if (it + 1 < ntiles) load_tile<D>(kseg, t0 + kMacroTokens, w.c1, stage);
    const uint16_t* buf = kt[it & 1];
    for (int st = role.wt; st < kMacroTokens / 32; st += role.WT) {
      const int64_t sub0 = t0 + st * 32;
      if (sub0 >= w.c1) break;
      const int nvalid = w.c1 - sub0 < 32 ? (int)(w.c1 - sub0) : 32;
      Frag kf[C::kSteps];
      read_kfrag<D>(buf, st, kf);
#pragma unroll
      for (int rb = 0; rb < 2; ++rb) {
        if (!blk_ok[rb]) continue;
        f32x16 acc = {};
#pragma unroll
        for (int ks = 0; ks < C::kSteps; ++ks)
          acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[ks].v, qf[rb][ks].v, acc, 0, 0, 0);
        // acc[i] = <k_token, q_row>, token = (i/4)*8 + (lane/32)*4 + i%4, row = lane%32
        if (nvalid < 32) {
#pragma unroll
          for (int i = 0; i < 16; ++i) {
            const int tok = (i >> 2) * 8 + (lane >> 5) * 4 + (i & 3);
            if (tok >= nvalid) acc[i] = -INFINITY;
          }
        }
        float tmax = acc[0];
#pragma unroll
        for (int i = 1; i < 16; ++i) tmax = fmaxf(tmax, acc[i]);
        const float mn = fmaxf(m[rb], tmax * a.c);
        float sum = 0.f;
#pragma unroll
        for (int i = 0; i < 16; ++i) sum += __builtin_amdgcn_exp2f(fmaf(acc[i], a.c, -mn));
        const float sn = s[rb] * __builtin_amdgcn_exp2f(m[rb] - mn) + sum;
        if (mn != -INFINITY) {
          s[rb] = sn;
          m[rb] = mn;
        }
      }
    }
    if (it + 1 < ntiles) store_tile<D>(kt[(it + 1) & 1], stage);
    __syncthreads();
  }

  // The two half-waves hold the same rows over different tokens.
#pragma unroll
  for (int rb = 0; rb < 2; ++rb) {
    const float mo = __shfl_xor(m[rb], 32);
    const float so = __shfl_xor(s[rb], 32);
    merge_stats(m[rb], s[rb], mo, so);
    if (lane < 32) xch[role.wt][role.wr * kRowsPerWave + rb * 32 + lane] = make_float2(m[rb], s[rb]);
  }
  __syncthreads();
  const int t = threadIdx.x;
  if (t < role.WR * kRowsPerWave) {
    const int rho = w.row0 + t;
    if (rho < w.rows) {
      float mm = xch[0][t].x, ss = xch[0][t].y;
      for (int q = 1; q < role.WT; ++q) merge_stats(mm, ss, xch[q][t].x, xch[q][t].y);
      const int64_t growtot = (int64_t)a.L * a.Hq * a.g_tot;
      a.stats[(int64_t)w.chunk * growtot + grow_of(a, w, rho)] = make_float2(mm, ss);
    }
  }
}

// ---------------------------------------------------------------------------- lse merge
__global__ __launch_bounds__(256) void k_guide_lse(GuideArgs a) {
  const int b = blockIdx.y;
  const int64_t g0 = a.bt.g_off[b];
  const int gb = (int)(a.bt.g_off[b + 1] - g0);
  const int64_t nb = a.bt.ctx_off[b + 1] - a.bt.ctx_off[b];
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= (int64_t)a.L * a.Hq * gb) return;
  const int64_t per_layer = (int64_t)a.Hq * gb;
  const int64_t l = idx / per_layer, rem = idx - l * per_layer;
  const int64_t qh = rem / gb, j = rem - qh * gb;
  const int64_t grow = (l * a.Hq + qh) * a.g_tot + g0 + j;
  const int64_t growtot = (int64_t)a.L * a.Hq * a.g_tot;
  const int nch = (int)((nb + kChunkTokens - 1) / kChunkTokens);
  float m = -INFINITY, s = 0.f;
  for (int c = 0; c < nch; ++c) {
    const float2 v = a.stats[(int64_t)c * growtot + grow];
    merge_stats(m, s, v.x, v.y);
  }
  a.lse2[grow] = m + log2f(s);
}

// ---------------------------------------------------------------------------- pass 2
template <int D>
__global__ __launch_bounds__(kGuideThreads, 2) void k_guide_attn(GuideArgs a) {
  Work w;
  if (!decode(a, w)) return;
  using C = Cfg<D>;
  __shared__ __attribute__((aligned(16))) uint16_t kt[2][kMacroTokens * C::kStride];
  __shared__ float red[2][4][kMacroTokens];

  const int lane = threadIdx.x & 63;
  const WaveRole role = wave_role(w);
  const int wrow0 = w.row0 + role.wr * kRowsPerWave;
  const bool blk_ok[2] = {wrow0 < w.rows, wrow0 + 32 < w.rows};

  Frag qf[2][C::kSteps];
  load_q<D>(a, w, wrow0, qf);
  // lse2 of the 16 rows this lane owns in each block: row = (i/4)*8 + (lane/32)*4 + i%4.
  float lz[2][16];
#pragma unroll
  for (int rb = 0; rb < 2; ++rb)
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int rho = wrow0 + rb * 32 + (i >> 2) * 8 + (lane >> 5) * 4 + (i & 3);
      lz[rb][i] = rho < w.rows ? a.lse2[grow_of(a, w, rho)] : INFINITY;
    }

  const uint16_t* kseg = a.k + ((int64_t)w.seg * a.n_tot + w.n0) * D;
  float* raw_out = a.raw + ((int64_t)w.rg * a.L * a.Hkv + w.seg) * a.n_tot + w.n0;
  const int ntiles = (int)((w.c1 - w.c0 + kMacroTokens - 1) / kMacroTokens);
  uint4 stage[C::kLoads];
  load_tile<D>(kseg, w.c0, w.c1, stage);
  store_tile<D>(kt[0], stage);
  __syncthreads();

  for (int it = 0; it < ntiles; ++it) {
    const int64_t t0 = w.c0 + (int64_t)it * kMacroTokens;
    if (it + 1 < ntiles) load_tile<D>(kseg, t0 + kMacroTokens, w.c1, stage);
    const uint16_t* buf = kt[it & 1];
    for (int st = role.wt; st < kMacroTokens / 32; st += role.WT) {
      if (t0 + st * 32 >= w.c1) break;
      Frag kf[C::kSteps];
      read_kfrag<D>(buf, st, kf);
      float part = 0.f;
#pragma unroll
      for (int rb = 0; rb < 2; ++rb) {
        if (!blk_ok[rb]) continue;
        f32x16 acc = {};
#pragma unroll
        for (int ks = 0; ks < C::kSteps; ++ks)
          acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qf[rb][ks].v, kf[ks].v, acc, 0, 0, 0);
        // acc[i] = <q_row, k_token>, row = (i/4)*8 + (lane/32)*4 + i%4, token = lane%32
#pragma unroll
        for (int i = 0; i < 16; ++i) part += __builtin_amdgcn_exp2f(fmaf(acc[i], a.c, -lz[rb][i]));
      }
      part += __shfl_xor(part, 32);
      if (lane < 32) red[it & 1][role.wr][st * 32 + lane] = part;
    }
    if (it + 1 < ntiles) store_tile<D>(kt[(it + 1) & 1], stage);
    __syncthreads();
    if (threadIdx.x < kMacroTokens) {
      const int64_t tok = t0 + threadIdx.x;
      if (tok < w.c1) {
        float v = red[it & 1][0][threadIdx.x];
        for (int q = 1; q < role.WR; ++q) v += red[it & 1][q][threadIdx.x];
        raw_out[tok] = v;
      }
    }
  }
}

// ---------------------------------------------------------------------------- pooling
__global__ __launch_bounds__(256) void k_guide_pool(GuideArgs a) {
  const int seg = blockIdx.y, b = blockIdx.z;
  const int64_t n0 = a.bt.ctx_off[b];
  const int64_t nb = a.bt.ctx_off[b + 1] - n0;
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= nb) return;
  const int gb = (int)(a.bt.g_off[b + 1] - a.bt.g_off[b]);
  const int nrg = (a.R * gb + kRowsPerGroup - 1) / kRowsPerGroup;
  const int64_t lh = (int64_t)a.L * a.Hkv;
  const float* raw = a.raw + (int64_t)seg * a.n_tot + n0;
  float acc = 0.f;
  for (int t = -a.pool_half; t <= a.pool_half; ++t) {
    const int64_t j = i + t;
    if (j < 0 || j >= nb) continue;
    for (int rg = 0; rg < nrg; ++rg) acc += raw[rg * lh * a.n_tot + j];
  }
  a.s_key[(int64_t)seg * a.n_tot + n0 + i] = acc * a.pool_inv;
}

template <int D>
hipError_t launch_d(const GuideArgs& a, hipStream_t stream) {
  int64_t max_nb = 0, max_gb = 0;
  for (int b = 0; b < a.bt.batch; ++b) {
    const int64_t nb = a.bt.ctx_off[b + 1] - a.bt.ctx_off[b];
    const int64_t gb = a.bt.g_off[b + 1] - a.bt.g_off[b];
    if (nb > max_nb) max_nb = nb;
    if (gb > max_gb) max_gb = gb;
  }
  const dim3 block(kGuideThreads);
  const dim3 grid((unsigned)(a.nrg_max * a.nchunk_pad), (unsigned)(a.L * a.Hkv), (unsigned)a.bt.batch);
  hipLaunchKernelGGL(k_guide_stats<D>, grid, block, 0, stream, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const dim3 lgrid((unsigned)((a.L * a.Hq * max_gb + 255) / 256), (unsigned)a.bt.batch);
  hipLaunchKernelGGL(k_guide_lse, lgrid, dim3(256), 0, stream, a);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_guide_attn<D>, grid, block, 0, stream, a);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  const dim3 pgrid((unsigned)((max_nb + 255) / 256), (unsigned)(a.L * a.Hkv), (unsigned)a.bt.batch);
  hipLaunchKernelGGL(k_guide_pool, pgrid, dim3(256), 0, stream, a);
  return hipGetLastError();
}

}  // namespace

GuideWorkspace guide_workspace_layout(int32_t L, int32_t Hq, int32_t Hkv, const int64_t* ctx_off,
                                      const int64_t* g_off, int32_t batch) {
  int64_t max_nb = 0, max_gb = 0;
  for (int b = 0; b < batch; ++b) {
    if (ctx_off[b + 1] - ctx_off[b] > max_nb) max_nb = ctx_off[b + 1] - ctx_off[b];
    if (g_off[b + 1] - g_off[b] > max_gb) max_gb = g_off[b + 1] - g_off[b];
  }
  const int64_t n_tot = ctx_off[batch], g_tot = g_off[batch];
  const int64_t R = Hq / Hkv;
  const int64_t nchunk = (max_nb + kChunkTokens - 1) / kChunkTokens;
  const int64_t nrg = (R * max_gb + kRowsPerGroup - 1) / kRowsPerGroup;
  auto up = [](size_t x) { return (x + 255) & ~(size_t)255; };
  GuideWorkspace w;
  w.stats_off = 0;
  w.lse_off = up((size_t)nchunk * L * Hq * g_tot * sizeof(float2));
  w.raw_off = w.lse_off + up((size_t)L * Hq * g_tot * sizeof(float));
  w.total = w.raw_off + up((size_t)nrg * L * Hkv * n_tot * sizeof(float));
  return w;
}

hipError_t launch_guide_scores(const GuideArgs& a, int head_dim, hipStream_t stream) {
  if (head_dim == 128) return launch_d<128>(a, stream);
  return launch_d<64>(a, stream);
}

}  // namespace tp
