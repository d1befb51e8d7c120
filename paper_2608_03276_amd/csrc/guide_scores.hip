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
// streamed HBM -> LDS in 128-token tiles with direct global-to-LDS loads (double-buffered,
// XOR-swizzled); the guide queries of a wave stay in registers for its whole chunk.  Each
// wave software-pipelines its 32x32 units: the MFMA chain of unit u+1 is interleaved with
// the exp/add work of unit u, so the matrix core and the vector ALU run concurrently.
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
  static constexpr int kPieces = D / 8;                     // 16-byte pieces per token row
  static constexpr int kRowBytes = D * 2;
  static constexpr int kTileBytes = kMacroTokens * kRowBytes;
  static constexpr int kRowsPerLoad = 1024 / kRowBytes;     // token rows one wave-wide 16 B load fills
  static constexpr int kLoadsPerWave = kTileBytes / 1024 / 4;
};

struct Work {
  int b, seg, l, h, rg, chunk;
  int64_t n0, nb, c0, c1, g0;
  int gb, rows, row0, nrows;
};

__device__ inline int uniform(int x) { return __builtin_amdgcn_readfirstlane(x); }

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

template <int D>
__device__ inline void load_q(const GuideArgs& a, const Work& w, int wrow0, Frag (&qf)[2][Cfg<D>::kSteps]) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int rb = 0; rb < 2; ++rb) {
    const int rho = wrow0 + rb * 32 + (lane & 31);
    if (rho < w.rows) {
      const uint16_t* src = a.q + grow_of(a, w, rho) * D + (lane >> 5) * (D / 2);
#pragma unroll
      for (int s = 0; s < Cfg<D>::kSteps; ++s) qf[rb][s].u = *(const uint4*)(src + 8 * s);
    } else {
#pragma unroll
      for (int s = 0; s < Cfg<D>::kSteps; ++s) qf[rb][s].u = make_uint4(0, 0, 0, 0);
    }
  }
}

// The K tile of 128 tokens sits in LDS without padding; the 16-byte piece p of token row r
// is stored at piece p ^ (r mod kPieces), which makes the fragment reads below conflict-free.
// Each wave fills its share with direct global->LDS loads (64 lanes x 16 B = 1 KB per
// instruction, lane i landing at byte 16 i).  Tokens past the chunk end re-load the last
// valid row, so every LDS byte holds finite data and no load leaves the sequence.
template <int D>
__device__ inline void issue_tile(const uint16_t* kseg, int64_t t0, int64_t c1, char* buf, int wave) {
  using C = Cfg<D>;
  const int lane = threadIdx.x & 63;
  const char* base = (const char*)(kseg + t0 * D);  // wave-uniform
  const int last = (int)(c1 - 1 - t0);               // last valid row of this tile
#pragma unroll
  for (int j = 0; j < C::kLoadsPerWave; ++j) {
    const int blk = wave * C::kLoadsPerWave + j;  // 1 KB block of the tile
    int r = blk * C::kRowsPerLoad + lane / C::kPieces;
    const int p = (lane % C::kPieces) ^ (r & (C::kPieces - 1));
    r = r < last ? r : last;
    __builtin_amdgcn_global_load_lds((const void*)(base + (uint32_t)(r * C::kRowBytes + p * 16)),
                                     (__attribute__((address_space(3))) void*)(buf + blk * 1024), 16, 0, 0);
  }
}

// K fragment of sub-tile `st` for this lane: token st*32 + lane%32, the d-columns of its
// half-wave (lane/32), k-step s covering columns half*D/2 + 8s .. +8.
template <int D>
__device__ inline void read_kfrag(const char* buf, int st, Frag (&kf)[Cfg<D>::kSteps]) {
  using C = Cfg<D>;
  const int lane = threadIdx.x & 63;
  const int r = st * 32 + (lane & 31);
  const char* row = buf + r * C::kRowBytes;
#pragma unroll
  for (int s = 0; s < C::kSteps; ++s) {
    const int p = (lane >> 5) * (C::kPieces / 2) + s;
    kf[s].u = *(const uint4*)(row + ((p ^ (r & (C::kPieces - 1))) * 16));
  }
}

template <int KS>
__device__ inline f32x16 mfma_chain(const Frag (&a)[KS], const Frag (&b)[KS]) {
  f32x16 acc = {};
#pragma unroll
  for (int s = 0; s < KS; ++s) acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[s].v, b[s].v, acc, 0, 0, 0);
  return acc;
}

__device__ inline void merge_stats(float& m, float& s, float m2, float s2) {
  const float mn = fmaxf(m, m2);
  if (mn == -INFINITY) return;
  s = s * __builtin_amdgcn_exp2f(m - mn) + s2 * __builtin_amdgcn_exp2f(m2 - mn);
  m = mn;
}

// MFMA / VALU interleave: after each MFMA of the next unit, let `n` VALU ops issue.
template <int KS, int N>
__device__ inline void interleave() {
#pragma unroll
  for (int i = 0; i < KS; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    __builtin_amdgcn_sched_group_barrier(0x002, N, 0);
  }
}

// ---------------------------------------------------------------------------- pass 1
// Online (max, sum) of the scaled logits of one unit (32 tokens x 32 rows): acc[i] is the
// logit of token (i/4)*8 + (lane/32)*4 + i%4 and row lane%32.
template <bool PARTIAL>
__device__ inline void stats_update(const f32x16& acc, float c, float& m, float& s, int nvalid) {
  const int lane = threadIdx.x & 63;
  float x[16];
#pragma unroll
  for (int i = 0; i < 16; ++i) x[i] = acc[i];
  if (PARTIAL) {
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int tok = (i >> 2) * 8 + (lane >> 5) * 4 + (i & 3);
      x[i] = tok < nvalid ? x[i] : -INFINITY;
    }
  }
  float t0 = fmaxf(fmaxf(x[0], x[1]), x[2]), t1 = fmaxf(fmaxf(x[3], x[4]), x[5]);
  float t2 = fmaxf(fmaxf(x[6], x[7]), x[8]), t3 = fmaxf(fmaxf(x[9], x[10]), x[11]);
  float t4 = fmaxf(fmaxf(x[12], x[13]), x[14]);
  const float tmax = fmaxf(fmaxf(fmaxf(t0, t1), x[15]), fmaxf(fmaxf(t2, t3), t4));
  const float mn = fmaxf(m, tmax * c);
  float e0 = 0.f, e1 = 0.f, e2 = 0.f, e3 = 0.f;
#pragma unroll
  for (int i = 0; i < 16; i += 4) {
    e0 += __builtin_amdgcn_exp2f(fmaf(x[i + 0], c, -mn));
    e1 += __builtin_amdgcn_exp2f(fmaf(x[i + 1], c, -mn));
    e2 += __builtin_amdgcn_exp2f(fmaf(x[i + 2], c, -mn));
    e3 += __builtin_amdgcn_exp2f(fmaf(x[i + 3], c, -mn));
  }
  const float sn = s * __builtin_amdgcn_exp2f(m - mn) + ((e0 + e1) + (e2 + e3));
  if (PARTIAL) {  // a lane whose tokens are all masked so far keeps (-inf, 0)
    const bool keep = mn == -INFINITY;
    s = keep ? s : sn;
    m = keep ? m : mn;
  } else {
    s = sn;
    m = mn;
  }
}

template <int D, int WR, bool PARTIAL>
__device__ inline void stats_macro(const char* buf, const Frag (&qf)[2][Cfg<D>::kSteps], float c, int wt,
                                   int64_t t0, int64_t c1, float (&m)[2], float (&s)[2]) {
  using C = Cfg<D>;
  constexpr int WT = 4 / WR, SUBS = 4 / WT, UNITS = 2 * SUBS;
  Frag kf[2][C::kSteps];
  read_kfrag<D>(buf, wt, kf[0]);
  f32x16 acc = mfma_chain<C::kSteps>(kf[0], qf[0]);
#pragma unroll
  for (int u = 0; u < UNITS; ++u) {
    const int si = u >> 1, rb = u & 1;
    f32x16 nxt = {};
    if (u + 1 < UNITS) {
      const int si1 = (u + 1) >> 1, rb1 = (u + 1) & 1;
      if (rb == 0 && si + 1 < SUBS) read_kfrag<D>(buf, wt + (si + 1) * WT, kf[(si + 1) & 1]);
      nxt = mfma_chain<C::kSteps>(kf[si1 & 1], qf[rb1]);
    }
    const int64_t sub0 = t0 + (wt + si * WT) * 32;
    const int nvalid = c1 - sub0 >= 32 ? 32 : (c1 > sub0 ? (int)(c1 - sub0) : 0);
    stats_update<PARTIAL>(acc, c, m[rb], s[rb], nvalid);
    interleave<C::kSteps, 7>();
    acc = nxt;
  }
}

template <int D>
__global__ __launch_bounds__(kGuideThreads, 2) void k_guide_stats(GuideArgs a) {
  Work w;
  if (!decode(a, w)) return;
  using C = Cfg<D>;
  __shared__ __attribute__((aligned(1024))) char kt[2][C::kTileBytes];
  __shared__ float2 xch[4][kRowsPerGroup];

  const int lane = threadIdx.x & 63;
  const int wave = uniform(threadIdx.x >> 6);
  const int WR = w.nrows > 128 ? 4 : (w.nrows > 64 ? 2 : 1);
  const int WT = 4 / WR;
  const int wr = wave % WR, wt = wave / WR;
  const int wrow0 = w.row0 + wr * kRowsPerWave;

  Frag qf[2][C::kSteps];
  load_q<D>(a, w, wrow0, qf);
  float m[2] = {-INFINITY, -INFINITY}, s[2] = {0.f, 0.f};

  const uint16_t* kseg = a.k + ((int64_t)w.seg * a.n_tot + w.n0) * D;
  const int ntiles = (int)((w.c1 - w.c0 + kMacroTokens - 1) / kMacroTokens);
  issue_tile<D>(kseg, w.c0, w.c1, kt[0], wave);
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();

  for (int it = 0; it < ntiles; ++it) {
    const int64_t t0 = w.c0 + (int64_t)it * kMacroTokens;
    if (it + 1 < ntiles) issue_tile<D>(kseg, t0 + kMacroTokens, w.c1, kt[(it + 1) & 1], wave);
    const char* buf = kt[it & 1];
    if (t0 + kMacroTokens <= w.c1) {
      if (WR == 4) stats_macro<D, 4, false>(buf, qf, a.c, wt, t0, w.c1, m, s);
      else if (WR == 2) stats_macro<D, 2, false>(buf, qf, a.c, wt, t0, w.c1, m, s);
      else stats_macro<D, 1, false>(buf, qf, a.c, wt, t0, w.c1, m, s);
    } else {
      if (WR == 4) stats_macro<D, 4, true>(buf, qf, a.c, wt, t0, w.c1, m, s);
      else if (WR == 2) stats_macro<D, 2, true>(buf, qf, a.c, wt, t0, w.c1, m, s);
      else stats_macro<D, 1, true>(buf, qf, a.c, wt, t0, w.c1, m, s);
    }
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
  }

  // The two half-waves hold the same rows over different tokens.
#pragma unroll
  for (int rb = 0; rb < 2; ++rb) {
    const float mo = __shfl_xor(m[rb], 32);
    const float so = __shfl_xor(s[rb], 32);
    merge_stats(m[rb], s[rb], mo, so);
    if (lane < 32) xch[wt][wr * kRowsPerWave + rb * 32 + lane] = make_float2(m[rb], s[rb]);
  }
  __syncthreads();
  const int t = threadIdx.x;
  if (t < WR * kRowsPerWave) {
    const int rho = w.row0 + t;
    if (rho < w.rows) {
      float mm = xch[0][t].x, ss = xch[0][t].y;
      for (int q = 1; q < WT; ++q) merge_stats(mm, ss, xch[q][t].x, xch[q][t].y);
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
// Normalised weights of one unit (32 rows x 32 tokens): acc[i] is the logit of row
// (i/4)*8 + (lane/32)*4 + i%4 and token lane%32; returns the lane's sum over its 16 rows.
__device__ inline float attn_sum(const f32x16& acc, float c, const float (&lz)[16]) {
  float e0 = 0.f, e1 = 0.f, e2 = 0.f, e3 = 0.f;
#pragma unroll
  for (int i = 0; i < 16; i += 4) {
    e0 += __builtin_amdgcn_exp2f(fmaf(acc[i + 0], c, -lz[i + 0]));
    e1 += __builtin_amdgcn_exp2f(fmaf(acc[i + 1], c, -lz[i + 1]));
    e2 += __builtin_amdgcn_exp2f(fmaf(acc[i + 2], c, -lz[i + 2]));
    e3 += __builtin_amdgcn_exp2f(fmaf(acc[i + 3], c, -lz[i + 3]));
  }
  return (e0 + e1) + (e2 + e3);
}

template <int D, int WR>
__device__ inline void attn_macro(const char* buf, const Frag (&qf)[2][Cfg<D>::kSteps], const float (&lz)[2][16],
                                  float c, int wt, float* red_row) {
  using C = Cfg<D>;
  constexpr int WT = 4 / WR, SUBS = 4 / WT, UNITS = 2 * SUBS;
  const int lane = threadIdx.x & 63;
  Frag kf[2][C::kSteps];
  read_kfrag<D>(buf, wt, kf[0]);
  f32x16 acc = mfma_chain<C::kSteps>(qf[0], kf[0]);
  float part = 0.f;
#pragma unroll
  for (int u = 0; u < UNITS; ++u) {
    const int si = u >> 1, rb = u & 1;
    f32x16 nxt = {};
    if (u + 1 < UNITS) {
      const int si1 = (u + 1) >> 1, rb1 = (u + 1) & 1;
      if (rb == 0 && si + 1 < SUBS) read_kfrag<D>(buf, wt + (si + 1) * WT, kf[(si + 1) & 1]);
      nxt = mfma_chain<C::kSteps>(qf[rb1], kf[si1 & 1]);
    }
    part += attn_sum(acc, c, lz[rb]);
    interleave<C::kSteps, 6>();
    if (rb == 1) {
      part += __shfl_xor(part, 32);
      red_row[(wt + si * WT) * 32 + (lane & 31)] = part;  // both half-waves hold the same sum
      part = 0.f;
    }
    acc = nxt;
  }
}

template <int D>
__global__ __launch_bounds__(kGuideThreads, 2) void k_guide_attn(GuideArgs a) {
  Work w;
  if (!decode(a, w)) return;
  using C = Cfg<D>;
  __shared__ __attribute__((aligned(1024))) char kt[2][C::kTileBytes];
  __shared__ float red[2][4][kMacroTokens];

  const int lane = threadIdx.x & 63;
  const int wave = uniform(threadIdx.x >> 6);
  const int WR = w.nrows > 128 ? 4 : (w.nrows > 64 ? 2 : 1);
  const int wr = wave % WR, wt = wave / WR;
  const int wrow0 = w.row0 + wr * kRowsPerWave;

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
  issue_tile<D>(kseg, w.c0, w.c1, kt[0], wave);
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();

  for (int it = 0; it < ntiles; ++it) {
    const int64_t t0 = w.c0 + (int64_t)it * kMacroTokens;
    if (it + 1 < ntiles) issue_tile<D>(kseg, t0 + kMacroTokens, w.c1, kt[(it + 1) & 1], wave);
    const char* buf = kt[it & 1];
    float* red_row = red[it & 1][wr];
    if (WR == 4) attn_macro<D, 4>(buf, qf, lz, a.c, wt, red_row);
    else if (WR == 2) attn_macro<D, 2>(buf, qf, lz, a.c, wt, red_row);
    else attn_macro<D, 1>(buf, qf, lz, a.c, wt, red_row);
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (threadIdx.x < kMacroTokens) {
      const int64_t tok = t0 + threadIdx.x;
      if (tok < w.c1) {
        float v = red[it & 1][0][threadIdx.x];
        for (int q = 1; q < WR; ++q) v += red[it & 1][q][threadIdx.x];
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
