// The prefill's attention for the appended guide rows (Sec. 3.2: the task guide is appended
// after the context and attends causally, so guide row j sees the N context keys and guide
// keys 0..j).  Its outputs are the rows' attention output O (what the prefill passes on) and
// each row's log-sum-exp over the keys it sees, which is the normaliser of the attention map
// Sec. 3.2 slices A from: tp_guide_scores_lse / tp_evict(guide_lse) take it, so the eviction
// needs one more sweep over K on top of this one instead of two.
//
// Flash-attention style, split over the context in chunks: one workgroup per (sequence,
// layer, KV head, chunk, group of <= 256 guide rows), eight waves, wave w owning 32 rows.  Per
// 32-token sub-tile, shared by the waves through LDS (double-buffered, one barrier per
// sub-tile):
//   S^T = K Q^T on v_mfma_f32_32x32x16_bf16 (tokens on M, rows on N), so a lane holds one row
//       and 16 tokens (the score passes' pass-1 layout) and the row's running maximum and sum
//       stay in the lane (and its partner lane 32 apart, which holds the other 16 tokens);
//   P  = exp2(S c - m), m raised only when a logit exceeds it by more than kLazyRaise (the
//       maximum needs only to be a logit already seen, so rescaling O is rare);
//   O^T += V^T P^T on the same instruction (d on M, rows on N): the B operand is the lane's own
//       16 probabilities in bf16, the contraction index mapped to exactly the tokens the lane
//       holds, and the A operand reads V transposed from LDS, where each sub-tile is staged
//       d-major.
// Each workgroup writes its rows' partial (max, sum) and unnormalised O; the guide's own keys
// are one more chunk, with the causal mask.  A merge kernel combines the chunks.
#include "tile_common.h"
#include "tp_internal.h"

namespace tp {
namespace {

constexpr int kAttnThreads = 512;  // 8 waves, one per 32-row block of a row group
constexpr int kAttnWaves = kAttnThreads / 64;
constexpr float kLazyRaise = 8.0f;  // log2 units: probabilities stay below 2^8 between raises
constexpr int kVtStride = 64;       // bytes per d-row of a transposed V sub-tile (32 tokens)

// Byte offset of token tk of d-row d in a transposed V sub-tile: groups of 4 tokens (8 bytes)
// are permuted within the row by d/8, so the 16 d-rows written together by one load of
// 8 d-values per thread do not all land on one bank.
__device__ inline int vt_off(int d, int tk) {
  return d * kVtStride + ((((tk >> 2) ^ (d >> 3)) & 7) << 3) + ((tk & 3) << 1);
}

// Issue the copy of K sub-tile rows [t0, t0 + 32) of `ksrc` (rows past ntok repeat its last
// row) into `kbuf` in the score passes' staged layout: the kilobyte pieces go to the first
// waves, one each, so the whole workgroup shares the tile.
template <int D>
__device__ inline void stage_k(const char* ksrc, int t0, int ntok, char* kbuf, int wave) {
  using C = Cfg<D>;
  constexpr int kKBs = 32 / C::kTokPerKB;
  if (wave >= kKBs) return;
  const int lane = threadIdx.x & 63;
  const int tl = wave * C::kTokPerKB + lane / C::kPieces;
  const int p = (lane % C::kPieces) ^ swz<D>(tl);
  const int tok = min(t0 + tl, ntok - 1);
  const char* src = ksrc + (uint32_t)tok * C::kRowBytes + p * 16;
  __builtin_amdgcn_global_load_lds((const void*)src, (__attribute__((address_space(3))) void*)(kbuf + wave * 1024), 16,
                                   0, 0);
}

// Thread t of the first 32 * D/8 threads holds 16 bytes (d-values 8p .. 8p+7 of token tk) of
// a V sub-tile: loaded here, written transposed by write_vt.
template <int D>
__device__ inline uint4 load_v(const uint16_t* vsrc, int t0, int ntok) {
  constexpr int kPieces = D / 8;
  const int tid = threadIdx.x;
  if (tid >= 32 * kPieces) return make_uint4(0, 0, 0, 0);
  const int tk = tid / kPieces, p = tid % kPieces;
  const int tok = min(t0 + tk, ntok - 1);
  return *(const uint4*)(vsrc + (int64_t)tok * D + p * 8);
}

template <int D>
__device__ inline void write_vt(char* vt, const uint4& x) {
  constexpr int kPieces = D / 8;
  const int tid = threadIdx.x;
  if (tid >= 32 * kPieces) return;
  const int tk = tid / kPieces, d0 = (tid % kPieces) * 8;
  const uint32_t w[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
  for (int e = 0; e < 8; ++e)
    *(uint16_t*)(vt + vt_off(d0 + e, tk)) = (uint16_t)(w[e >> 1] >> (16 * (e & 1)));
}

// A operand of O^T += V^T P^T for k-step s2 and d-block db: V^T[d][k] with d = 32 db + lane%32
// and the contraction index k = 8 (lane/32) + j standing for token 16 s2 + 8 (j/4) +
// 4 (lane/32) + j%4, the tokens whose probabilities the lane holds (acc[8 s2 + j]).
__device__ inline Frag read_vfrag(const char* vt, int db, int s2) {
  const int lane = threadIdx.x & 63;
  const int d = 32 * db + (lane & 31);
  const int h = lane >> 5;
  Frag f;
  const uint2 lo = *(const uint2*)(vt + vt_off(d, 16 * s2 + 4 * h));
  const uint2 hi = *(const uint2*)(vt + vt_off(d, 16 * s2 + 8 + 4 * h));
  f.u = make_uint4(lo.x, lo.y, hi.x, hi.y);
  return f;
}

struct AttnUnit {
  int b, seg, l, h, rg, chunk;
  bool guide;              // the guide's own keys (causal) rather than a context chunk
  int64_t n0, nb, g0;
  int gb, rows, row0, nrows, ntok, slot;
};

__device__ inline bool attn_unit(const AttnArgs& a, AttnUnit& u) {
  u.b = blockIdx.z / a.nrg_max;
  u.rg = blockIdx.z % a.nrg_max;
  u.seg = blockIdx.y;
  u.chunk = blockIdx.x;
  u.l = u.seg / a.Hkv;
  u.h = u.seg % a.Hkv;
  u.n0 = a.bt.ctx_off[u.b];
  u.nb = a.bt.ctx_off[u.b + 1] - u.n0;
  u.g0 = a.bt.g_off[u.b];
  u.gb = (int)(a.bt.g_off[u.b + 1] - u.g0);
  u.rows = a.R * u.gb;
  u.row0 = u.rg * kRowsPerGroup;
  if (u.row0 >= u.rows) return false;
  u.nrows = u.rows - u.row0 < kRowsPerGroup ? u.rows - u.row0 : kRowsPerGroup;
  const int nch = (int)((u.nb + a.chunk - 1) / a.chunk);
  if (u.chunk < nch) {
    u.guide = false;
    const int64_t c0 = (int64_t)u.chunk * a.chunk;
    u.ntok = (int)(u.nb - c0 < a.chunk ? u.nb - c0 : a.chunk);
    u.slot = u.chunk;
    return true;
  }
  if (a.kg != nullptr && u.chunk == a.nchunk_max) {
    u.guide = true;
    u.ntok = u.gb;
    u.slot = a.nchunk_max;
    return true;
  }
  return false;
}

template <int D>
__global__ __launch_bounds__(kAttnThreads, 1) void k_guide_fwd(AttnArgs a) {
  AttnUnit u;
  if (!attn_unit(a, u)) return;
  using C = Cfg<D>;
  constexpr int KS = C::kSteps;
  constexpr int NDB = D / 32;  // 32-wide d-blocks of O
  __shared__ __attribute__((aligned(1024))) char kst[2][C::kStageBytes];
  __shared__ __attribute__((aligned(16))) char vts[2][D * kVtStride];
  const int lane = threadIdx.x & 63;
  const int wave = uniform(threadIdx.x >> 6);
  const bool active = 32 * wave < u.nrows;
  // this lane's guide row (rows past the group's end repeat its last row; never written)
  const int rho_raw = u.row0 + 32 * wave + (lane & 31);
  const bool row_ok = rho_raw < u.row0 + u.nrows;
  const int rho = row_ok ? rho_raw : u.row0 + u.nrows - 1;
  const int r = rho / u.gb, j = rho % u.gb;
  const int64_t grow = ((int64_t)u.l * a.Hq + (int64_t)u.h * a.R + r) * a.g_tot + u.g0 + j;
  // the K fragments' contraction order: half-wave h holds d-columns h D/2 + 8 s .. + 8 at k-step s
  Frag qf[KS];
#pragma unroll
  for (int s = 0; s < KS; ++s) qf[s].u = *(const uint4*)(a.q + grow * D + (lane >> 5) * (D / 2) + 8 * s);
  const uint16_t* ksrc;
  const uint16_t* vsrc;
  if (u.guide) {
    ksrc = a.kg + ((int64_t)u.seg * a.g_tot + u.g0) * D;
    vsrc = a.vg + ((int64_t)u.seg * a.g_tot + u.g0) * D;
  } else {
    ksrc = a.k + ((int64_t)u.seg * a.n_tot + u.n0 + (int64_t)u.chunk * a.chunk) * D;
    vsrc = a.v + ((int64_t)u.seg * a.n_tot + u.n0 + (int64_t)u.chunk * a.chunk) * D;
  }
  const int nsub = (u.ntok + 31) / 32;

  float m = kNoMax, lsum = 0.f;
  f32x16 ot[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db) ot[db] = (f32x16){};

  stage_k<D>((const char*)ksrc, 0, u.ntok, kst[0], wave);
  write_vt<D>(vts[0], load_v<D>(vsrc, 0, u.ntok));
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  for (int t = 0; t < nsub; ++t) {
    const int cur = t & 1, nxt = cur ^ 1;
    uint4 vn = make_uint4(0, 0, 0, 0);
    if (t + 1 < nsub) {
      stage_k<D>((const char*)ksrc, 32 * (t + 1), u.ntok, kst[nxt], wave);
      vn = load_v<D>(vsrc, 32 * (t + 1), u.ntok);
    }
    if (active) {
      Frag kf[KS];
      read_kfrag<D>(kst[cur], kf);
      f32x16 acc = {};
#pragma unroll
      for (int s = 0; s < KS; ++s) acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[s].v, qf[s].v, acc, 0, 0, 0);
      // acc[i]: token 32 t + (i/4)*8 + (lane/32)*4 + i%4 of the unit, the lane's row
      float mx = -INFINITY;
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int tok = 32 * t + (i >> 2) * 8 + (lane >> 5) * 4 + (i & 3);
        const bool seen = tok < u.ntok && (!u.guide || tok <= j);
        acc[i] = seen ? acc[i] : -INFINITY;
        mx = fmaxf(mx, acc[i]);
      }
      mx = fmaxf(mx, __shfl_xor(mx, 32)) * a.c;  // the row's maximum over the sub-tile (c > 0)
      const bool raise = mx > m + kLazyRaise;
      if (__builtin_amdgcn_ballot_w64(raise)) {  // rare after a row's first sub-tile
        const float mn = raise ? mx : m;
        const float al = __builtin_amdgcn_exp2f(m - mn);
        lsum *= al;
#pragma unroll
        for (int db = 0; db < NDB; ++db)
#pragma unroll
          for (int i = 0; i < 16; ++i) ot[db][i] *= al;
        m = mn;
      }
      float p[16];
      float ps = 0.f;
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        p[i] = __builtin_amdgcn_exp2f(fmaf(acc[i], a.c, -m));
        ps += p[i];
      }
      lsum += ps;
      bf16x8 pb[2];
#pragma unroll
      for (int s2 = 0; s2 < 2; ++s2)
#pragma unroll
        for (int jj = 0; jj < 8; ++jj) pb[s2][jj] = (__bf16)p[8 * s2 + jj];
#pragma unroll
      for (int db = 0; db < NDB; ++db)
#pragma unroll
        for (int s2 = 0; s2 < 2; ++s2) {
          const Frag vf = read_vfrag(vts[cur], db, s2);
          ot[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf.v, pb[s2], ot[db], 0, 0, 0);
        }
    }
    if (t + 1 < nsub) write_vt<D>(vts[nxt], vn);
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
  }
  if (!active) return;
  lsum += __shfl_xor(lsum, 32);  // the row's other 16 tokens of every sub-tile
  if (!row_ok) return;
  const int64_t rows_tot = (int64_t)a.L * a.Hq * a.g_tot;
  const int64_t prow = (int64_t)u.slot * rows_tot + grow;
  if (lane < 32) a.pstat[prow] = make_float2(m, lsum);
  float* po = a.po + prow * D;
  // ot[db][i]: d = 32 db + (i/4)*8 + (lane/32)*4 + i%4 of the lane's row
#pragma unroll
  for (int db = 0; db < NDB; ++db)
#pragma unroll
    for (int q = 0; q < 4; ++q)
      *(float4*)(po + 32 * db + 8 * q + 4 * (lane >> 5)) =
          make_float4(ot[db][4 * q], ot[db][4 * q + 1], ot[db][4 * q + 2], ot[db][4 * q + 3]);
}

// One wave per guide row: the chunks' partial (max, sum) and O combined into the row's output
// and its natural-log normaliser.
template <int D>
__global__ __launch_bounds__(256) void k_guide_fwd_merge(AttnArgs a) {
  const int b = blockIdx.y;
  const int lane = threadIdx.x & 63;
  const int64_t g0 = a.bt.g_off[b];
  const int gb = (int)(a.bt.g_off[b + 1] - g0);
  const int64_t nb = a.bt.ctx_off[b + 1] - a.bt.ctx_off[b];
  const int64_t idx = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (idx >= (int64_t)a.L * a.Hq * gb) return;
  const int64_t per_layer = (int64_t)a.Hq * gb;
  const int64_t l = idx / per_layer, rem = idx - l * per_layer;
  const int64_t qh = rem / gb, jj = rem - qh * gb;
  const int64_t grow = (l * a.Hq + qh) * a.g_tot + g0 + jj;
  const int64_t rows_tot = (int64_t)a.L * a.Hq * a.g_tot;
  const int nch = (int)((nb + a.chunk - 1) / a.chunk);
  const int nslot = a.kg != nullptr ? nch + 1 : nch;
  auto slot_of = [&](int c) { return c < nch ? c : a.nchunk_max; };
  float mstar = kNoMax;
  for (int c = 0; c < nslot; ++c) mstar = fmaxf(mstar, a.pstat[(int64_t)slot_of(c) * rows_tot + grow].x);
  float tot = 0.f;
  float acc[D / 64] = {};
  for (int c = 0; c < nslot; ++c) {
    const int64_t prow = (int64_t)slot_of(c) * rows_tot + grow;
    const float2 st = a.pstat[prow];
    const float w = __builtin_amdgcn_exp2f(st.x - mstar);
    tot += w * st.y;
#pragma unroll
    for (int e = 0; e < D / 64; ++e) acc[e] += w * a.po[prow * D + lane + 64 * e];
  }
#pragma unroll
  for (int e = 0; e < D / 64; ++e) a.o[grow * D + lane + 64 * e] = acc[e] / tot;
  if (lane == 0) a.lse[grow] = (mstar + log2f(tot)) * 0.69314718055994531f;
}

}  // namespace

AttnWorkspace attn_workspace_layout(int32_t L, int32_t Hq, int32_t Hkv, int32_t head_dim, const int64_t* ctx_off,
                                    const int64_t* g_off, int32_t batch) {
  (void)Hkv;
  int64_t max_nb = 0;
  for (int b = 0; b < batch; ++b)
    if (ctx_off[b + 1] - ctx_off[b] > max_nb) max_nb = ctx_off[b + 1] - ctx_off[b];
  const int64_t chunk = attn_chunk_tokens(ctx_off, batch);
  const int64_t nslot = (max_nb + chunk - 1) / chunk + 1;  // the context chunks, then the guide keys
  const int64_t rows = (int64_t)L * Hq * g_off[batch];
  auto up = [](size_t x) { return (x + 255) & ~(size_t)255; };
  AttnWorkspace w;
  w.pstat_off = 0;
  w.po_off = up((size_t)nslot * rows * sizeof(float2));
  w.total = w.po_off + up((size_t)nslot * rows * head_dim * sizeof(float));
  return w;
}

hipError_t launch_guide_attention(const AttnArgs& a, int head_dim, hipStream_t stream) {
  int64_t max_gb = 0;
  for (int b = 0; b < a.bt.batch; ++b)
    if (a.bt.g_off[b + 1] - a.bt.g_off[b] > max_gb) max_gb = a.bt.g_off[b + 1] - a.bt.g_off[b];
  const dim3 grid((unsigned)(a.nchunk_max + (a.kg != nullptr ? 1 : 0)), (unsigned)(a.L * a.Hkv),
                  (unsigned)(a.bt.batch * a.nrg_max));
  const dim3 mgrid((unsigned)((a.L * a.Hq * max_gb + 3) / 4), (unsigned)a.bt.batch);
  if (head_dim == 128) {
    hipLaunchKernelGGL(k_guide_fwd<128>, grid, dim3(kAttnThreads), 0, stream, a);
    hipLaunchKernelGGL(k_guide_fwd_merge<128>, mgrid, dim3(256), 0, stream, a);
  } else {
    hipLaunchKernelGGL(k_guide_fwd<64>, grid, dim3(kAttnThreads), 0, stream, a);
    hipLaunchKernelGGL(k_guide_fwd_merge<64>, mgrid, dim3(256), 0, stream, a);
  }
  return hipGetLastError();
}

}  // namespace tp
