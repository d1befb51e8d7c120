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
// orientations because the A and B operand layouts of the instruction coincide.
//
// A workgroup (8 waves, one per CU) takes one chunk of 8192 tokens and one group of <= 256
// guide rows.  The group's queries sit in LDS for the whole chunk.  Each wave streams its
// own 32-token K sub-tiles: an asynchronous global->LDS copy into the wave's private
// staging buffer runs while the wave computes the previous sub-tile from registers, so no
// barrier is needed inside the main loop and the K fragments take no prefetch registers.
// Inside a sub-tile the wave is software-pipelined: the MFMAs of one pair of 32-row blocks
// run while the vector ALU does the softmax work of the previous pair.
#include "tile_common.h"
#include "tp_internal.h"

namespace tp {
namespace {

struct Work {
  int b, seg, l, h, rg, chunk;
  int64_t n0, nb, c0, c1, g0;
  int gb, rows, row0, nrows;
};


// Workgroup -> (sequence, row group, chunk, segment).  Each sequence owns a contiguous range
// of workgroup ids (wg_off).  Within it the work units (segment, chunk) are numbered
// consecutively and dealt round-robin to the 8 XCDs, as consecutive workgroup ids are, so
// every XCD gets an even share whatever the number of chunks; the row groups of one unit get
// ids 8 apart, so they land on the same XCD and share the chunk's K through its L2.
__device__ inline bool decode(const GuideArgs& a, Work& w) {
  const int x = blockIdx.x;
  int b = 0;
  while (b + 1 < a.bt.batch && x >= a.wg_off[b + 1]) ++b;
  w.b = b;
  const int xb = x - a.wg_off[b];
  w.n0 = a.bt.ctx_off[b];
  w.nb = a.bt.ctx_off[b + 1] - w.n0;
  w.g0 = a.bt.g_off[b];
  w.gb = (int)(a.bt.g_off[b + 1] - w.g0);
  w.rows = a.R * w.gb;
  const int nrg = (w.rows + kRowsPerGroup - 1) / kRowsPerGroup;
  const int nchunk = (int)((w.nb + a.chunk - 1) / a.chunk);
  const int xcd = xb & 7, slot = xb >> 3;
  w.rg = slot % nrg;
  const int64_t unit = (int64_t)(slot / nrg) * 8 + xcd;
  if (unit >= (int64_t)a.L * a.Hkv * nchunk) return false;  // padding to a multiple of 8
  w.seg = (int)(unit / nchunk);
  w.chunk = (int)(unit % nchunk);
  w.l = w.seg / a.Hkv;
  w.h = w.seg % a.Hkv;
  w.c0 = (int64_t)w.chunk * a.chunk;
  w.c1 = w.c0 + a.chunk < w.nb ? w.c0 + a.chunk : w.nb;
  w.row0 = w.rg * kRowsPerGroup;
  w.nrows = w.rows - w.row0 < kRowsPerGroup ? w.rows - w.row0 : kRowsPerGroup;
  return true;
}

// Global row id (index into q_guide rows, stats and lse) of guide row rho of the segment.
__device__ inline int64_t grow_of(const GuideArgs& a, const Work& w, int rho) {
  const int r = rho / w.gb, j = rho - r * w.gb;
  const int64_t qh = (int64_t)w.h * a.R + r;
  return ((int64_t)w.l * a.Hq + qh) * a.g_tot + w.g0 + j;
}

// The row group's guide queries in LDS: local row rr at rr * kStride bytes.  The 16-byte pad
// per row makes 16 consecutive rows start on different bank groups, so the fragment reads
// below are conflict-free, and every fragment address is one per-lane base plus a constant.
// Rows past the group's end repeat its last row (finite data, discarded later).
template <int D>
__device__ inline void stage_q(const GuideArgs& a, const Work& w, char* qs, int nrows_pad) {
  using C = Cfg<D>;
  for (int t = threadIdx.x; t < nrows_pad * C::kPieces; t += kGuideThreads) {
    const int rr = t / C::kPieces, p = t % C::kPieces;
    const int src_row = rr < w.nrows ? rr : w.nrows - 1;
    const uint4 v = *(const uint4*)(a.q + grow_of(a, w, w.row0 + src_row) * D + p * 8);
    *(uint4*)(qs + rr * C::kStride + p * 16) = v;
  }
}

// Q fragment of local row block rb: row 32 rb + lane%32, the d-columns of this half-wave.
template <int D>
__device__ inline void read_qfrag(const char* qs, int rb, Frag (&qf)[Cfg<D>::kSteps]) {
  using C = Cfg<D>;
  const int lane = threadIdx.x & 63;
  const char* base = qs + (lane & 31) * C::kStride + (lane >> 5) * C::kRowBytes / 2 + rb * 32 * C::kStride;
#pragma unroll
  for (int s = 0; s < C::kSteps; ++s) qf[s].u = *(const uint4*)(base + 16 * s);
}

// Issue the copy of the sub-tile starting at chunk token t0 into `kbuf`: each instruction
// moves 1 KB of consecutive K rows (coalesced); lane i fills slot i of that kilobyte, so it
// fetches the piece that the swizzle assigns to that slot.  Tokens past the chunk's `ntok`
// repeat its last token (finite data that pass 1 masks and pass 2 never stores).
template <int D>
__device__ inline void dma_subtile(const char* kchunk, int t0, int ntok, char* kbuf) {
  using C = Cfg<D>;
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int j = 0; j < 32 / C::kTokPerKB; ++j) {
    const int tl = j * C::kTokPerKB + lane / C::kPieces;
    const int p = (lane % C::kPieces) ^ swz<D>(tl);
    const int tok = min(t0 + tl, ntok - 1);
    const char* src = kchunk + (uint32_t)tok * C::kRowBytes + p * 16;
    __builtin_amdgcn_global_load_lds((const void*)src, (__attribute__((address_space(3))) void*)(kbuf + j * 1024), 16,
                                     0, 0);
  }
}

// Issue-priority balancing of the two waves that share a SIMD (waves w and w ^ 4).  With equal
// priority the older wave wins most issue slots, finishes its sub-tiles early and leaves
// the other to run alone at the end of the workgroup.  After each sub-tile a wave publishes
// its count and raises its priority while it is behind its partner.  This changes only the
// timing, never which wave computes what.
__device__ inline void balance_issue(int* progress, int wave, int done) {
  if ((threadIdx.x & 63) == 0) progress[wave] = done;
  const int other = uniform(progress[wave ^ 4]);
  if (done < other)
    __builtin_amdgcn_s_setprio(2);
  else if (done == other)
    __builtin_amdgcn_s_setprio(1);
  else
    __builtin_amdgcn_s_setprio(0);
}

// The staging buffer has landed (the wave's copies are complete).  The memory clobber keeps
// the compiler from moving LDS reads of the buffer above the wait.
__device__ inline void wait_copies() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }
// The fragment reads of the buffer are complete, so it may be overwritten.
__device__ inline void wait_lds_reads() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }

// Two independent MFMA chains: row blocks rb, rb+1 against one K sub-tile.  With INIT the
// chains accumulate onto the values already in c0, c1; otherwise they start from zero.
template <int KS, bool Q_IS_A, bool INIT = false>
__device__ inline void mfma_pair(const Frag (&q0)[KS], const Frag (&q1)[KS], const Frag (&k)[KS], f32x16& c0,
                                 f32x16& c1) {
  if (!INIT) {
    c0 = (f32x16){};
    c1 = (f32x16){};
  }
#pragma unroll
  for (int s = 0; s < KS; ++s) {
    if (Q_IS_A) {
      c0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(q0[s].v, k[s].v, c0, 0, 0, 0);
      c1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(q1[s].v, k[s].v, c1, 0, 0, 0);
    } else {
      c0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(k[s].v, q0[s].v, c0, 0, 0, 0);
      c1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(k[s].v, q1[s].v, c1, 0, 0, 0);
    }
  }
}

// Instruction order of one pipeline step: NDS0 LDS reads first, then a little vector work
// (NV0 plain, NT0 transcendental instructions) while they land, then each MFMA followed by
// an even share of the remaining vector work of the previous pair (NV plain, NT
// transcendental, counted separately because the scheduler classes them separately) and
// one of the NDS LDS reads that fetch the next step's query fragments.  The matrix core,
// the vector ALU and the LDS stay busy together, and the LDS latency is covered by a step.
template <int NDS0, int NV0, int NT0, int NDS, int NMFMA, int NV, int NT>
__device__ inline void step_schedule() {
  if (NDS0 > 0) __builtin_amdgcn_sched_group_barrier(0x100, NDS0, 0);
  if (NV0 > 0) __builtin_amdgcn_sched_group_barrier(0x002, NV0, 0);
  if (NT0 > 0) __builtin_amdgcn_sched_group_barrier(0x400, NT0, 0);
#pragma unroll
  for (int i = 0; i < NMFMA; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    __builtin_amdgcn_sched_group_barrier(0x002, NV, 0);
    __builtin_amdgcn_sched_group_barrier(0x400, NT, 0);
    if (i < NDS) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
  }
  __builtin_amdgcn_sched_barrier(0);
}

// Keeps the vector work of a pipeline step inside the step: without a use here the
// compiler sinks it past the loop's branches, away from the MFMAs it should overlap.
__device__ inline void pin(float a, float b, float c, float d) { asm volatile("" ::"v"(a), "v"(b), "v"(c), "v"(d)); }

// ---------------------------------------------------------------------------- pass 1
// Online (max, sum) of one unit (32 tokens x 32 rows): acc[i] is the logit of token
// (i/4)*8 + (lane/32)*4 + i%4 and row lane%32.  c > 0, so max(x) * c = max(x * c).
__device__ inline void stats_update(const f32x16& acc, float c, float& m, float& s) {
  const float mn = fmaxf(m, max16(acc) * c);
  float e[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) e[j] = __builtin_amdgcn_exp2f(fmaf(acc[j], c, -mn));
#pragma unroll
  for (int i = 4; i < 16; i += 4)
#pragma unroll
    for (int j = 0; j < 4; ++j) e[j] += __builtin_amdgcn_exp2f(fmaf(acc[i + j], c, -mn));
  s = fmaf(s, __builtin_amdgcn_exp2f(m - mn), (e[0] + e[1]) + (e[2] + e[3]));
  m = mn;
}

// The unit's terms exp2(x*c - m) against the lane's current maximum m, summed.
__device__ inline float unit_sum(const f32x16& acc, float c, float m) {
  float e[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) e[j] = __builtin_amdgcn_exp2f(fmaf(acc[j], c, -m));
#pragma unroll
  for (int i = 4; i < 16; i += 4)
#pragma unroll
    for (int j = 0; j < 4; ++j) e[j] += __builtin_amdgcn_exp2f(fmaf(acc[i + j], c, -m));
  return (e[0] + e[1]) + (e[2] + e[3]);
}

// Lazily updated maximum: the pair's terms are summed against the lanes' current maxima
// and accepted while a unit's sum stays below 2^64, i.e. while no logit exceeds m by more
// than about 60 (log2 domain); s then holds sum exp2(x*c - m) for an m that is a logit
// already seen, which is all the normaliser needs.  A larger sum (the first unit of a row,
// whose m is still the empty value kNoMax, or a new extreme) is discarded and the unit is
// redone by the exact online update, which raises m.  This drops the per-logit max and the
// rescaling from the common case.
constexpr float kLazyLimit = 18446744073709551616.0f;  // 2^64

// One sub-tile of pass 1, software-pipelined over the NP row-block pairs: step p issues the
// MFMAs of pair p (query fragments qa, qb, fetched during the previous step) while the
// vector ALU turns the pending pair (pair p-1, or the previous sub-tile's last pair when
// p = 0) into row statistics and the LDS delivers the query fragments of the next pair.
template <int D, int NP>
__device__ inline void stats_steps(const char* qs, const Frag (&kf)[Cfg<D>::kSteps], Frag (&qa)[Cfg<D>::kSteps],
                                   Frag (&qb)[Cfg<D>::kSteps], f32x16& p0, f32x16& p1, float (&sm)[2 * NP],
                                   float (&ss)[2 * NP], float c) {
  using C = Cfg<D>;
  constexpr int NM = 2 * C::kSteps;  // MFMAs per step
#pragma unroll
  for (int p = 0; p < NP; ++p) {
    f32x16 n0, n1;
    mfma_pair<C::kSteps, false>(qa, qb, kf, n0, n1);
    const int pn = p + 1 < NP ? p + 1 : 0;
    read_qfrag<D>(qs, 2 * pn, qa);
    read_qfrag<D>(qs, 2 * pn + 1, qb);
    const int rb = p == 0 ? 2 * NP - 2 : 2 * p - 2;
    const float t0 = unit_sum(p0, c, sm[rb]), t1 = unit_sum(p1, c, sm[rb + 1]);
    const bool big0 = !(t0 < kLazyLimit), big1 = !(t1 < kLazyLimit);
    ss[rb] += big0 ? 0.f : t0;
    ss[rb + 1] += big1 ? 0.f : t1;
    pin(ss[rb], ss[rb + 1], t0, t1);
    // 2 x (16 fma + 15 add) + compares, selects and adds; 32 exp2
    step_schedule<0, 0, 0, NM, NM, (68 + NM - 1) / NM, 32 / NM>();
    if (__builtin_amdgcn_ballot_w64(big0 || big1)) {  // rare: exact update of those units
      if (big0) stats_update(p0, c, sm[rb], ss[rb]);
      if (big1) stats_update(p1, c, sm[rb + 1], ss[rb + 1]);
    }
    p0 = n0;
    p1 = n1;
  }
}

// The ragged last sub-tile of a chunk: tokens at or past `nvalid` get logit -inf.
template <int D, int NP>
__device__ inline void stats_tail(const char* qs, const Frag (&kf)[Cfg<D>::kSteps], int nvalid, float (&sm)[2 * NP],
                                  float (&ss)[2 * NP], float c) {
  using C = Cfg<D>;
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int p = 0; p < NP; ++p) {
    Frag q0[C::kSteps], q1[C::kSteps];
    read_qfrag<D>(qs, 2 * p, q0);
    read_qfrag<D>(qs, 2 * p + 1, q1);
    f32x16 a0, a1;
    mfma_pair<C::kSteps, false>(q0, q1, kf, a0, a1);
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int tok = (i >> 2) * 8 + (lane >> 5) * 4 + (i & 3);
      a0[i] = tok < nvalid ? a0[i] : -INFINITY;
      a1[i] = tok < nvalid ? a1[i] : -INFINITY;
    }
    stats_update(a0, c, sm[2 * p], ss[2 * p]);
    stats_update(a1, c, sm[2 * p + 1], ss[2 * p + 1]);
  }
}

template <int D, int NP>
__global__ __launch_bounds__(kGuideThreads, 1) void k_guide_stats(GuideArgs a) {
  Work w;
  if (!decode(a, w)) return;
  using C = Cfg<D>;
  constexpr int NB = 2 * NP;  // 32-row blocks staged (rows past the group repeat its last row)
  __shared__ __attribute__((aligned(1024))) char qs[NB * 32 * C::kStride];
  __shared__ __attribute__((aligned(1024))) char kst[kGuideWaves * C::kStageBytes];
  const int lane = threadIdx.x & 63;
  const int wave = uniform(threadIdx.x >> 6);
  char* kbuf = kst + wave * C::kStageBytes;
  const char* kchunk = (const char*)(a.k + ((int64_t)w.seg * a.n_tot + w.n0 + w.c0) * D);
  const int ntok = (int)(w.c1 - w.c0);
  const int nfull = ntok / 32;
  int st = wave;
  if (st < nfull) dma_subtile<D>(kchunk, 32 * st, ntok, kbuf);
  stage_q<D>(a, w, qs, NB * 32);
  __syncthreads();

  float sm[NB], ss[NB];
#pragma unroll
  for (int i = 0; i < NB; ++i) {
    sm[i] = kNoMax;
    ss[i] = 0.f;
  }
  // full sub-tiles st = wave, wave + 8, ...
  Frag kf[C::kSteps], qa[C::kSteps], qb[C::kSteps];
  f32x16 p0, p1;
#pragma unroll
  for (int i = 0; i < 16; ++i) p0[i] = p1[i] = -INFINITY;  // empty pipeline slot
  read_qfrag<D>(qs, 0, qa);
  read_qfrag<D>(qs, 1, qb);
  __shared__ int progress[kGuideWaves];
  if (threadIdx.x < kGuideWaves) progress[threadIdx.x] = 0;
  __syncthreads();
  for (int done = 0; st < nfull; st += kGuideWaves) {
    wait_copies();
    read_kfrag<D>(kbuf, kf);
    wait_lds_reads();
    if (st + kGuideWaves < nfull) dma_subtile<D>(kchunk, 32 * (st + kGuideWaves), ntok, kbuf);
    stats_steps<D, NP>(qs, kf, qa, qb, p0, p1, sm, ss, a.c);
    balance_issue(progress, wave, ++done);
  }
  __builtin_amdgcn_s_setprio(0);
  stats_update(p0, a.c, sm[NB - 2], ss[NB - 2]);
  stats_update(p1, a.c, sm[NB - 1], ss[NB - 1]);
  if (ntok > 32 * nfull && wave == nfull % kGuideWaves) {
    dma_subtile<D>(kchunk, 32 * nfull, ntok, kbuf);
    wait_copies();
    read_kfrag<D>(kbuf, kf);
    stats_tail<D, NP>(qs, kf, ntok - 32 * nfull, sm, ss, a.c);
  }

  // merge the half-waves (same rows, other tokens), then the waves, through LDS (the query
  // buffer is free now)
  __syncthreads();
  float2* xch = (float2*)qs;  // [wave][NB * 32]
  static_assert(kGuideWaves * NB * 32 * sizeof(float2) <= sizeof(qs), "exchange buffer");
#pragma unroll
  for (int rb = 0; rb < NB; ++rb) {
    merge_stats(sm[rb], ss[rb], __shfl_xor(sm[rb], 32), __shfl_xor(ss[rb], 32));
    if (lane < 32) xch[wave * NB * 32 + rb * 32 + lane] = make_float2(sm[rb], ss[rb]);
  }
  __syncthreads();
  const int64_t growtot = (int64_t)a.L * a.Hq * a.g_tot;
  for (int t = threadIdx.x; t < w.nrows; t += kGuideThreads) {
    float mm = xch[t].x, s2 = xch[t].y;
#pragma unroll
    for (int q = 1; q < kGuideWaves; ++q) merge_stats(mm, s2, xch[q * NB * 32 + t].x, xch[q * NB * 32 + t].y);
    a.stats[(int64_t)w.chunk * growtot + grow_of(a, w, w.row0 + t)] = make_float2(mm, s2);
  }
}

// ---------------------------------------------------------------------------- guide keys
// With the guide's own keys (the paper-literal slice of the causal attention over context +
// appended guide, Sec. 3.2), guide row j's normaliser also takes the logits of guide keys
// 0..j.  One workgroup takes up to 256 guide rows of a (sequence, layer, KV head); the
// guide keys of that head are staged in LDS kGuideKeyTile at a time, and every lane (one
// row each, its query in registers) walks the keys in the same order, so all lanes read the
// same key row at once (an LDS broadcast).  The row's (max, sum) over its keys t <= j goes
// to the extra statistics slot nchunk_max, which the merge below treats as one more chunk.
constexpr int kGuideKeyTile = 64;

template <int D>
__global__ __launch_bounds__(256) void k_guide_key_stats(GuideArgs a) {
  const int b = blockIdx.z, seg = blockIdx.y;
  const int64_t g0 = a.bt.g_off[b];
  const int gb = (int)(a.bt.g_off[b + 1] - g0);
  const int rows = a.R * gb;
  const int rho = blockIdx.x * 256 + threadIdx.x;  // guide row of the segment: (r, j)
  if ((int)blockIdx.x * 256 >= rows) return;       // the whole block has no rows
  const int64_t l = seg / a.Hkv, h = seg % a.Hkv;
  const bool live = rho < rows;
  const int r = live ? rho / gb : 0, j = live ? rho % gb : -1;
  const int64_t grow = ((l * a.Hq + h * a.R + r) * a.g_tot) + g0 + (live ? j : 0);
  __shared__ uint4 keys[kGuideKeyTile][D / 8];
  uint4 qv[D / 8];  // the row's query, bf16 pairs
  {
    const uint4* qrow = (const uint4*)(a.q + grow * D);
#pragma unroll
    for (int p = 0; p < D / 8; ++p) qv[p] = qrow[p];
  }
  // the block's rows need keys 0 .. max j; its last row has the largest j unless it wraps
  const int last = min(rows, (int)(blockIdx.x + 1) * 256) - 1;
  const int nkeys = ((int)blockIdx.x * 256) / gb == last / gb ? last % gb + 1 : gb;
  const uint4* kg = (const uint4*)(a.kg + ((l * a.Hkv + h) * a.g_tot + g0) * D);
  float m = kNoMax, s = 0.f;
  for (int t0 = 0; t0 < nkeys; t0 += kGuideKeyTile) {
    const int nt = min(kGuideKeyTile, nkeys - t0);
    __syncthreads();
    for (int i = threadIdx.x; i < nt * (D / 8); i += 256) keys[i / (D / 8)][i % (D / 8)] = kg[(int64_t)(t0 + i / (D / 8)) * (D / 8) + i % (D / 8)];
    __syncthreads();
    const int tend = min(nt, j - t0 + 1);  // keys t0 .. j of this tile (none for idle lanes)
    for (int t = 0; t < tend; ++t) {
      // fp32 dot product of bf16 pairs (v_dot2_f32_bf16), four independent partial sums
      float part[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int p = 0; p < D / 8; ++p) {
        const uint4 u = keys[t][p];
        const uint32_t kw[4] = {u.x, u.y, u.z, u.w};
        const uint32_t qw[4] = {qv[p].x, qv[p].y, qv[p].z, qv[p].w};
#pragma unroll
        for (int e = 0; e < 4; ++e)
          part[e] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, qw[e]),
                                                    __builtin_bit_cast(bf16x2, kw[e]), part[e], false);
      }
      merge_stats(m, s, ((part[0] + part[1]) + (part[2] + part[3])) * a.c, 1.0f);
    }
  }
  if (live) a.stats[(int64_t)a.nchunk_max * ((int64_t)a.L * a.Hq * a.g_tot) + grow] = make_float2(m, s);
}

// ---------------------------------------------------------------------------- lse merge
// One thread per guide row: merge the row's per-chunk (max, sum) pairs (and, with guide
// keys, the guide-key slot) into lse2.
template <int D>
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
  const int nch = (int)((nb + a.chunk - 1) / a.chunk);
  float m = kNoMax, s = 0.f;
  for (int c = 0; c < nch; ++c) {
    const float2 v = a.stats[(int64_t)c * growtot + grow];
    merge_stats(m, s, v.x, v.y);
  }
  if (a.kg != nullptr) {
    const float2 v = a.stats[(int64_t)a.nchunk_max * growtot + grow];
    merge_stats(m, s, v.x, v.y);
  }
  a.lse2[grow] = m + log2f(s);
}

// ---------------------------------------------------------------------------- pass 2
// The MFMA chains of pass 2 start from -lse2/c instead of zero, so a unit's accumulator
// holds x - lse2/c and the normalised weight is exp2(acc * c).  acc[i] belongs to row
// (i/4)*8 + (lane/32)*4 + i%4 and token lane%32; the lane sums its 16 rows.
__device__ inline float attn_sum(const f32x16& acc, float c) {
  float e[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) e[j] = __builtin_amdgcn_exp2f(acc[j] * c);
#pragma unroll
  for (int i = 4; i < 16; i += 4)
#pragma unroll
    for (int j = 0; j < 4; ++j) e[j] += __builtin_amdgcn_exp2f(acc[i + j] * c);
  return (e[0] + e[1]) + (e[2] + e[3]);
}

// Accumulator start values of row block rb: -lse2/c of the lane's 16 rows.
__device__ inline void read_lz(const float* lz_s, int rb, f32x16& acc) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int g = 0; g < 4; ++g) {
    const float4 v = *(const float4*)(lz_s + rb * 32 + g * 8 + (lane >> 5) * 4);
    acc[4 * g + 0] = v.x;
    acc[4 * g + 1] = v.y;
    acc[4 * g + 2] = v.z;
    acc[4 * g + 3] = v.w;
  }
}

// The sum over rows is finished for a sub-tile once its last pair has been summed: add the
// other half-wave's rows and store the token's value.
__device__ inline void attn_flush(float part, float* raw_out, int tok0, int ntok) {
  const int lane = threadIdx.x & 63;
  const float v = part + __shfl_xor(part, 32);
  const int tok = tok0 + lane;
  if (tok0 >= 0 && lane < 32 && tok < ntok) raw_out[tok] = v;
}

// One sub-tile of pass 2, pipelined like pass 1.  `part` carries the partial row sum of the
// sub-tile whose pairs are in the vector stage; it is flushed (for the sub-tile starting at
// token `prev_tok0`) when that sub-tile's last pair has been added.
template <int D, int NP>
__device__ inline void attn_steps(const char* qs, const float* lz_s, const Frag (&kf)[Cfg<D>::kSteps],
                                  Frag (&qa)[Cfg<D>::kSteps], Frag (&qb)[Cfg<D>::kSteps], f32x16& p0, f32x16& p1,
                                  float& part, int prev_tok0, float* raw_out, int ntok, float c) {
  using C = Cfg<D>;
#pragma unroll
  for (int p = 0; p < NP; ++p) {
    f32x16 n0, n1;
    read_lz(lz_s, 2 * p, n0);
    read_lz(lz_s, 2 * p + 1, n1);
    mfma_pair<C::kSteps, true, true>(qa, qb, kf, n0, n1);
    const int pn = p + 1 < NP ? p + 1 : 0;
    read_qfrag<D>(qs, 2 * pn, qa);
    read_qfrag<D>(qs, 2 * pn + 1, qb);
    part += attn_sum(p0, c) + attn_sum(p1, c);
    pin(part, part, part, part);
    step_schedule<8, 8, 4, 2 * C::kSteps, 2 * C::kSteps, 56 / (2 * C::kSteps), 28 / (2 * C::kSteps)>();
    if (p == 0) {
      attn_flush(part, raw_out, prev_tok0, ntok);
      part = 0.f;
    }
    p0 = n0;
    p1 = n1;
  }
}

template <int D, int NP>
__global__ __launch_bounds__(kGuideThreads, 1) void k_guide_attn(GuideArgs a) {
  Work w;
  if (!decode(a, w)) return;
  using C = Cfg<D>;
  constexpr int NB = 2 * NP;
  __shared__ __attribute__((aligned(1024))) char qs[NB * 32 * C::kStride];
  __shared__ __attribute__((aligned(1024))) char kst[kGuideWaves * C::kStageBytes];
  __shared__ __attribute__((aligned(16))) float lz_s[NB * 32];
  const int wave = uniform(threadIdx.x >> 6);
  char* kbuf = kst + wave * C::kStageBytes;
  const int64_t tok0 = (int64_t)w.seg * a.n_tot + w.n0 + w.c0;  // first token row of the chunk
  const char* kchunk = (const char*)(a.k + tok0 * D);
  const int ntok = (int)(w.c1 - w.c0);
  // every sub-tile, the ragged last one included: its repeated tokens are never stored
  const int nsub = (ntok + 31) / 32;
  int st = wave;
  if (st < nsub) dma_subtile<D>(kchunk, 32 * st, ntok, kbuf);
  stage_q<D>(a, w, qs, NB * 32);
  for (int t = threadIdx.x; t < NB * 32; t += kGuideThreads)  // padding rows: exp2(-inf) = 0
    lz_s[t] = t < w.nrows ? -a.lse2[grow_of(a, w, w.row0 + t)] / a.c : -INFINITY;
  __syncthreads();

  float* raw_out = a.raw + ((int64_t)w.rg * a.L * a.Hkv + w.seg) * a.n_tot + w.n0 + w.c0;
  Frag kf[C::kSteps], qa[C::kSteps], qb[C::kSteps];
  f32x16 p0, p1;
#pragma unroll
  for (int i = 0; i < 16; ++i) p0[i] = p1[i] = -INFINITY;  // empty pipeline slot: sums to 0
  float part = 0.f;
  int prev = -1;  // first chunk token of the sub-tile in the vector stage (none yet)
  read_qfrag<D>(qs, 0, qa);
  read_qfrag<D>(qs, 1, qb);
  __shared__ int progress[kGuideWaves];
  if (threadIdx.x < kGuideWaves) progress[threadIdx.x] = 0;
  __syncthreads();
  for (int done = 0; st < nsub; st += kGuideWaves) {
    wait_copies();
    read_kfrag<D>(kbuf, kf);
    wait_lds_reads();
    if (st + kGuideWaves < nsub) dma_subtile<D>(kchunk, 32 * (st + kGuideWaves), ntok, kbuf);
    attn_steps<D, NP>(qs, lz_s, kf, qa, qb, p0, p1, part, prev, raw_out, ntok, a.c);
    prev = 32 * st;
    balance_issue(progress, wave, ++done);
  }
  __builtin_amdgcn_s_setprio(0);
  part += attn_sum(p0, a.c) + attn_sum(p1, a.c);
  attn_flush(part, raw_out, prev, ntok);
}

// ---------------------------------------------------------------------------- pooling
// s_key = (1/(R K)) * sum over the window of the raw sums of all row groups (zero outside the
// sequence).  A block stages kPoolTile + 2*half raw values (summed over row groups) in LDS
// with coalesced loads, then each thread sums its windows from LDS; windows wider than
// kPoolMaxHalf use the direct loop.
constexpr int kPoolTile = 4096;
constexpr int kPoolMaxHalf = 512;

__device__ inline float raw_at(const GuideArgs& a, const float* raw, int nrg, int64_t j) {
  const int64_t lh = (int64_t)a.L * a.Hkv;
  float v = 0.f;
  for (int rg = 0; rg < nrg; ++rg) v += raw[rg * lh * a.n_tot + j];
  return v;
}

__global__ __launch_bounds__(256) void k_guide_pool(GuideArgs a) {
  __shared__ float buf[kPoolTile + 2 * kPoolMaxHalf];
  const int seg = blockIdx.y, b = blockIdx.z;
  const int64_t n0 = a.bt.ctx_off[b];
  const int64_t nb = a.bt.ctx_off[b + 1] - n0;
  const int64_t i0 = (int64_t)blockIdx.x * kPoolTile;
  if (i0 >= nb) return;
  const int gb = (int)(a.bt.g_off[b + 1] - a.bt.g_off[b]);
  const int nrg = (a.R * gb + kRowsPerGroup - 1) / kRowsPerGroup;
  const float* raw = a.raw + (int64_t)seg * a.n_tot + n0;
  float* out = a.s_key + (int64_t)seg * a.n_tot + n0;
  const int half = a.pool_half;
  if (half > kPoolMaxHalf) {  // wide windows: direct sums
    for (int u = 0; u < kPoolTile / 256; ++u) {
      const int64_t i = i0 + threadIdx.x + 256 * u;
      if (i >= nb) break;
      float acc = 0.f;
      for (int t = -half; t <= half; ++t)
        if (i + t >= 0 && i + t < nb) acc += raw_at(a, raw, nrg, i + t);
      out[i] = acc * a.pool_inv;
    }
    return;
  }
  const int nstage = kPoolTile + 2 * half;
  for (int t0 = 0; t0 < nstage; t0 += 256 * 8) {  // eight loads in flight per thread
    float v[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int t = t0 + 256 * e + threadIdx.x;
      const int64_t j = i0 - half + t;
      v[e] = (t < nstage && j >= 0 && j < nb) ? raw_at(a, raw, nrg, j) : 0.f;
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int t = t0 + 256 * e + threadIdx.x;
      if (t < nstage) buf[t] = v[e];
    }
  }
  __syncthreads();
#pragma unroll
  for (int u = 0; u < kPoolTile / 256; ++u) {
    const int l = threadIdx.x + 256 * u;
    if (i0 + l >= nb) break;
    float acc = 0.f;
    for (int t = 0; t <= 2 * half; ++t) acc += buf[l + t];
    out[i0 + l] = acc * a.pool_inv;
  }
}

// Row normalisers supplied by the caller (natural log) -> the log2 domain of pass 2.
__global__ __launch_bounds__(256) void k_lse_import(const float* lse, float* lse2, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i < n) lse2[i] = (float)((double)lse[i] * 1.4426950408889634);
}

template <int D, int NP>
hipError_t launch_pass(const GuideArgs& a, bool attn, hipStream_t stream) {
  const unsigned nwg = (unsigned)a.wg_off[a.bt.batch];
  if (nwg == 0) return hipSuccess;
  if (attn) {
    hipLaunchKernelGGL((k_guide_attn<D, NP>), dim3(nwg), dim3(kGuideThreads), 0, stream, a);
  } else if constexpr (NP != 3) {  // pass 1 has no 3-pair class (see launch_d)
    hipLaunchKernelGGL((k_guide_stats<D, NP>), dim3(nwg), dim3(kGuideThreads), 0, stream, a);
  }
  return hipGetLastError();
}

// One launch per class of sequences that need the same number NP of staged row-block pairs
// (NP = ceil(min(R G_b, 256) / 64)), so short guides do not pay for 256 rows; each class's
// arguments give the other sequences empty workgroup ranges.
template <int D>
hipError_t launch_d(const GuideArgs& a, hipStream_t stream, hipEvent_t* ev, GuideBetween between, void* ctx) {
  static_assert(kChunkSmall % (32 * kGuideWaves) == 0, "every wave owns whole sub-tiles of a chunk");
  int64_t max_nb = 0, max_gb = 0;
  // per pass and class NP (1..4 staged row-block pairs) the launch arguments, with the other
  // classes' sequences given empty workgroup ranges.  Pass 1 has no NP = 3 class: its
  // three-pair kernel needs more VGPRs than the four-pair one (248 against 228) and would
  // leave no room for the quantisation tp_evict runs beside pass 1, so 129..192 rows are
  // padded to four pairs there (the padding rows' statistics are never stored).
  GuideArgs cls[2][4];
  int64_t wg[2][4] = {{0, 0, 0, 0}, {0, 0, 0, 0}};
  for (int pass = 0; pass < 2; ++pass)
    for (int c = 0; c < 4; ++c) {
      cls[pass][c] = a;
      cls[pass][c].wg_off[0] = 0;
    }
  for (int b = 0; b < a.bt.batch; ++b) {
    const int64_t nb = a.bt.ctx_off[b + 1] - a.bt.ctx_off[b];
    const int64_t gb = a.bt.g_off[b + 1] - a.bt.g_off[b];
    if (nb > max_nb) max_nb = nb;
    if (gb > max_gb) max_gb = gb;
    const int64_t rows = (int64_t)a.R * gb;
    const int np = (int)(((rows < kRowsPerGroup ? rows : kRowsPerGroup) + 63) / 64);
    const int64_t units = (int64_t)a.L * a.Hkv * ((nb + a.chunk - 1) / a.chunk);
    const int64_t seq_wg = (units + 7) / 8 * 8 * ((rows + kRowsPerGroup - 1) / kRowsPerGroup);
    wg[0][np == 3 ? 3 : np - 1] += seq_wg;
    wg[1][np - 1] += seq_wg;
    for (int pass = 0; pass < 2; ++pass)
      for (int c = 0; c < 4; ++c) cls[pass][c].wg_off[b + 1] = (int32_t)wg[pass][c];
  }
  for (int pass = 0; pass < 2; ++pass) {  // the large classes first: shorter tail
    if (pass == 0 && a.lse_in) {  // normalisers given: no pass 1
      hipError_t e = ev ? hipEventRecord(ev[0], stream) : hipSuccess;
      if (e != hipSuccess) return e;
      const int64_t n = (int64_t)a.L * a.Hq * a.g_tot;
      hipLaunchKernelGGL(k_lse_import, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, stream, a.lse_in, a.lse2, n);
      e = hipGetLastError();
      if (e == hipSuccess && ev) e = hipEventRecord(ev[1], stream);
      if (e == hipSuccess && between) e = between(ctx);
      if (e != hipSuccess) return e;
      continue;
    }
    hipError_t e = launch_pass<D, 4>(cls[pass][3], pass == 1, stream);
    if (e == hipSuccess) e = launch_pass<D, 3>(cls[pass][2], pass == 1, stream);
    if (e == hipSuccess) e = launch_pass<D, 2>(cls[pass][1], pass == 1, stream);
    if (e == hipSuccess) e = launch_pass<D, 1>(cls[pass][0], pass == 1, stream);
    if (e == hipSuccess && ev) e = hipEventRecord(ev[pass == 0 ? 0 : 2], stream);
    if (e != hipSuccess) return e;
    if (pass == 0) {
      if (a.kg != nullptr) {
        const dim3 kgrid((unsigned)((a.R * max_gb + 255) / 256), (unsigned)(a.L * a.Hkv), (unsigned)a.bt.batch);
        hipLaunchKernelGGL(k_guide_key_stats<D>, kgrid, dim3(256), 0, stream, a);
      }
      const dim3 lgrid((unsigned)((a.L * a.Hq * max_gb + 255) / 256), (unsigned)a.bt.batch);
      hipLaunchKernelGGL(k_guide_lse<D>, lgrid, dim3(256), 0, stream, a);
      e = hipGetLastError();
      if (e == hipSuccess && ev) e = hipEventRecord(ev[1], stream);
      if (e == hipSuccess && between) e = between(ctx);
      if (e != hipSuccess) return e;
    }
  }
  if (a.skip_pool) return hipSuccess;  // the split selection pools the raw sums itself
  const dim3 pgrid((unsigned)((max_nb + kPoolTile - 1) / kPoolTile), (unsigned)(a.L * a.Hkv), (unsigned)a.bt.batch);
  hipLaunchKernelGGL(k_guide_pool, pgrid, dim3(256), 0, stream, a);
  hipError_t e = hipGetLastError();
  if (e == hipSuccess && ev && ev[3]) e = hipEventRecord(ev[3], stream);
  return e;
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
  const int64_t chunk = chunk_tokens(ctx_off, batch);
  const int64_t nchunk = (max_nb + chunk - 1) / chunk;
  const int64_t nrg = (R * max_gb + kRowsPerGroup - 1) / kRowsPerGroup;
  auto up = [](size_t x) { return (x + 255) & ~(size_t)255; };
  GuideWorkspace w;
  w.stats_off = 0;  // nchunk slots of per-chunk statistics, plus one for the guide keys
  w.lse_off = up((size_t)(nchunk + 1) * L * Hq * g_tot * sizeof(float2));
  w.raw_off = w.lse_off + up((size_t)L * Hq * g_tot * sizeof(float));
  w.total = w.raw_off + up((size_t)nrg * L * Hkv * n_tot * sizeof(float));
  return w;
}

hipError_t launch_guide_scores(const GuideArgs& a, int head_dim, hipStream_t stream, hipEvent_t* ev,
                               GuideBetween between, void* ctx) {
  if (head_dim == 128) return launch_d<128>(a, stream, ev, between, ctx);
  return launch_d<64>(a, stream, ev, between, ctx);
}

}  // namespace tp
