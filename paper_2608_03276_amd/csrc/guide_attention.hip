// The prefill's attention for the appended guide rows (Sec. 3.2: the task guide is appended
// after the context and attends causally, so guide row j sees the N context keys and guide
// keys 0..j).  Its outputs are the rows' attention output O (what the prefill passes on) and
// each row's log-sum-exp over the keys it sees, which is the normaliser of the attention map
// Sec. 3.2 slices A from: tp_guide_scores_lse / tp_evict(guide_lse) take it, so the eviction
// needs one more sweep over K on top of this one instead of two.
//
// Flash-attention style, split over the context in chunks: one workgroup per (sequence,
// layer, KV head, chunk, group of <= 256 guide rows), eight waves (two per SIMD, so that one
// wave's exponentials overlap the other's MFMAs), wave w owning rows 32w .. 32w + 31.  The
// chunk's 32-token sub-tiles of K and V stream through a ring of LDS slots filled by direct
// global->LDS copies issued several sub-tiles ahead (one barrier per pair of sub-tiles), and every
// wave reads the whole sub-tile.  Per sub-tile, on v_mfma_f32_32x32x16_bf16:
//   S^T = K Q^T (tokens on M, rows on N): a lane holds one row and 16 of the 32 tokens (its
//       partner lane 32 apart holds the other 16), so the row's running maximum and sum stay
//       in the lane pair;
//   P  = exp2(S c - m) against the pair's current maximum m, which is raised (with O and the
//       sum rescaled) only when a lane's 16 terms would sum past 2^32; m is always a logit
//       already seen, which is all the normaliser needs;
//   O^T += V^T P^T (d on M, rows on N): the B operand is the lane's own 16 probabilities in
//       bf16, the contraction index mapped to exactly the tokens the lane holds; the A
//       operand comes from the token-major V sub-tile through transposing LDS reads.
// Each workgroup writes its rows' partial (max, sum) and unnormalised O; the guide's own keys
// are one more chunk, with the causal mask.  A merge kernel combines the chunks.
// An instance per code format also performs step 2 (Eq. 2, Sec. 3.3) on the V sub-tiles it
// stages (tp_guide_attention_quantize), so the quantised cache and the value scores come from
// this one read of V.
#include "quant_row.h"
#include "tile_common.h"
#include "tp_internal.h"

#include <type_traits>

namespace tp {
namespace {

constexpr int kAttnThreads = 512;  // 8 waves, two per SIMD, 32 rows each
constexpr int kAttnWaves = kAttnThreads / 64;
constexpr float kAttnLazyLimit = 4294967296.0f;  // 2^32: a lane's 16 terms against a stale maximum
constexpr int kAttnNoQuant = -1;  // the instance that leaves V's step 2 to its own kernel

typedef short v4i16 __attribute__((ext_vector_type(4)));

template <int D>
struct AttnCfg {
  static constexpr int kTileBytes = 32 * D * 2;                // one 32-token K (or V) sub-tile
  static constexpr int kSlotBytes = 2 * kTileBytes;            // a ring slot: K, then V
  static constexpr int kCopies = kSlotBytes / 1024 / kAttnWaves;  // 1 KB copies per wave per sub-tile
  static constexpr int kRing = D == 128 ? 9 : 16;             // slots: 144 KB / 128 KB of LDS
  static_assert(kRing * kSlotBytes <= 160 * 1024, "LDS of one CU");
  static_assert(kRing >= 7 && kRing - 6 <= 12 && (kRing - 6) * kCopies <= 63,
                "the pair protocol's lookahead, wait_copies_but cases and the vmcnt range");
};

// V sub-tiles are staged like K (16-byte piece p of token tl in slot p ^ swzv(tl)) with their
// own permutation, chosen for the transposing reads: a half-wave reads 4 consecutive tokens,
// 4 pieces each (16 lanes: 2 pieces each), and swzv gives the 4 tokens disjoint bank sets in
// both groupings (a 256-byte row covers every bank of the 64).
template <int D>
__device__ inline int swzv(int tl) {
  if (D == 128) return (0xCA60 >> (4 * (tl & 3))) & 15;  // 0, 6, 10, 12
  return 2 * (tl & 3);
}

// One global->LDS copy of 16 bytes per lane: lane i's bytes from src land at LDS byte
// lds + 16 i.  Inline assembly rather than the builtin, because the compiler cannot tell the
// ring's slots apart and would drain every copy in flight before each LDS read of the ring;
// completion is tracked by the explicit vmcnt waits below instead.  One wait state separates
// the M0 write from the copy that reads it.
__device__ inline void copy16(const void* src, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(src), "s"(lds) : "memory", "m0");
}

// Copy j (0 .. 2 kTileBytes / 1 KB - 1) of a sub-tile, 1 KB: K's first, then V's, kCopies to a
// wave.  Returns whether it is V's and gives the lane's token in the sub-tile and the byte
// offset of its swizzled 16-byte piece within that token's row.
template <int D>
__device__ inline bool copy_lane(int j, int& tl, int& piece) {
  using C = Cfg<D>;
  constexpr int kKB = 32 / C::kTokPerKB;  // 1 KB copies per 32-token tile
  const int lane = threadIdx.x & 63;
  const bool isv = j >= kKB;
  const int jj = isv ? j - kKB : j;
  tl = jj * C::kTokPerKB + lane / C::kPieces;
  piece = ((lane % C::kPieces) ^ (isv ? swzv<D>(tl) : swz<D>(tl))) * 16;
  return isv;
}

// Issue this wave's share of the copies of sub-tile rows [t0, t0 + 32) of K and V into the
// slot at LDS byte `slot` (rows past ntok repeat the last row: finite data the masks drop).
template <int D>
__device__ inline void copy_subtile(const char* kbase, const char* vbase, int t0, int ntok, uint32_t slot, int wave) {
#pragma unroll
  for (int i = 0; i < AttnCfg<D>::kCopies; ++i) {
    const int j = wave * AttnCfg<D>::kCopies + i;  // wave-uniform
    int tl, piece;
    const bool isv = copy_lane<D>(j, tl, piece);
    const int tok = min(t0 + tl, ntok - 1);
    copy16((isv ? vbase : kbase) + (uint32_t)tok * Cfg<D>::kRowBytes + piece, slot + (uint32_t)j * 1024u);
  }
}

// The scalar-address form of copy16: the lane's bytes come from sbase + voff, sbase
// wave-uniform.
__device__ inline void copy16s(uint32_t voff, const void* sbase, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(voff), "s"(sbase), "s"(lds)
               : "memory", "m0");
}

// The lane's offsets for copy_whole, fixed for the kernel.
template <int D>
__device__ inline void copy_offsets(uint32_t (&voff)[AttnCfg<D>::kCopies], int wave) {
#pragma unroll
  for (int i = 0; i < AttnCfg<D>::kCopies; ++i) {
    int tl, piece;
    copy_lane<D>(wave * AttnCfg<D>::kCopies + i, tl, piece);
    voff[i] = (uint32_t)(tl * Cfg<D>::kRowBytes + piece);
  }
}

// copy_subtile for a sub-tile whose 32 rows all exist: no clamp, and the row address is a
// wave-uniform base plus the lane's fixed offset, so issuing a copy takes no vector work.
template <int D>
__device__ inline void copy_whole(const char* kbase, const char* vbase, int t0, const uint32_t (&voff)[AttnCfg<D>::kCopies],
                                  uint32_t slot, int wave) {
  constexpr int kKB = 32 / Cfg<D>::kTokPerKB;
#pragma unroll
  for (int i = 0; i < AttnCfg<D>::kCopies; ++i) {
    const int j = wave * AttnCfg<D>::kCopies + i;  // wave-uniform
    const char* base = (j >= kKB ? vbase : kbase) + (int64_t)t0 * Cfg<D>::kRowBytes;
    copy16s(voff[i], base, slot + (uint32_t)j * 1024u);
  }
}

// Wait until at most k sub-tiles' copies of this wave are still in flight (copies complete in
// issue order).  k is wave-uniform and at most kRing - 6 (12).
template <int PER>
__device__ inline void wait_copies_but(int k) {
  switch (k) {
    case 0: asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); break;
    case 1: asm volatile("s_waitcnt vmcnt(%0)" ::"n"(PER) : "memory"); break;
    case 2: asm volatile("s_waitcnt vmcnt(%0)" ::"n"(2 * PER) : "memory"); break;
    case 3: asm volatile("s_waitcnt vmcnt(%0)" ::"n"(3 * PER) : "memory"); break;
    case 4: asm volatile("s_waitcnt vmcnt(%0)" ::"n"(4 * PER) : "memory"); break;
    case 5: asm volatile("s_waitcnt vmcnt(%0)" ::"n"(5 * PER) : "memory"); break;
    case 6: asm volatile("s_waitcnt vmcnt(%0)" ::"n"(6 * PER) : "memory"); break;
    case 7: asm volatile("s_waitcnt vmcnt(%0)" ::"n"(7 * PER) : "memory"); break;
    case 8: asm volatile("s_waitcnt vmcnt(%0)" ::"n"(8 * PER) : "memory"); break;
    case 9: asm volatile("s_waitcnt vmcnt(%0)" ::"n"(9 * PER) : "memory"); break;
    case 10: asm volatile("s_waitcnt vmcnt(%0)" ::"n"(10 * PER) : "memory"); break;
    case 11: asm volatile("s_waitcnt vmcnt(%0)" ::"n"(11 * PER) : "memory"); break;
    default: asm volatile("s_waitcnt vmcnt(%0)" ::"n"(12 * PER) : "memory"); break;
  }
}

// Every wave's copies up to the waited point have landed and every wave's LDS reads before
// this point are complete: the barrier without the full memory fence of __syncthreads, which
// would also drain the copies still in flight.  The LDS wait is the builtin (vmcnt and expcnt
// left at their maxima, lgkmcnt 0), which the compiler sees: it then knows the fragments read
// before the barrier have arrived and adds no wait of its own for them after it.
__device__ inline void ring_barrier() {
  __builtin_amdgcn_s_waitcnt(0xC07F);
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// A operand of O^T += V^T P^T for d-block db and k-step s2, from the token-major V sub-tile:
// lane l needs V^T[d][k] for d = 32 db + l%32 and k = 8 (l/32) + e, e = 0..7, standing for
// token 16 s2 + 8 (e/4) + 4 (l/32) + e%4 (the tokens whose probabilities the lane holds).
// A transposing read hands lane i of each 16-lane group element e from the 8 bytes that lane
// 4e + i/4 of the group addressed, element i%4; so source lane s addresses the 4 d-values
// 32 db + 16 ((l/16)%2) + 4 (s%4) .. +3 of token 16 s2 + 8 call + 4 (l/32) + s/4.
template <int D>
__device__ inline Frag read_vfrag(const char* vtile, int db, int s2) {
  using C = Cfg<D>;
  const int lane = threadIdx.x & 63;
  const int h = lane >> 5, g = (lane >> 4) & 1, s = lane & 15;
  const int col = 32 * db + 16 * g + 4 * (s & 3);  // first d-value addressed
  union {
    v4i16 v;
    uint2 u;
  } r[2];
#pragma unroll
  for (int call = 0; call < 2; ++call) {
    const int tl = 16 * s2 + 8 * call + 4 * h + (s >> 2);
    const char* addr = vtile + tl * C::kRowBytes + (((col >> 3) ^ swzv<D>(tl)) << 4) + ((col & 7) << 1);
    r[call].v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) v4i16*)addr);
  }
  Frag f;
  f.u = make_uint4(r[0].u.x, r[0].u.y, r[1].u.x, r[1].u.y);
  return f;
}

__device__ inline float terms(const f32x16& s, float c, float m, float (&p)[16]) {
#pragma unroll
  for (int i = 0; i < 16; ++i) p[i] = __builtin_amdgcn_exp2f(fmaf(s[i], c, -m));
  float e[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) e[j] = (p[j] + p[4 + j]) + (p[8 + j] + p[12 + j]);
  return (e[0] + e[1]) + (e[2] + e[3]);
}

// The rare exact update of the lane pair's maximum (a row's first sub-tile, or a logit more
// than about 32 above its maximum in log2 units): m raised to the sub-tile's maximum, the sum
// and the output rescaled, the terms recomputed.  Both lanes of a row take it together.
template <int NDB>
__device__ inline void raise_max(const f32x16& s, float c, float& m, float& l, f32x16 (&ot)[NDB], float (&p)[16],
                                 float& ps) {
  float mx = max16(s) * c;  // c > 0
  mx = fmaxf(mx, __shfl_xor(mx, 32));
  const float mn = fmaxf(m, mx);
  const float al = __builtin_amdgcn_exp2f(m - mn);
  l *= al;
#pragma unroll
  for (int db = 0; db < NDB; ++db)
#pragma unroll
    for (int i = 0; i < 16; ++i) ot[db][i] *= al;
  m = mn;
  ps = terms(s, c, m, p);
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

// QK: kAttnNoQuant, or the QKind of the codes when the kernel also performs step 2 (Eq. 2)
// on the V sub-tiles it stages: the workgroup of a context chunk's first row group quantises
// each token row of the chunk once, from LDS (the arithmetic of quant_row.h, bit-identical to
// the quantisation kernel's).
template <int D, int QK>
__global__ __launch_bounds__(kAttnThreads, 1) void k_guide_fwd(AttnArgs a) {
  AttnUnit u;
  if (!attn_unit(a, u)) return;
  using C = Cfg<D>;
  using AC = AttnCfg<D>;
  constexpr int KS = C::kSteps;
  constexpr int NDB = D / 32;  // 32-wide d-blocks of O
  constexpr int RING = AC::kRing;
  constexpr bool QUANT = QK != kAttnNoQuant;
  constexpr int QKC = QUANT ? QK : 0;
  constexpr int QNP = D / 64;     // the quantisation: 16-byte pieces of a V row per lane,
  constexpr int QLPT = 8;         // lanes per row (8 rows per wave)
  // the ring, then (QUANT) the quantisation tables
  __shared__ __attribute__((aligned(1024))) char ring[RING * AC::kSlotBytes + (QUANT ? sizeof(QuantTables) : 0)];
  QuantTables& tab = *(QuantTables*)(ring + RING * AC::kSlotBytes);
  const int lane = threadIdx.x & 63;
  const int wave = uniform(threadIdx.x >> 6);
  const bool active = 32 * wave < u.nrows;
  // this lane's guide row (rows past the group's end repeat its last row and are never
  // written)
  const int rho_raw = u.row0 + 32 * wave + (lane & 31);
  const bool row_ok = rho_raw < u.row0 + u.nrows;
  const int rho = row_ok ? rho_raw : u.row0 + u.nrows - 1;
  const int r = rho / u.gb, jrow = rho % u.gb;
  const int64_t grow = ((int64_t)u.l * a.Hq + (int64_t)u.h * a.R + r) * a.g_tot + u.g0 + jrow;
  // the K fragments' contraction order: half-wave h holds d-columns h D/2 + 8 s .. + 8
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
  const char* kb = (const char*)ksrc;
  const char* vb = (const char*)vsrc;
  const int ntok = u.ntok;
  const int nsub = (ntok + 31) / 32;

  float m = kNoMax, lsum = 0.f;
  f32x16 ot[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db) ot[db] = (f32x16){};

  // The query loads complete here, in a wait the compiler knows of: it then has no load of
  // its own in flight inside the loop and inserts no waits there (which, blind to the ring's
  // copies, would drain them).
  __builtin_amdgcn_s_waitcnt(0);
  const uint32_t ring_lds = (uint32_t)__builtin_amdgcn_readfirstlane(
      (int)(uintptr_t)(__attribute__((address_space(3))) char*)ring);
  // Software pipeline: iteration t issues, interleaved with the exponentials of sub-tile t,
  // the MFMAs of S for sub-tile t + 1 and of O += V P for sub-tile t - 1 (neither depends on
  // those exponentials, so the matrix pipe has work while the vector ALU computes them).  Each
  // step refills the fragment registers its two MFMAs have just consumed with the next
  // iteration's (V of sub-tile t, K of sub-tile t + 2), so those reads have most of an
  // iteration to land before they are used.  A raise of the maximum in
  // iteration t rescales O after sub-tile t - 1 has been added with the old maximum.
  // Sub-tile x lives in ring slot x mod RING; its last reads are those of iteration x.  The
  // iterations run in pairs (t even, t + 1) with one barrier after each pair: after it, the
  // copies of sub-tiles t + RING - 2 and t + RING - 1 go into the slots of t - 2 and t - 1,
  // and the barrier closing iteration t + 1 follows the landing of sub-tile t + 5 (the last
  // one the next pair reads).
  uint32_t cvoff[AC::kCopies];
  copy_offsets<D>(cvoff, wave);
  if (QUANT) build_tables(tab, a.qmax, a.ro.off);  // read after the prologue's barrier
  // prologue: sub-tiles 0 .. RING-3 in flight; 0 .. 3 landed before the loop
  for (int t = 0; t < RING - 2 && t < nsub; ++t)
    copy_subtile<D>(kb, vb, 32 * t, ntok, ring_lds + (uint32_t)(t * AC::kSlotBytes), wave);
  wait_copies_but<AC::kCopies>(max(min(RING - 3, nsub - 1) - 3, 0));
  ring_barrier();
  Frag kf[KS];
  Frag vf[NDB][2];  // V of the sub-tile whose O += V P is pending (zero before the first)
  bf16x8 pb[2];     // its probabilities
#pragma unroll
  for (int db = 0; db < NDB; ++db) vf[db][0].u = vf[db][1].u = make_uint4(0, 0, 0, 0);
  pb[0] = pb[1] = (bf16x8){};
  f32x16 sc = {};
  if (active) {
    read_kfrag<D>(ring, kf);
#pragma unroll
    for (int s = 0; s < KS; ++s) sc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[s].v, qf[s].v, sc, 0, 0, 0);
    if (nsub > 1) read_kfrag<D>(ring + AC::kSlotBytes, kf);
  }
  __builtin_amdgcn_s_waitcnt(0xC07F);  // as at every barrier: no LDS read in flight into the loop
  // iteration t of the pipeline, with `cur` the slot of sub-tile t: consumes S of sub-tile t
  // (st) and leaves S of sub-tile t + 1 in sn; FULL marks a sub-tile of the context with all
  // 32 tokens present and sub-tile t + 2 existing (no mask, no bounds test)
  const auto iteration = [&](int t, int cur, f32x16& st, f32x16& sn, auto full) {
    constexpr bool FULL = decltype(full)::value;
    const char* slot = ring + cur * AC::kSlotBytes;
    // st[i]: token 32 t + (i/4)*8 + (lane/32)*4 + i%4 of the unit, the lane's row
    if (!FULL && (32 * (t + 1) > ntok || u.guide)) {
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int tok = 32 * t + (i >> 2) * 8 + (lane >> 5) * 4 + (i & 3);
        const bool seen = tok < ntok && (!u.guide || tok <= jrow);
        st[i] = seen ? st[i] : -INFINITY;
      }
    }
    // S of sub-tile t + 1 (past the end: a repeat of the last sub-tile, never used) and
    // O += V P of sub-tile t - 1, one MFMA of each per step (S first: its chain is
    // dependent), each step also computing 16 / KS of the exponentials of sub-tile t and
    // adding those of the step before (an exponential's result is not read right after it),
    // then reading the fragments of the next iteration into the registers just consumed; the
    // scheduling barriers keep the steps in this order.
    static_assert(KS == 2 * NDB, "as many S steps as O steps");
    constexpr int TPS = 16 / KS;  // terms per step
    float p[16];
    float e[4] = {-0.f, -0.f, -0.f, -0.f};  // -0 + x == x: the first additions fold away
    const bool kread = FULL || t + 2 < nsub;
    const int k2 = cur + 2 >= RING ? cur + 2 - RING : cur + 2;
    const char* kslot = ring + k2 * AC::kSlotBytes;
    const char* vtile = slot + AC::kTileBytes;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      sn = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[s].v, qf[s].v, s == 0 ? (f32x16){} : sn, 0, 0, 0);
      ot[s % NDB] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf[s % NDB][s / NDB].v, pb[s / NDB], ot[s % NDB], 0, 0, 0);
#pragma unroll
      for (int j = 0; j < TPS; ++j) {
        const int i = TPS * s + j;
        p[i] = __builtin_amdgcn_exp2f(fmaf(st[i], a.c, -m));
        if (s > 0) e[(i - TPS) & 3] += p[i - TPS];
      }
      // refill the fragments this step's MFMAs consumed: V of sub-tile t, K of sub-tile t + 2
      vf[s % NDB][s / NDB] = read_vfrag<D>(vtile, s % NDB, s / NDB);
      if (kread) read_kfrag_step<D>(kslot, kf[s], s);
      __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
      if (s > 0)
        __builtin_amdgcn_sched_group_barrier(0x002, TPS * 2, 0);
      else
        __builtin_amdgcn_sched_group_barrier(0x002, TPS, 0);
      __builtin_amdgcn_sched_group_barrier(0x400, TPS, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 3, 0);
      __builtin_amdgcn_sched_barrier(0);
    }
#pragma unroll
    for (int j = 0; j < TPS; ++j) e[(16 - TPS + j) & 3] += p[16 - TPS + j];
    float ps = (e[0] + e[1]) + (e[2] + e[3]);
    const bool big = !(ps < kAttnLazyLimit);
    const uint64_t bal = __builtin_amdgcn_ballot_w64(big);
    if (bal) {
      const uint32_t pair = (uint32_t)bal | (uint32_t)(bal >> 32);
      if ((pair >> (lane & 31)) & 1u) raise_max<NDB>(st, a.c, m, lsum, ot, p, ps);
    }
    lsum += ps;
#pragma unroll
    for (int s2 = 0; s2 < 2; ++s2)
#pragma unroll
      for (int jj = 0; jj < 8; ++jj) pb[s2][jj] = (__bf16)p[8 * s2 + jj];
  };
  // Step 2 of the token rows of a pair of sub-tiles: waves 0-3 take sub-tile t, 4-7 sub-tile
  // t + 1, 8 rows each, a lane QNP adjacent 16-byte pieces of its row; read from the staged V
  // tile, quantised, scale and codes stored.  Only the workgroup of the chunk's first row
  // group does this.  Its stores are vector-memory operations like the ring's copies and may
  // complete out of order with them, so this instance waits for all of a wave's memory
  // operations at each barrier (vmcnt(0)), which leaves each pair's copies the pair's
  // duration to land.
  const bool qwg = QUANT && !u.guide && u.rg == 0;
  const QuantFmt qfmt{a.qfmt == TP_QFMT_INT, a.qfmt == TP_QFMT_INT && a.bits <= 4, a.qmax};
  const int64_t qrow0 = (int64_t)u.seg * a.n_tot + u.n0 + (int64_t)u.chunk * a.chunk;
  const int qtl = 8 * (wave & 3) + lane / QLPT;  // the lane's row of its sub-tile
  const int qj = lane % QLPT;                     // and its first piece, QNP qj
  const auto quant_pair = [&](int t, int cur, int c1) {
    const int x = t + (wave >> 2);
    if (x >= nsub) return;  // wave-uniform
    const char* vt = ring + (wave < 4 ? cur : c1) * AC::kSlotBytes + AC::kTileBytes + qtl * C::kRowBytes;
    uint4 xv[QNP];
#pragma unroll
    for (int n = 0; n < QNP; ++n) xv[n] = *(const uint4*)(vt + (((QNP * qj + n) ^ swzv<D>(qtl)) << 4));
    uint2 cd[QNP];
    const float gamma = quant_pieces<QLPT, QKC, QNP>(xv, tab, qfmt, cd);
    const int tok = 32 * x + qtl;
    if (tok < ntok) {  // rows past the chunk's end repeat its last row
      const int64_t row = qrow0 + tok;
      if (qj == 0) a.scales[row] = gamma;
      store_code_pieces<D, QKC, QNP>(a.vq, row, qj, cd);
    }
  };
  using Full = std::integral_constant<bool, true>;
  using Any = std::integral_constant<bool, false>;
  f32x16 sc2;  // S of the odd sub-tile of a pair
  int cur = 0;  // slot of sub-tile t
  int t = 0;
  // Pairs whose copies are whole context sub-tiles (t + RING - 1 <= nsub - 2): no bounds
  // tests, a fixed wait and copies addressed from a wave-uniform base.
  if (!u.guide) {
    for (; t + RING < nsub; t += 2) {
      const int f1 = cur >= 2 ? cur - 2 : cur + RING - 2;
      copy_whole<D>(kb, vb, 32 * (t + RING - 2), cvoff, ring_lds + (uint32_t)(f1 * AC::kSlotBytes), wave);
      const int f2 = cur >= 1 ? cur - 1 : cur + RING - 1;
      copy_whole<D>(kb, vb, 32 * (t + RING - 1), cvoff, ring_lds + (uint32_t)(f2 * AC::kSlotBytes), wave);
      const int c1 = cur + 1 == RING ? 0 : cur + 1;
      if (qwg) quant_pair(t, cur, c1);
      if (active) {
        iteration(t, cur, sc, sc2, Full{});
        iteration(t + 1, c1, sc2, sc, Full{});
      }
      // sub-tile t + 5 has landed for every wave; those of t + 6 .. t + RING - 1 may not have
      if (QUANT)
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
      else
        asm volatile("s_waitcnt vmcnt(%0)" ::"n"((RING - 6) * AC::kCopies) : "memory");
      ring_barrier();
      cur = c1 + 1 == RING ? 0 : c1 + 1;
    }
  }
  for (; t < nsub; t += 2) {
    // the slots of sub-tiles t - 2 and t - 1, read before the last barrier
    const int f1 = cur >= 2 ? cur - 2 : cur + RING - 2;
    const int f2 = cur >= 1 ? cur - 1 : cur + RING - 1;
    if (t + RING - 2 < nsub)
      copy_subtile<D>(kb, vb, 32 * (t + RING - 2), ntok, ring_lds + (uint32_t)(f1 * AC::kSlotBytes), wave);
    if (t + RING - 1 < nsub)
      copy_subtile<D>(kb, vb, 32 * (t + RING - 1), ntok, ring_lds + (uint32_t)(f2 * AC::kSlotBytes), wave);
    const int c1 = cur + 1 == RING ? 0 : cur + 1;
    if (qwg) quant_pair(t, cur, c1);
    if (active) {
      iteration(t, cur, sc, sc2, Any{});
      if (t + 1 < nsub) iteration(t + 1, c1, sc2, sc, Any{});
    }
    // sub-tile t + 5 has landed for every wave; copies of t + 6 .. may stay in flight
    if (QUANT)
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    else
      wait_copies_but<AC::kCopies>(max(min(t + RING - 1, nsub - 1) - (t + 5), 0));
    ring_barrier();
    cur = c1 + 1 == RING ? 0 : c1 + 1;
  }
  if (active) {  // O += V P of the last sub-tile
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int s2 = 0; s2 < 2; ++s2)
        ot[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf[db][s2].v, pb[s2], ot[db], 0, 0, 0);
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

template <int D>
void launch_fwd(const AttnArgs& a, dim3 grid, hipStream_t stream) {
  if (a.vq == nullptr) {
    hipLaunchKernelGGL((k_guide_fwd<D, kAttnNoQuant>), grid, dim3(kAttnThreads), 0, stream, a);
    return;
  }
  switch (qkind_of(a.qfmt, a.bits)) {
    case kQInt8:
      hipLaunchKernelGGL((k_guide_fwd<D, kQInt8>), grid, dim3(kAttnThreads), 0, stream, a);
      break;
    case kQByte:
      hipLaunchKernelGGL((k_guide_fwd<D, kQByte>), grid, dim3(kAttnThreads), 0, stream, a);
      break;
    case kQNibble:
      hipLaunchKernelGGL((k_guide_fwd<D, kQNibble>), grid, dim3(kAttnThreads), 0, stream, a);
      break;
    default:
      hipLaunchKernelGGL((k_guide_fwd<D, kQE4M3>), grid, dim3(kAttnThreads), 0, stream, a);
  }
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
    launch_fwd<128>(a, grid, stream);
    hipLaunchKernelGGL(k_guide_fwd_merge<128>, mgrid, dim3(256), 0, stream, a);
  } else {
    launch_fwd<64>(a, grid, stream);
    hipLaunchKernelGGL(k_guide_fwd_merge<64>, mgrid, dim3(256), 0, stream, a);
  }
  return hipGetLastError();
}

}  // namespace tp
