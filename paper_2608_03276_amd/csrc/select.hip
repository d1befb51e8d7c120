// Step 3 of the eviction path: the combined score (Eq. 3, or a variant from the
// aggregation table of Sec. 4.4) and the top-k kept set of every (sequence, layer, KV head)
// (Sec. 3.4; uniform per-head budget, Sec. 4 setup).
//
// One 1024-thread workgroup per segment.  The combined score S is written once (fp32) and
// ranked through the order-preserving map of its bit pattern to uint32:
//   - a radix select finds the k-th largest key T and how many keys equal to T are needed
//     (ties go to the lower index): a 12-bit histogram of the top digit while S is formed,
//     then the keys in T's top-digit bucket are collected into LDS (when they fit; else the
//     remaining digits re-read S from memory) and their 12-bit and 8-bit digits are ranked
//     there, so S is read back only twice (collection and compaction) instead of once per
//     digit;
//   - an ordered compaction then emits, in ascending token order, every index with key > T
//     plus the first `need` indices with key == T: its output slot is
//     #(key > T before i) + min(#(key == T before i), need), from one block-wide scan of a
//     packed (greater, equal) count per tile.
// Only integer LDS atomics (histogram counts) are used, so the result is deterministic.
#include <mutex>

#include "tp_internal.h"

namespace tp {
namespace {

constexpr int kSelThreads = 1024;
constexpr int kSelWaves = kSelThreads / 64;
constexpr int kPerThread = 4;
constexpr int kBatch = 16;  // keys each thread loads before it touches the histogram
constexpr int kTopBits = 12;              // first digit: bits 31..20 of the key
constexpr int kBins = 1 << kTopBits;      // histogram bins (the 8-bit last digit uses 256)
constexpr int kCandCap = 16384;           // keys of the threshold's top-digit bucket held in LDS

__device__ inline uint32_t order_key(float s) {
  uint32_t b = __float_as_uint(s);
  if (b == 0x80000000u) b = 0u;  // -0 ranks with +0
  return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}

__device__ inline float combine(int rule, float s, float g, double na, double nb) {
  switch (rule) {
    case TP_COMBINE_KEY_ONLY:
      return s;
    case TP_COMBINE_HARMONIC: {
      const double den = (double)s + (double)g;
      return den > 0.0 ? (float)((2.0 * (double)s * (double)g) / den) : 0.0f;
    }
    case TP_COMBINE_NORM_ADD: {
      const double ta = na > 0.0 ? (double)s / na : 0.0;
      const double tb = nb > 0.0 ? (double)g / nb : 0.0;
      return (float)(ta + tb);
    }
    default:
      return s * g;
  }
}

// Wave 0: the digit of the k-th largest key among the histogram's nbins (highest first) and
// how many keys of that digit are still needed (krem counts from the top).  Lane l owns the
// per = nbins/64 digits below nbins - per*l.
__device__ inline void pick_digit(const uint32_t* hist, int nbins, uint32_t krem, uint32_t* sel) {
  const int lane = threadIdx.x & 63;
  const int per = nbins / 64;
  uint32_t lsum = 0;
  for (int e = 0; e < per; ++e) lsum += hist[nbins - 1 - per * lane - e];
  uint32_t incl = lsum;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const uint32_t y = __shfl_up(incl, off);
    if (lane >= off) incl += y;
  }
  const uint32_t excl = incl - lsum;
  if (excl < krem && krem <= incl) {
    uint32_t cum = excl;
    for (int e = 0; e < per; ++e) {
      const uint32_t c = hist[nbins - 1 - per * lane - e];
      if (cum + c >= krem) {
        sel[0] = (uint32_t)(nbins - 1 - per * lane - e);
        sel[1] = krem - cum;
        break;
      }
      cum += c;
    }
  }
}

// Exclusive block scan of v over NW waves (NW * 64 threads); returns the prefix and sets
// `total`.  sh holds NW + 1 words.
template <int NW = kSelWaves>
__device__ inline uint32_t block_scan(uint32_t v, uint32_t* sh, uint32_t& total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  uint32_t x = v;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const uint32_t y = __shfl_up(x, off);
    if (lane >= off) x += y;
  }
  if (lane == 63) sh[wave] = x;
  __syncthreads();
  if (wave == 0) {
    const uint32_t w = lane < NW ? sh[lane] : 0u;
    uint32_t s = w;
#pragma unroll
    for (int off = 1; off < NW; off <<= 1) {
      const uint32_t y = __shfl_up(s, off);
      if (lane >= off) s += y;
    }
    if (lane < NW) sh[lane] = s - w;
    if (lane == NW - 1) sh[NW] = s;
  }
  __syncthreads();
  const uint32_t r = x - v + sh[wave];
  total = sh[NW];
  __syncthreads();
  return r;
}

__global__ __launch_bounds__(kSelThreads) void k_select(SelectArgs a) {
  const int seg = blockIdx.x, b = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int64_t n0 = a.bt.ctx_off[b];
  const int64_t nb = a.bt.ctx_off[b + 1] - n0;
  const int64_t k = a.k[b];
  const float* sk = a.s_key + (int64_t)seg * a.n_tot + n0;
  const float* sc = a.scales + (int64_t)seg * a.n_tot + n0;
  float* sb = a.s_buf + (int64_t)seg * a.n_tot + n0;
  int32_t* out = a.kept + (int64_t)seg * a.k_tot + a.kept_off[b];

  __shared__ uint32_t hist[kBins];
  __shared__ uint32_t cand[kCandCap];
  __shared__ uint32_t scan_sh[kSelWaves + 1];
  __shared__ double dred[kSelWaves][2];
  __shared__ uint32_t sel[2];  // picked digit, keys of it still needed
  __shared__ uint32_t ncand;

  double norm_a = 0.0, norm_b = 0.0;
  if (a.rule == TP_COMBINE_NORM_ADD) {
    double s1 = 0.0, s2 = 0.0;
    for (int64_t i = tid; i < nb; i += kSelThreads) {
      const double x = sk[i], y = sc[i];
      s1 += x * x;
      s2 += y * y;
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
      s1 += __shfl_xor(s1, off);
      s2 += __shfl_xor(s2, off);
    }
    if (lane == 0) {
      dred[wave][0] = s1;
      dred[wave][1] = s2;
    }
    __syncthreads();
    double t1 = 0.0, t2 = 0.0;
    for (int w = 0; w < kSelWaves; ++w) {
      t1 += dred[w][0];
      t2 += dred[w][1];
    }
    norm_a = sqrt(t1);
    norm_b = sqrt(t2);
  }

  for (int i = tid; i < kBins; i += kSelThreads) hist[i] = 0;
  __syncthreads();
  // batches of kBatch keys per thread: the loads of a batch are in flight together
  for (int64_t i0 = 0; i0 < nb; i0 += (int64_t)kSelThreads * kBatch) {
    float x[kBatch], y[kBatch];
#pragma unroll
    for (int e = 0; e < kBatch; ++e) {
      const int64_t i = i0 + (int64_t)e * kSelThreads + tid;
      x[e] = i < nb ? sk[i] : 0.f;
      y[e] = i < nb ? sc[i] : 0.f;
    }
#pragma unroll
    for (int e = 0; e < kBatch; ++e) {
      const int64_t i = i0 + (int64_t)e * kSelThreads + tid;
      if (i < nb) {
        const float S = combine(a.rule, x[e], y[e], norm_a, norm_b);
        sb[i] = S;
        atomicAdd(&hist[order_key(S) >> (32 - kTopBits)], 1u);
      }
    }
  }
  __syncthreads();

  if (wave == 0) pick_digit(hist, kBins, (uint32_t)k, sel);
  __syncthreads();
  uint32_t prefix = sel[0], krem = sel[1];
  const uint32_t bucket = hist[prefix];  // keys sharing T's top digit
  const bool in_lds = bucket <= (uint32_t)kCandCap;
  if (tid == 0) ncand = 0;
  __syncthreads();
  if (in_lds) {  // collect that bucket's keys (their order does not matter: only counts are used)
    for (int64_t i0 = 0; i0 < nb; i0 += (int64_t)kSelThreads * kBatch) {
      float x[kBatch];
#pragma unroll
      for (int e = 0; e < kBatch; ++e) {
        const int64_t i = i0 + (int64_t)e * kSelThreads + tid;
        x[e] = i < nb ? sb[i] : 0.f;
      }
#pragma unroll
      for (int e = 0; e < kBatch; ++e) {
        const int64_t i = i0 + (int64_t)e * kSelThreads + tid;
        const uint32_t key = order_key(x[e]);
        const bool hit = i < nb && (key >> (32 - kTopBits)) == prefix;
        const uint64_t m = __builtin_amdgcn_ballot_w64(hit);
        if (m != 0) {  // one LDS atomic per wave
          uint32_t base = 0;
          if (lane == 0) base = atomicAdd(&ncand, (uint32_t)__builtin_popcountll(m));
          base = __shfl(base, 0);
          const uint32_t rank = __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
          if (hit && base + rank < (uint32_t)kCandCap) cand[base + rank] = key;
        }
      }
    }
    __syncthreads();
  }
  // the two remaining digits: bits 19..8 (12 bits), then bits 7..0 (8 bits)
  for (int pass = 0; pass < 2; ++pass) {
    const int shift = pass == 0 ? 8 : 0;
    const int nbins = pass == 0 ? kBins : 256;
    const uint32_t mask = (uint32_t)nbins - 1u;
    for (int i = tid; i < nbins; i += kSelThreads) hist[i] = 0;
    __syncthreads();
    if (in_lds) {
      for (uint32_t i = tid; i < bucket; i += kSelThreads) {
        const uint32_t key = cand[i];
        if ((key >> (shift + (pass == 0 ? 12 : 8))) == prefix) atomicAdd(&hist[(key >> shift) & mask], 1u);
      }
    } else {
      for (int64_t i0 = 0; i0 < nb; i0 += (int64_t)kSelThreads * kBatch) {
        float x[kBatch];
#pragma unroll
        for (int e = 0; e < kBatch; ++e) {
          const int64_t i = i0 + (int64_t)e * kSelThreads + tid;
          x[e] = i < nb ? sb[i] : 0.f;
        }
#pragma unroll
        for (int e = 0; e < kBatch; ++e) {
          const int64_t i = i0 + (int64_t)e * kSelThreads + tid;
          const uint32_t key = order_key(x[e]);
          if (i < nb && (key >> (shift + (pass == 0 ? 12 : 8))) == prefix) atomicAdd(&hist[(key >> shift) & mask], 1u);
        }
      }
    }
    __syncthreads();
    if (wave == 0) pick_digit(hist, nbins, krem, sel);
    __syncthreads();
    prefix = (prefix << (pass == 0 ? 12 : 8)) | sel[0];
    krem = sel[1];
    __syncthreads();
  }
  const uint32_t T = prefix, need = krem;

  uint32_t gt_run = 0, eq_run = 0;
  for (int64_t t0 = 0; t0 < nb; t0 += (int64_t)kSelThreads * kPerThread) {
    const int64_t i0 = t0 + (int64_t)tid * kPerThread;
    uint32_t keys[kPerThread];
    uint32_t gtc = 0, eqc = 0;
#pragma unroll
    for (int e = 0; e < kPerThread; ++e) {
      const int64_t i = i0 + e;
      keys[e] = i < nb ? order_key(sb[i]) : 0u;
      if (i < nb) {
        gtc += keys[e] > T;
        eqc += keys[e] == T;
      }
    }
    uint32_t total;
    const uint32_t ex = block_scan((gtc << 16) | eqc, scan_sh, total);
    uint32_t gx = gt_run + (ex >> 16), qx = eq_run + (ex & 0xFFFFu);
#pragma unroll
    for (int e = 0; e < kPerThread; ++e) {
      const int64_t i = i0 + e;
      if (i >= nb) break;
      if (keys[e] > T) {
        const uint32_t pos = gx + (qx < need ? qx : need);
        if (pos < (uint32_t)k) out[pos] = (int32_t)i;
        ++gx;
      } else if (keys[e] == T) {
        if (qx < need && gx + qx < (uint32_t)k) out[gx + qx] = (int32_t)i;
        ++qx;
      }
    }
    gt_run += total >> 16;
    eq_run += total & 0xFFFFu;
  }
}

// ---------------------------------------------------------------------------- split selection
// The same selection with each segment's tokens cut into parts of kSelPartTokens, so a
// segment is worked on by several workgroups, each of which handles its part in one step (all
// of its loads in flight together).  No workgroup waits for another (five launches, each
// reading what the previous ones wrote), and only integer counts are combined, so the result
// does not depend on the order in which workgroups run:
//   k_sel_score    per part: (pooling of pass 2's raw sums, when fused) the combined score S,
//                  written once, and the part's histogram of the 12-bit top digit of its keys;
//   k_sel_pick     per segment: the parts' histograms summed, the top digit of the k-th key;
//   k_sel_collect  per part: the part's keys in that digit's bucket into the segment's
//                  candidate list (each part at the offset its predecessors' counts give), and
//                  the count of its keys above the bucket;
//   k_sel_refine   per segment: the remaining 20 bits of the threshold key T ranked over the
//                  candidates in LDS (from S in memory when the bucket exceeds the list),
//                  how many keys equal to T are needed, and per part the counts of keys > T
//                  and == T before it;
//   k_sel_emit     per part: the ordered compaction of the part from those starting counts.
constexpr int kPartThreads = 512;
constexpr int kScorePer = kSelPartTokens / kPartThreads;  // tokens per thread in k_sel_score
constexpr int kCollectPer = kSelPartTokens / kPartThreads;
constexpr int kEmitThreads = 256;
constexpr int kEmitPer = kSelPartTokens / kEmitThreads;   // tokens per thread in k_sel_emit
constexpr int kPoolHaloMax = 512;             // wider pooling windows sum straight from memory
constexpr int kHistWords = kBins / 2;         // a part histogram: 16-bit counts, two per word
constexpr int kLdsParts = 2048;               // parts whose counts k_sel_refine keeps in LDS
static_assert(kSelPartTokens < 65536, "per-part counts fit 16 bits");
static_assert(kSelPartTokens == kPartThreads * kScorePer && kSelPartTokens == kEmitThreads * kEmitPer, "tiling");

// Count of bin `bin` in a part's packed histogram.
__device__ inline uint32_t part_count(const uint32_t* hp, uint32_t bin) {
  return (hp[bin >> 1] >> (16 * (bin & 1))) & 0xFFFFu;
}

// Lanes below this one in a wave's ballot mask.
__device__ inline uint32_t lanes_below(uint64_t m) {
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
}

struct PartRange {
  int64_t n0, nb, i0, i1;  // sequence start, length; the part's tokens [i0, i1) within it
};

__device__ inline bool part_range(const SelectArgs& a, int p, int b, PartRange& r) {
  r.n0 = a.bt.ctx_off[b];
  r.nb = a.bt.ctx_off[b + 1] - r.n0;
  r.i0 = (int64_t)p * kSelPartTokens;
  r.i1 = r.i0 + kSelPartTokens < r.nb ? r.i0 + kSelPartTokens : r.nb;
  return r.i0 < r.nb;
}

__device__ inline int parts_of(int64_t nb) { return (int)((nb + kSelPartTokens - 1) / kSelPartTokens); }

// Sum of the row groups' raw sums at token j, in row-group order (as the pooling kernel).
__device__ inline float raw_sum(const float* raw, int nrg, int64_t stride, int64_t j) {
  float v = raw[j];
  for (int rg = 1; rg < nrg; ++rg) v += raw[rg * stride + j];
  return v;
}

// The pooled value at LDS position l (the window's first element): the window summed left to
// right from zero, as the pooling kernel does; HALF = -1 takes the window's half-width from h.
template <int HALF>
__device__ inline float window_sum(const float* tile, int l, int h) {
  float acc = 0.f;
  if (HALF >= 0) {
#pragma unroll
    for (int t = 0; t <= 2 * HALF; ++t) acc += tile[l + t];
  } else {
    for (int t = 0; t <= 2 * h; ++t) acc += tile[l + t];
  }
  return acc;
}

// HALF: the pooling half-width this instance is specialised for (-1: any width up to
// kPoolHaloMax staged in LDS, -2: wider windows summed from memory, -3: no pooling here, the
// key score is read).
template <int HALF>
__global__ __launch_bounds__(kPartThreads) void k_sel_score(SelectArgs a, int seg0, int segments) {
  const int p = blockIdx.x, seg = seg0 + blockIdx.y, b = blockIdx.z, tid = threadIdx.x;
  PartRange r;
  if (!part_range(a, p, b, r)) return;
  constexpr bool kStaged = HALF >= -1;
  __shared__ uint32_t hist[kBins];
  __shared__ float tile[kStaged ? kSelPartTokens + 2 * kPoolHaloMax : 1];
  for (int i = tid; i < kBins; i += kPartThreads) hist[i] = 0;
  const int64_t base = (int64_t)seg * a.n_tot + r.n0;
  const int ntok = (int)(r.i1 - r.i0);
  const int half = HALF >= 0 ? HALF : a.pool_half;
  const int nrg = a.nrg[b];
  const int64_t rstride = (int64_t)segments * a.n_tot;  // one row group's [L*Hkv][N_tot]
  float sk[kScorePer], g[kScorePer];
  // every load of the part in flight together: the scales, and the raw sums of the part and
  // its halo into LDS (zero outside the sequence) or the key scores
#pragma unroll
  for (int e = 0; e < kScorePer; ++e) {
    const int l = tid + kPartThreads * e;
    g[e] = l < ntok ? a.scales[base + r.i0 + l] : 0.f;
  }
  if (kStaged) {
    const float* raw = a.raw + base;
    const int nstage = ntok + 2 * half;
    constexpr int kStageMax = (kSelPartTokens + 2 * kPoolHaloMax + kPartThreads - 1) / kPartThreads;
    float v[kStageMax];
#pragma unroll
    for (int e = 0; e < kStageMax; ++e) {
      const int t = tid + kPartThreads * e;
      const int64_t j = r.i0 - half + t;
      v[e] = (t < nstage && j >= 0 && j < r.nb) ? raw_sum(raw, nrg, rstride, j) : 0.f;
    }
#pragma unroll
    for (int e = 0; e < kStageMax; ++e) {
      const int t = tid + kPartThreads * e;
      if (t < nstage) tile[t] = v[e];
    }
  } else if (HALF == -3) {
#pragma unroll
    for (int e = 0; e < kScorePer; ++e) {
      const int l = tid + kPartThreads * e;
      sk[e] = l < ntok ? a.s_key[base + r.i0 + l] : 0.f;
    }
  }
  __syncthreads();
  if (kStaged) {
#pragma unroll
    for (int e = 0; e < kScorePer; ++e) {
      const int l = tid + kPartThreads * e;
      sk[e] = l < ntok ? window_sum<HALF>(tile, l, half) * a.pool_inv : 0.f;
    }
  } else if (HALF == -2) {  // wide windows: direct sums, as the pooling kernel's direct path
    const float* raw = a.raw + base;
#pragma unroll
    for (int e = 0; e < kScorePer; ++e) {
      const int64_t i = r.i0 + tid + kPartThreads * e;
      float acc = 0.f;
      if (i < r.i1)
        for (int t = -half; t <= half; ++t)
          if (i + t >= 0 && i + t < r.nb) acc += raw_sum(raw, nrg, rstride, i + t);
      sk[e] = acc * a.pool_inv;
    }
  }
#pragma unroll
  for (int e = 0; e < kScorePer; ++e) {
    const int l = tid + kPartThreads * e;
    if (l < ntok) {
      if (HALF != -3) a.s_key_out[base + r.i0 + l] = sk[e];
      const float S = combine(a.rule, sk[e], g[e], 0.0, 0.0);
      a.s_buf[base + r.i0 + l] = S;
      atomicAdd(&hist[order_key(S) >> (32 - kTopBits)], 1u);
    }
  }
  __syncthreads();
  uint32_t* hp = a.hist + ((int64_t)seg * a.part_tot + a.part_off[b] + p) * kHistWords;
  for (int w = tid; w < kHistWords; w += kPartThreads) hp[w] = hist[2 * w] | (hist[2 * w + 1] << 16);
}

__global__ __launch_bounds__(kSelThreads) void k_sel_pick(SelectArgs a) {
  const int seg = blockIdx.x, b = blockIdx.y, tid = threadIdx.x;
  const int64_t nb = a.bt.ctx_off[b + 1] - a.bt.ctx_off[b];
  const int np = parts_of(nb);
  __shared__ uint32_t hist[kBins];
  __shared__ uint32_t sel[2];
  const uint32_t* h0 = a.hist + ((int64_t)seg * a.part_tot + a.part_off[b]) * kHistWords;
  // thread t sums words t and t + 1024 over the parts, eight parts' loads at a time
  for (int w = tid; w < kHistWords; w += kSelThreads) {
    uint32_t lo = 0, hi = 0;
    for (int p0 = 0; p0 < np; p0 += 8) {
      uint32_t v[8];
#pragma unroll
      for (int q = 0; q < 8; ++q) v[q] = p0 + q < np ? h0[(int64_t)(p0 + q) * kHistWords + w] : 0u;
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        lo += v[q] & 0xFFFFu;
        hi += v[q] >> 16;
      }
    }
    hist[2 * w] = lo;
    hist[2 * w + 1] = hi;
  }
  __syncthreads();
  if (tid < 64) pick_digit(hist, kBins, (uint32_t)a.k[b], sel);
  __syncthreads();
  const uint32_t bdig = sel[0];
  if (tid == 0) a.info[(int64_t)seg * a.bt.batch + b] = make_uint4(bdig, sel[1], hist[bdig], 0u);
  // each part's first slot in the candidate list: the running sum of the parts' counts of the
  // picked digit (the histogram's LDS is reused for the counts)
  uint32_t* cs = a.cstart + (int64_t)seg * a.part_tot + a.part_off[b];
  __syncthreads();
  if (np <= kBins) {
    for (int q = tid; q < np; q += kSelThreads) hist[q] = part_count(h0 + (int64_t)q * kHistWords, bdig);
    __syncthreads();
    if (tid == 0) {
      uint32_t run = 0;
      for (int q = 0; q < np; ++q) {
        const uint32_t c = hist[q];
        hist[q] = run;
        run += c;
      }
    }
    __syncthreads();
    for (int q = tid; q < np; q += kSelThreads) cs[q] = hist[q];
  } else if (tid == 0) {
    uint32_t run = 0;
    for (int q = 0; q < np; ++q) {
      cs[q] = run;
      run += part_count(h0 + (int64_t)q * kHistWords, bdig);
    }
  }
}

__global__ __launch_bounds__(kPartThreads) void k_sel_collect(SelectArgs a) {
  const int p = blockIdx.x, seg = blockIdx.y, b = blockIdx.z, tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  PartRange r;
  if (!part_range(a, p, b, r)) return;
  // thread t holds the part's tokens c * 4 * kPartThreads + 4 t .. + 3 for each of kCollectLoads
  // 16-byte loads (coalesced; one float at a time where the segment is not 16-byte aligned)
  constexpr int kCollectLoads = kCollectPer / 4;
  const float* sb = a.s_buf + (int64_t)seg * a.n_tot + r.n0;
  const int ntok = (int)(r.i1 - r.i0);
  const bool vec = (((int64_t)seg * a.n_tot + r.n0) & 3) == 0;
  float4 x[kCollectLoads];
#pragma unroll
  for (int c = 0; c < kCollectLoads; ++c) {
    const int t = c * 4 * kPartThreads + 4 * tid;
    if (vec && t + 3 < ntok) {
      x[c] = *(const float4*)(sb + r.i0 + t);
    } else {
      x[c].x = t < ntok ? sb[r.i0 + t] : 0.f;
      x[c].y = t + 1 < ntok ? sb[r.i0 + t + 1] : 0.f;
      x[c].z = t + 2 < ntok ? sb[r.i0 + t + 2] : 0.f;
      x[c].w = t + 3 < ntok ? sb[r.i0 + t + 3] : 0.f;
    }
  }
  const uint4 info = a.info[(int64_t)seg * a.bt.batch + b];
  const uint32_t bdig = info.x, bucket = info.z;
  const int64_t cap = a.cand_off[b + 1] - a.cand_off[b];
  const bool store = bucket <= (uint64_t)cap;
  const uint32_t* h0 = a.hist + ((int64_t)seg * a.part_tot + a.part_off[b]) * kHistWords;
  const uint32_t start = a.cstart[(int64_t)seg * a.part_tot + a.part_off[b] + p];  // the earlier parts' keys
  uint32_t* cand = a.cand + (int64_t)seg * a.cand_tot + a.cand_off[b] + start;
  __shared__ uint32_t ncand;
  __shared__ uint32_t above_w[kPartThreads / 64];
  if (tid == 0) ncand = 0;
  __syncthreads();
  uint32_t above = 0;
#pragma unroll
  for (int c = 0; c < kCollectLoads; ++c) {
    const int t = c * 4 * kPartThreads + 4 * tid;
    const float v[4] = {x[c].x, x[c].y, x[c].z, x[c].w};
    uint32_t key[4], hits = 0;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      key[j] = order_key(v[j]);
      const uint32_t d = key[j] >> (32 - kTopBits);
      const bool valid = t + j < ntok;
      above += (valid && d > bdig) ? 1u : 0u;
      hits |= (store && valid && d == bdig) ? 1u << j : 0u;
    }
    if (__builtin_amdgcn_ballot_w64(hits != 0) != 0) {  // rare: the bucket holds ~1/50 of the keys
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const bool hit = (hits >> j) & 1u;
        const uint64_t m = __builtin_amdgcn_ballot_w64(hit);
        if (m != 0) {  // one LDS atomic per wave; the order of the keys does not matter
          uint32_t base = 0;
          if (lane == 0) base = atomicAdd(&ncand, (uint32_t)__builtin_popcountll(m));
          base = __shfl(base, 0);
          if (hit) cand[base + lanes_below(m)] = key[j];
        }
      }
    }
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) above += __shfl_xor(above, off);
  if (lane == 0) above_w[wave] = above;
  __syncthreads();
  if (tid == 0) {
    uint32_t t = 0;
    for (int w = 0; w < kPartThreads / 64; ++w) t += above_w[w];
    a.pcount[(int64_t)seg * a.part_tot + a.part_off[b] + p] = make_uint2(t, part_count(h0 + (int64_t)p * kHistWords, bdig));
  }
}

// Block-wide sum of one value per thread (1024 threads); every thread gets the total.
__device__ inline uint32_t block_sum(uint32_t v, uint32_t* sh) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
  if (lane == 0) sh[wave] = v;
  __syncthreads();
  uint32_t t = 0;
  for (int w = 0; w < kSelWaves; ++w) t += sh[w];
  __syncthreads();
  return t;
}

__global__ __launch_bounds__(kSelThreads) void k_sel_refine(SelectArgs a) {
  const int seg = blockIdx.x, b = blockIdx.y, tid = threadIdx.x, wave = tid >> 6;
  const int64_t n0 = a.bt.ctx_off[b];
  const int64_t nb = a.bt.ctx_off[b + 1] - n0;
  const int np = parts_of(nb);
  const uint4 info = a.info[(int64_t)seg * a.bt.batch + b];
  const uint32_t bucket = info.z;
  const int64_t cap = a.cand_off[b + 1] - a.cand_off[b];
  const bool in_lds = bucket <= (uint64_t)cap;
  const uint32_t* cg = a.cand + (int64_t)seg * a.cand_tot + a.cand_off[b];
  const float* sb = a.s_buf + (int64_t)seg * a.n_tot + n0;
  const uint2* pc = a.pcount + (int64_t)seg * a.part_tot + a.part_off[b];
  __shared__ uint32_t hist[kBins];
  __shared__ uint32_t cand[kSelCandCap];
  __shared__ uint32_t sel[2];
  __shared__ uint32_t red[kSelWaves];
  __shared__ uint32_t pstart[kLdsParts + 1];     // first candidate slot of each part
  __shared__ uint32_t pabove[kLdsParts];         // keys above the top-digit bucket, per part
  __shared__ uint32_t pgt[kLdsParts], peq[kLdsParts];
  const bool parts_in_lds = in_lds && np <= kLdsParts;
  if (in_lds)
    for (uint32_t i = tid; i < bucket; i += kSelThreads) cand[i] = cg[i];
  if (parts_in_lds) {
    const uint32_t* cs = a.cstart + (int64_t)seg * a.part_tot + a.part_off[b];
    for (int q = tid; q < np; q += kSelThreads) {
      pstart[q] = cs[q];
      pabove[q] = pc[q].x;
      pgt[q] = peq[q] = 0;
    }
    if (tid == 0) pstart[np] = bucket;
  }
  uint32_t prefix = info.x, krem = info.y;
  // the two remaining digits: bits 19..8 (12 bits), then bits 7..0 (8 bits)
  for (int pass = 0; pass < 2; ++pass) {
    const int shift = pass == 0 ? 8 : 0;
    const int nbins = pass == 0 ? kBins : 256;
    const uint32_t mask = (uint32_t)nbins - 1u;
    for (int i = tid; i < nbins; i += kSelThreads) hist[i] = 0;
    __syncthreads();
    if (in_lds) {
      for (uint32_t i = tid; i < bucket; i += kSelThreads) {
        const uint32_t key = cand[i];
        if ((key >> (shift + (pass == 0 ? 12 : 8))) == prefix) atomicAdd(&hist[(key >> shift) & mask], 1u);
      }
    } else {
      for (int64_t i0 = 0; i0 < nb; i0 += (int64_t)kSelThreads * kBatch) {
        float x[kBatch];
#pragma unroll
        for (int e = 0; e < kBatch; ++e) {
          const int64_t i = i0 + (int64_t)e * kSelThreads + tid;
          x[e] = i < nb ? sb[i] : 0.f;
        }
#pragma unroll
        for (int e = 0; e < kBatch; ++e) {
          const int64_t i = i0 + (int64_t)e * kSelThreads + tid;
          const uint32_t key = order_key(x[e]);
          if (i < nb && (key >> (shift + (pass == 0 ? 12 : 8))) == prefix) atomicAdd(&hist[(key >> shift) & mask], 1u);
        }
      }
    }
    __syncthreads();
    if (wave == 0) pick_digit(hist, nbins, krem, sel);
    __syncthreads();
    prefix = (prefix << (pass == 0 ? 12 : 8)) | sel[0];
    krem = sel[1];
    __syncthreads();
  }
  const uint32_t T = prefix, need = krem;
  // per part, the keys > T and == T; their running sums over the parts are each part's start
  uint2* pr = a.pref + (int64_t)seg * a.part_tot + a.part_off[b];
  if (parts_in_lds) {
    for (uint32_t i = tid; i < bucket; i += kSelThreads) {
      const uint32_t key = cand[i];
      if (key < T) continue;
      int lo = 0, hi = np;  // the part whose slot range holds i
      while (hi - lo > 1) {
        const int mid = (lo + hi) >> 1;
        if (pstart[mid] <= i) lo = mid; else hi = mid;
      }
      atomicAdd(key > T ? &pgt[lo] : &peq[lo], 1u);
    }
    __syncthreads();
    if (tid == 0) {  // running sums from LDS; the parts' starts are written in parallel below
      uint32_t gsum = 0, qsum = 0;
      for (int q = 0; q < np; ++q) {
        const uint32_t g = pabove[q] + pgt[q], e = peq[q];
        pgt[q] = gsum;
        peq[q] = qsum;
        gsum += g;
        qsum += e;
      }
    }
    __syncthreads();
    for (int q = tid; q < np; q += kSelThreads) pr[q] = make_uint2(pgt[q], peq[q]);
  } else {
    uint32_t gsum = 0, qsum = 0, slot = 0;
    for (int q = 0; q < np; ++q) {
      const uint2 c = pc[q];  // keys above the top-digit bucket, keys in it
      uint32_t gt = 0, eq = 0;
      if (in_lds) {
        for (uint32_t i = slot + tid; i < slot + c.y; i += kSelThreads) {
          gt += cand[i] > T;
          eq += cand[i] == T;
        }
      } else {
        const int64_t i1 = (int64_t)(q + 1) * kSelPartTokens < nb ? (int64_t)(q + 1) * kSelPartTokens : nb;
        for (int64_t i = (int64_t)q * kSelPartTokens + tid; i < i1; i += kSelThreads) {
          const uint32_t key = order_key(sb[i]);
          gt += key > T && (key >> (32 - kTopBits)) == info.x;  // keys above the bucket are in c.x
          eq += key == T;
        }
      }
      gt = block_sum(gt, red);
      eq = block_sum(eq, red);
      if (tid == 0) pr[q] = make_uint2(gsum, qsum);
      gsum += c.x + gt;
      qsum += eq;
      slot += c.y;
    }
  }
  if (tid == 0) a.thr[(int64_t)seg * a.bt.batch + b] = make_uint2(T, need);
}

__global__ __launch_bounds__(kEmitThreads) void k_sel_emit(SelectArgs a) {
  const int p = blockIdx.x, seg = blockIdx.y, b = blockIdx.z, tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  PartRange r;
  if (!part_range(a, p, b, r)) return;
  // wave w owns the part's tokens [w * kEmitRun, (w + 1) * kEmitRun) as kEmitChunks chunks
  // of 256 consecutive tokens; lane l holds the chunk's tokens 4l .. 4l + 3 (one 16-byte load,
  // coalesced).  A token's rank among the chunk's kept tokens before it is the lanes below
  // with such tokens (ballot per element slot, mbcnt) plus the lane's own earlier elements.
  constexpr int kEmitRun = kSelPartTokens / (kEmitThreads / 64);
  constexpr int kEmitChunks = kEmitRun / 256;
  const float* sb = a.s_buf + (int64_t)seg * a.n_tot + r.n0;
  const int ntok = (int)(r.i1 - r.i0);       // tokens of the part
  const int w0 = wave * kEmitRun;            // first token of the wave's run, from the part's start
  // 16-byte loads when the segment's scores start on a 16-byte boundary (s_buf is 16-byte
  // aligned, r.i0 and t are multiples of 4), else one float at a time (a ragged batch)
  const bool vec = (((int64_t)seg * a.n_tot + r.n0) & 3) == 0;
  float4 x[kEmitChunks];
#pragma unroll
  for (int c = 0; c < kEmitChunks; ++c) {
    const int t = w0 + c * 256 + 4 * lane;
    if (vec && t + 3 < ntok) {
      x[c] = *(const float4*)(sb + r.i0 + t);
    } else {
      x[c].x = t < ntok ? sb[r.i0 + t] : 0.f;
      x[c].y = t + 1 < ntok ? sb[r.i0 + t + 1] : 0.f;
      x[c].z = t + 2 < ntok ? sb[r.i0 + t + 2] : 0.f;
      x[c].w = t + 3 < ntok ? sb[r.i0 + t + 3] : 0.f;
    }
  }
  const uint2 th = a.thr[(int64_t)seg * a.bt.batch + b];
  const uint32_t T = th.x, need = th.y;
  const uint2 st = a.pref[(int64_t)seg * a.part_tot + a.part_off[b] + p];
  const uint32_t k = (uint32_t)a.k[b];
  int32_t* out = a.kept + (int64_t)seg * a.k_tot + a.kept_off[b];
  // per chunk and element slot, the lanes with a key > T / == T
  uint32_t gmask[kEmitChunks], emask[kEmitChunks];  // bit j: the lane's element j
  uint32_t gw = 0, qw = 0;
#pragma unroll
  for (int c = 0; c < kEmitChunks; ++c) {
    const int t = w0 + c * 256 + 4 * lane;
    const float v[4] = {x[c].x, x[c].y, x[c].z, x[c].w};
    uint32_t gm = 0, em = 0;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const uint32_t key = order_key(v[j]);
      const bool valid = t + j < ntok;
      gm |= (valid && key > T) ? 1u << j : 0u;
      em |= (valid && key == T) ? 1u << j : 0u;
    }
    gmask[c] = gm;
    emask[c] = em;
    gw += __builtin_popcount(gm);
    qw += __builtin_popcount(em);
  }
  // the wave's totals, then the earlier waves' through LDS
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    gw += __shfl_xor(gw, off);
    qw += __shfl_xor(qw, off);
  }
  __shared__ uint2 wave_tot[kEmitThreads / 64];
  if (lane == 0) wave_tot[wave] = make_uint2(gw, qw);
  __syncthreads();
  uint32_t gx = st.x, qx = st.y;  // keys > T and == T before this wave's run
  for (int w = 0; w < wave; ++w) {
    gx += wave_tot[w].x;
    qx += wave_tot[w].y;
  }
#pragma unroll
  for (int c = 0; c < kEmitChunks; ++c) {
    const uint32_t gm = gmask[c], em = emask[c];
    // keys of the lanes below: sum over the four element slots of the slot's ballot
    uint32_t gb = 0, eb = 0, gtot = 0, etot = 0;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const uint64_t mg = __builtin_amdgcn_ballot_w64((gm >> j) & 1u);
      const uint64_t me = __builtin_amdgcn_ballot_w64((em >> j) & 1u);
      gb += lanes_below(mg);
      eb += lanes_below(me);
      gtot += __builtin_popcountll(mg);
      etot += __builtin_popcountll(me);
    }
    if (gm | em) {
      const int t = w0 + c * 256 + 4 * lane;
      uint32_t g_before = gx + gb, q_before = qx + eb;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        if ((gm >> j) & 1u) {
          const uint32_t pos = g_before + (q_before < need ? q_before : need);
          if (pos < k) out[pos] = (int32_t)(r.i0 + t + j);
          ++g_before;
        } else if ((em >> j) & 1u) {
          if (q_before < need && g_before + q_before < k) out[g_before + q_before] = (int32_t)(r.i0 + t + j);
          ++q_before;
        }
      }
    }
    gx += gtot;
    qx += etot;
  }
}

constexpr int kMaxScratchDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxScratchDevices];  // per device: its copy of `scratch`, once resolved

}  // namespace

// Staging of the combined scores for tp_combine_select_topk_static (callers that cannot
// allocate): a file-scope device array, one copy per GPU the library's code is loaded on,
// kept until the process ends.  In host code `scratch` names a host-side stand-in, never a
// device address: each GPU's copy is found by hipGetSymbolAddress on that GPU, and only that
// address is handed to kernels.
static __device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

SelectWorkspace select_workspace_layout(int64_t segments, const int64_t* ctx_off, int32_t batch) {
  auto up = [](size_t x) { return (x + 255) & ~(size_t)255; };
  SelectWorkspace w;
  int64_t parts = 0, cands = 0;
  for (int b = 0; b < batch; ++b) {
    const int64_t nb = ctx_off[b + 1] - ctx_off[b];
    parts += (nb + kSelPartTokens - 1) / kSelPartTokens;
    cands += nb < kSelCandCap ? nb : kSelCandCap;
  }
  w.part_tot = parts;
  w.cand_tot = cands;
  const size_t segs = (size_t)segments;
  w.s_off = 0;
  w.hist_off = up((size_t)segs * ctx_off[batch] * sizeof(float));
  w.info_off = w.hist_off + up(segs * parts * (kBins / 2) * sizeof(uint32_t));
  w.thr_off = w.info_off + up(segs * batch * sizeof(uint4));
  w.pcount_off = w.thr_off + up(segs * batch * sizeof(uint2));
  w.pref_off = w.pcount_off + up(segs * parts * sizeof(uint2));
  w.cstart_off = w.pref_off + up(segs * parts * sizeof(uint2));
  w.cand_off = w.cstart_off + up(segs * parts * sizeof(uint32_t));
  w.total = w.cand_off + up(segs * cands * sizeof(uint32_t));
  return w;
}

hipError_t launch_select_score(const SelectArgs& a, int seg_begin, int seg_end, int segments, hipStream_t stream) {
  if (a.rule == TP_COMBINE_NORM_ADD || seg_end <= seg_begin) return hipSuccess;  // k_select forms S itself
  const dim3 parts((unsigned)a.part_max, (unsigned)(seg_end - seg_begin), (unsigned)a.bt.batch);
  const dim3 pb(kPartThreads);
  if (a.raw == nullptr)
    hipLaunchKernelGGL(k_sel_score<-3>, parts, pb, 0, stream, a, seg_begin, segments);
  else if (a.pool_half > kPoolHaloMax)
    hipLaunchKernelGGL(k_sel_score<-2>, parts, pb, 0, stream, a, seg_begin, segments);
  else if (a.pool_half == 2)  // pooling kernel 5, the benches' choice
    hipLaunchKernelGGL(k_sel_score<2>, parts, pb, 0, stream, a, seg_begin, segments);
  else if (a.pool_half == 0)
    hipLaunchKernelGGL(k_sel_score<0>, parts, pb, 0, stream, a, seg_begin, segments);
  else
    hipLaunchKernelGGL(k_sel_score<-1>, parts, pb, 0, stream, a, seg_begin, segments);
  return hipGetLastError();
}

hipError_t launch_select(const SelectArgs& a, int segments, hipStream_t stream, hipEvent_t after_score,
                         int scored_begin, int scored_end) {
  const dim3 segs((unsigned)segments, (unsigned)a.bt.batch);
  if (a.rule == TP_COMBINE_NORM_ADD) {  // the segment's norms come first: one workgroup per segment
    if (after_score) {
      const hipError_t e = hipEventRecord(after_score, stream);
      if (e != hipSuccess) return e;
    }
    hipLaunchKernelGGL(k_select, segs, dim3(kSelThreads), 0, stream, a);
    return hipGetLastError();
  }
  const dim3 parts((unsigned)a.part_max, (unsigned)segments, (unsigned)a.bt.batch);
  if (scored_end <= scored_begin) scored_begin = scored_end = 0;
  hipError_t e = launch_select_score(a, 0, scored_begin, segments, stream);
  if (e == hipSuccess) e = launch_select_score(a, scored_end, segments, segments, stream);
  if (e == hipSuccess && after_score) e = hipEventRecord(after_score, stream);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_sel_pick, segs, dim3(kSelThreads), 0, stream, a);
  hipLaunchKernelGGL(k_sel_collect, parts, dim3(kPartThreads), 0, stream, a);
  hipLaunchKernelGGL(k_sel_refine, segs, dim3(kSelThreads), 0, stream, a);
  hipLaunchKernelGGL(k_sel_emit, parts, dim3(kEmitThreads), 0, stream, a);
  return hipGetLastError();
}

hipError_t static_scratch(hipStream_t stream, void** ptr) {
  int dev = 0;
  hipError_t e = stream ? hipStreamGetDevice(stream, &dev) : hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxScratchDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    // once per device, with that device current: the address of its copy of the array
    int cur = 0;
    e = hipGetDevice(&cur);
    if (e == hipSuccess && cur != dev) e = hipSetDevice(dev);
    void* p = nullptr;
    if (e == hipSuccess) e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (cur != dev) {
      const hipError_t e2 = hipSetDevice(cur);
      if (e == hipSuccess) e = e2;
    }
    if (e != hipSuccess) return e;
    if (p == nullptr) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = p;
  }
  *ptr = g_scratch_ptr[dev];
  return hipSuccess;
}

}  // namespace tp
