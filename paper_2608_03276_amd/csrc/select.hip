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

// Exclusive block scan of v (1024 threads); returns the prefix and sets `total`.
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
    const uint32_t w = lane < kSelWaves ? sh[lane] : 0u;
    uint32_t s = w;
#pragma unroll
    for (int off = 1; off < kSelWaves; off <<= 1) {
      const uint32_t y = __shfl_up(s, off);
      if (lane >= off) s += y;
    }
    if (lane < kSelWaves) sh[lane] = s - w;
    if (lane == kSelWaves - 1) sh[kSelWaves] = s;
  }
  __syncthreads();
  const uint32_t r = x - v + sh[wave];
  total = sh[kSelWaves];
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

hipError_t launch_select(const SelectArgs& a, int segments, hipStream_t stream) {
  hipLaunchKernelGGL(k_select, dim3((unsigned)segments, (unsigned)a.bt.batch), dim3(kSelThreads), 0, stream, a);
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
