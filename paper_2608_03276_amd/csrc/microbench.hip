// Microbenchmarks that re-derive, on the machine itself, the ceilings the eviction path is
// measured against: streaming HBM copy and read bandwidth, how much a re-read issued by the
// next launch gains from the caches, the bf16 MFMA rate, the v_exp_f32 and plain fp32 VALU
// rates, and the shader clock under load.  Measurement only:
// nothing here is part of the eviction path.  The caller allocates every buffer and times
// the launches with its own events on `stream`; every kernel stays inside the sizes it is
// given and every loop has a fixed trip count.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

__global__ __launch_bounds__(256) void k_copy(const uint4* __restrict__ src, uint4* __restrict__ dst, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256) dst[i] = src[i];
}

__global__ __launch_bounds__(256) void k_read(const uint4* __restrict__ src, int64_t n, uint32_t* sink) {
  uint32_t acc = 0;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256) {
    const uint4 v = src[i];
    acc ^= v.x ^ v.y ^ v.z ^ v.w;
  }
  if (acc == 0x9E3779B9u) sink[0] = acc;  // keeps the loads; practically never stored
}

// Eight independent chains per lane so the issue rate, not the latency, is measured.
__global__ __launch_bounds__(256) void k_exp(float* out, int iters) {
  float x[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) x[j] = threadIdx.x * 1e-3f + 0.1f * j;
  for (int i = 0; i < iters; ++i)
#pragma unroll
    for (int j = 0; j < 8; ++j) x[j] = __builtin_amdgcn_exp2f(x[j]);
  float s = 0.f;
#pragma unroll
  for (int j = 0; j < 8; ++j) s += x[j];
  out[(int64_t)blockIdx.x * 256 + threadIdx.x] = s;
}

__global__ __launch_bounds__(256) void k_fma(float* out, int iters) {
  float x[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) x[j] = threadIdx.x * 1e-3f + 0.1f * j;
  for (int i = 0; i < iters; ++i)
#pragma unroll
    for (int j = 0; j < 8; ++j) x[j] = fmaf(x[j], 0.999f, 0.001f);
  float s = 0.f;
#pragma unroll
  for (int j = 0; j < 8; ++j) s += x[j];
  out[(int64_t)blockIdx.x * 256 + threadIdx.x] = s;
}

// Four independent accumulator chains of v_mfma_f32_32x32x16_bf16 per wave; also reports
// the shader cycles and the 100 MHz real-time ticks each wave spent, for the clock.
__global__ __launch_bounds__(256) void k_mfma(float* out, uint64_t* cycles, int iters) {
  bf16x8 a, b;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    a[i] = (__bf16)(threadIdx.x * 0.001f + i);
    b[i] = (__bf16)(i * 0.5f);
  }
  f32x16 c0 = {}, c1 = {}, c2 = {}, c3 = {};
  const uint64_t t0 = __builtin_readcyclecounter();
  const uint64_t r0 = __builtin_amdgcn_s_memrealtime();
  for (int i = 0; i < iters; ++i) {
    c0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c0, 0, 0, 0);
    c1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c1, 0, 0, 0);
    c2 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c2, 0, 0, 0);
    c3 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c3, 0, 0, 0);
  }
  const uint64_t t1 = __builtin_readcyclecounter();
  const uint64_t r1 = __builtin_amdgcn_s_memrealtime();
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < 16; ++i) s += c0[i] + c1[i] + c2[i] + c3[i];
  out[(int64_t)blockIdx.x * 256 + threadIdx.x] = s;
  if ((threadIdx.x & 63) == 0) {
    const int64_t w = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    cycles[2 * w] = t1 - t0;
    cycles[2 * w + 1] = r1 - r0;
  }
}

}  // namespace

extern "C" {

// src, dst: device, >= n16 * 16 bytes each.  grid: workgroups of 256 threads.
int mb_copy(const void* src, void* dst, int64_t n16, int grid, void* stream) {
  hipLaunchKernelGGL(k_copy, dim3(grid), dim3(256), 0, (hipStream_t)stream, (const uint4*)src, (uint4*)dst, n16);
  return (int)hipGetLastError();
}

// sink: device, >= 4 bytes.
int mb_read(const void* src, int64_t n16, void* sink, int grid, void* stream) {
  hipLaunchKernelGGL(k_read, dim3(grid), dim3(256), 0, (hipStream_t)stream, (const uint4*)src, n16, (uint32_t*)sink);
  return (int)hipGetLastError();
}

// Two read passes over `bytes` of src, either whole (chunk_bytes >= bytes: the buffer, then the
// buffer again) or chunk by chunk (each chunk of chunk_bytes read, then read again at once, the
// next chunk after that): whether a chunk read again by the next launch comes from a cache.
// src: device, >= bytes (a multiple of 16); the last chunk is clipped to the buffer.
int mb_two_pass(const void* src, int64_t bytes, int64_t chunk_bytes, void* sink, int grid, void* stream) {
  if (chunk_bytes > bytes) chunk_bytes = bytes;
  for (int64_t off = 0; off < bytes; off += chunk_bytes) {
    const int64_t len = chunk_bytes < bytes - off ? chunk_bytes : bytes - off;
    const uint4* p = (const uint4*)((const char*)src + off);
    for (int r = 0; r < 2; ++r)
      hipLaunchKernelGGL(k_read, dim3(grid), dim3(256), 0, (hipStream_t)stream, p, len / 16, (uint32_t*)sink);
  }
  return (int)hipGetLastError();
}

// out: device fp32, >= blocks * 256 elements.  Work: blocks * 256 * iters * 8 exp2.
int mb_exp(float* out, int blocks, int iters, void* stream) {
  hipLaunchKernelGGL(k_exp, dim3(blocks), dim3(256), 0, (hipStream_t)stream, out, iters);
  return (int)hipGetLastError();
}

// Same shape as mb_exp with fma: blocks * 256 * iters * 8 fused multiply-adds.
int mb_fma(float* out, int blocks, int iters, void* stream) {
  hipLaunchKernelGGL(k_fma, dim3(blocks), dim3(256), 0, (hipStream_t)stream, out, iters);
  return (int)hipGetLastError();
}

// out: device fp32, >= blocks * 256; cycles: device, >= blocks * 4 * 2 uint64 (per wave:
// shader cycles, real-time ticks).  Work: blocks * 4 waves * iters * 4 MFMAs of 32768 flop.
int mb_mfma(float* out, uint64_t* cycles, int blocks, int iters, void* stream) {
  hipLaunchKernelGGL(k_mfma, dim3(blocks), dim3(256), 0, (hipStream_t)stream, out, cycles, iters);
  return (int)hipGetLastError();
}

}  // extern "C"
