/*
 * Device evaluation of the seeded input generator defined in synth_core.h, so
 * full-size inputs (tens of GB) are drawn in HBM directly.  Built with
 * -ffp-contract=off; the values equal the host build's bit for bit.
 */
#include <hip/hip_runtime.h>
#include <stdint.h>
#include "synth_core.h"

__global__ void syn_fill_kernel(uint16_t* __restrict__ dst, syn_spec sp, int64_t seq, int64_t H,
                                int64_t ntot, int64_t off, int64_t n, int64_t d) {
  const int64_t lh = blockIdx.y;
  const int64_t l = lh / H, h = lh % H;
  const uint64_t key = syn_key(sp.seed, (uint64_t)sp.tag, (uint64_t)seq, (uint64_t)l, (uint64_t)h);
  const int64_t total = n * d;
  uint16_t* base = dst + (lh * ntot + off) * d;
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total;
       e += (int64_t)gridDim.x * blockDim.x) {
    const int64_t t = e / d, c = e - t * d;
    const double f = syn_token_factor(&sp, (uint64_t)seq, (uint64_t)l, (uint64_t)h, (uint64_t)n, (uint64_t)t);
    base[e] = syn_element(key, sp.dist, (uint64_t)t, (uint64_t)d, (uint64_t)c, f);
  }
}

/* Device counterpart of syn_host_fill: dst is a device [L][H][ntot][d] bf16 tensor.
   Returns 0 on success, the hipError_t value otherwise. */
extern "C" int syn_dev_fill(void* dst, const syn_spec* sp, int64_t seq, int64_t L, int64_t H,
                            int64_t ntot, int64_t off, int64_t n, int64_t d, void* stream) {
  if (n <= 0 || L <= 0 || H <= 0) return 0;
  if (off < 0 || off + n > ntot || d <= 0) return (int)hipErrorInvalidValue;
  const int64_t total = n * d;
  int64_t blocks = (total + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  dim3 grid((unsigned)blocks, (unsigned)(L * H));
  hipLaunchKernelGGL(syn_fill_kernel, grid, dim3(256), 0, (hipStream_t)stream, (uint16_t*)dst, *sp,
                     seq, H, ntot, off, n, d);
  return (int)hipGetLastError();
}
