// Matrix-core throughput probe: a measurement aid, not a step of the model.
// Each wave keeps eight independent bf16 32x32x16 products in flight for
// `iters` rounds, the issue pattern that reaches the matrix cores' peak (an
// accumulator is reused only every eighth product, well past the product's
// latency). Every operand element is bf16(x), so each accumulator element
// ends at 16 x^2 iters, which the caller can check exactly.
#include "kernels.h"

namespace orbit {
namespace {

constexpr int kProbeChains = 8;

__global__ void __launch_bounds__(256) mfma_probe_kernel(int iters, float x, float* __restrict__ out) {
  bf16x8 a;
#pragma unroll
  for (int i = 0; i < 8; ++i) a[i] = (bf16)x;
  f32x16 acc[kProbeChains];
#pragma unroll
  for (int c = 0; c < kProbeChains; ++c)
#pragma unroll
    for (int v = 0; v < 16; ++v) acc[c][v] = 0.f;
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int c = 0; c < kProbeChains; ++c) acc[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, a, acc[c], 0, 0, 0);
  }
  float s = 0.f;
#pragma unroll
  for (int c = 0; c < kProbeChains; ++c) s += acc[c][0];
  if ((threadIdx.x & 63) == 0) out[(int64_t)blockIdx.x * 4 + (threadIdx.x >> 6)] = s;
}

}  // namespace

double mfma_probe_flops(int blocks, int iters) { return (double)blocks * 4 * iters * kProbeChains * 32.0 * 32 * 16 * 2; }

orbit_status mfma_probe(int blocks, int iters, float x, float* out, hipStream_t s) {
  KernelInfo ki{"mfma_probe", mfma_probe_flops(blocks, iters), 0.0};
  return launch(ki, mfma_probe_kernel, dim3((unsigned)blocks), dim3(256), 0, s, iters, x, out);
}

}  // namespace orbit
