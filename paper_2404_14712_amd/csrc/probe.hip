// Matrix-core throughput probe: a measurement aid, not a step of the model.
// Each wave keeps eight independent bf16 32x32x16 products in flight for
// `iters` rounds, the issue pattern that reaches the matrix cores' peak (an
// accumulator is reused only every eighth product, well past the product's
// latency). Both operands of every product are the lane's fragment: all
// elements bf16(x) (seed 0), or x times a seeded pattern of 8-bit mantissas
// in [-2, 2) (the matrix cores draw more power, and the clock drops, when the
// operand bits vary as in real data). Accumulator element (0, 0) ends at
// iters times the sum of the squares of lanes 0 and 32's fragments.
#include "kernels.h"

namespace orbit {
namespace {

constexpr int kProbeChains = 8;

// the pattern value of fragment element i of lane l: ((h & 255) - 128) / 64
// with h a multiplicative hash of (seed, 8 l + i)
ORBIT_DEV float probe_pattern(unsigned seed, int l, int i) {
  unsigned h = (seed ^ (unsigned)(8 * l + i)) * 0x9E3779B1u;
  h ^= h >> 15;
  h *= 0x85EBCA77u;
  h ^= h >> 13;
  return (float)((int)(h & 255u) - 128) * (1.f / 64.f);
}

__global__ void __launch_bounds__(256) mfma_probe_kernel(int iters, unsigned seed, float x, float* __restrict__ out) {
  const int lane = threadIdx.x & 63;
  bf16x8 a;
#pragma unroll
  for (int i = 0; i < 8; ++i) a[i] = (bf16)(seed ? x * probe_pattern(seed, lane, i) : x);
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
  if (lane == 0) out[(int64_t)blockIdx.x * 4 + (threadIdx.x >> 6)] = s;
}

}  // namespace

double mfma_probe_flops(int blocks, int iters) { return (double)blocks * 4 * iters * kProbeChains * 32.0 * 32 * 16 * 2; }

orbit_status mfma_probe(int blocks, int iters, unsigned seed, float x, float* out, hipStream_t s) {
  KernelInfo ki{"mfma_probe", mfma_probe_flops(blocks, iters), 0.0};
  return launch(ki, mfma_probe_kernel, dim3((unsigned)blocks), dim3(256), 0, s, iters, seed, x, out);
}

}  // namespace orbit
