// Mean squared error and its gradient with a fixed-order (deterministic)
// two-stage reduction.
#include <algorithm>

#include "kernels.h"

namespace orbit {
namespace {

constexpr int kMseBlocks = 1024;

__global__ void __launch_bounds__(256) mse_partial(const float* __restrict__ pred, const float* __restrict__ tgt,
                                                   int64_t n, float gscale, float* __restrict__ dpred,
                                                   float* __restrict__ part) {
  __shared__ float red[4];
  float s = 0.f;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256) {
    const float r = pred[i] - tgt[i];
    s += r * r;
    if (dpred) dpred[i] = r * gscale;
  }
  s = wave_sum(s);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = s;
  __syncthreads();
  if (threadIdx.x == 0) part[blockIdx.x] = (red[0] + red[1]) + (red[2] + red[3]);
}

__global__ void __launch_bounds__(256) mse_final(const float* __restrict__ part, int nparts, double inv_n,
                                                 float* loss) {
  __shared__ double red[256];
  double s = 0.0;
  for (int i = threadIdx.x; i < nparts; i += 256) s += part[i];
  red[threadIdx.x] = s;
  __syncthreads();
  for (int o = 128; o >= 1; o >>= 1) {
    if ((int)threadIdx.x < o) red[threadIdx.x] += red[threadIdx.x + o];
    __syncthreads();
  }
  if (threadIdx.x == 0) loss[0] = (float)(red[0] * inv_n);
}

// Latitude-weighted squared error on predictions in token layout [T, out]
// (the training loss of Sec. IV), one block per token. Element c of token t
// lies on grid row y = (l / Wp) * 4 + (c % 16) / 4 (l = t % L; 4x4 patches,
// pixel index v*16 + i*4 + j). Its weight is cos(latitude) over the mean of
// cos over the H rows: with cell centres at -pi/2 + (y + 1/2) pi / H,
// cos(lat_y) = sin((y + 1/2) pi / H), whose sum over the rows is
// 1 / sin(pi / (2H)), so w_y = H sin(pi / (2H)) sin((y + 1/2) pi / H).
__global__ void __launch_bounds__(256) wmse_partial(const float* __restrict__ pred, const float* __restrict__ tgt,
                                                    int L, int Wp, int H, int out, float gscale,
                                                    float* __restrict__ dpred, float* __restrict__ part) {
  __shared__ float red[4];
  constexpr float kPi = 3.14159265358979f;
  const int t = blockIdx.x;
  const int y0 = ((t % L) / Wp) * 4;
  const float norm = (float)H * sinf(kPi / (2.f * (float)H));
  float w[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) w[i] = norm * sinf(((float)(y0 + i) + 0.5f) * (kPi / (float)H));
  const float* p = pred + (int64_t)t * out;
  const float* q = tgt + (int64_t)t * out;
  float* d = dpred ? dpred + (int64_t)t * out : nullptr;
  float s = 0.f;
  for (int c = threadIdx.x; c < out; c += 256) {
    const int ir = (c >> 2) & 3;
    const float wc = ir == 0 ? w[0] : ir == 1 ? w[1] : ir == 2 ? w[2] : w[3];
    const float r = p[c] - q[c];
    s += wc * r * r;
    if (d) d[c] = wc * r * gscale;
  }
  s = wave_sum(s);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = s;
  __syncthreads();
  if (threadIdx.x == 0) part[t] = (red[0] + red[1]) + (red[2] + red[3]);
}

}  // namespace

size_t wmse_workspace_bytes(int64_t tokens) { return align_up((size_t)tokens * sizeof(float)); }

orbit_status wmse(const float* pred, const float* tgt, int B, int L, int Wp, int H, int out, float scale,
                  float* loss, float* dpred, void* ws, hipStream_t s) {
  const int64_t T = (int64_t)B * L;
  const double n = (double)T * out;
  float* part = static_cast<float*>(ws);
  KernelInfo kp{"wmse_partial", 4.0 * n, (dpred ? 12.0 : 8.0) * n};
  ORBIT_TRY(launch(kp, wmse_partial, dim3((unsigned)T), dim3(256), 0, s, pred, tgt, L, Wp, H, out,
                   (float)(2.0 / n * scale), dpred, part));
  KernelInfo kf{"mse_final", 0.0, 4.0 * T};
  return launch(kf, mse_final, dim3(1), dim3(256), 0, s, (const float*)part, (int)T, 1.0 / n, loss);
}

size_t mse_workspace_bytes(int64_t n) {
  (void)n;
  return align_up(kMseBlocks * sizeof(float));
}

orbit_status mse(const float* pred, const float* tgt, int64_t n, float scale, float* loss, float* dpred, void* ws,
                 hipStream_t s) {
  const int blocks = (int)std::max<int64_t>(1, std::min<int64_t>(kMseBlocks, cdiv(n, 256)));
  float* part = static_cast<float*>(ws);
  KernelInfo kp{"mse_partial", 3.0 * n, (dpred ? 12.0 : 8.0) * n};
  ORBIT_TRY(launch(kp, mse_partial, dim3(blocks), dim3(256), 0, s, pred, tgt, n,
                   (float)(2.0 / (double)n * scale), dpred, part));
  KernelInfo kf{"mse_final", 0.0, 4.0 * blocks};
  return launch(kf, mse_final, dim3(1), dim3(256), 0, s, (const float*)part, blocks, 1.0 / (double)n, loss);
}

}  // namespace orbit
