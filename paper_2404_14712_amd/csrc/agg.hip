// Cross-attention variable aggregation (one learned query over the V variable
// tokens of each patch), forward and backward, in the exact refolded form:
//
//   score_{t,h,v} = q_h . (W_k^h x_{t,v} + b_k^h) / sqrt(dh)
//                 = x_{t,v} . u_h / sqrt(dh) + const_h,   u_h = W_k^h q_h
//   (the constant is the same for every v and drops out of the softmax), and
//   zh_{t,h} = sum_v a_{t,h,v} (W_v^h x_{t,v} + b_v^h) = W_v^h xbar_{t,h} + b_v^h
//   with xbar_{t,h} = sum_v a_{t,h,v} x_{t,v}  (the weights sum to one).
//
// So the per-token key/value projections (2 T V d A flops) are never formed:
// the token tensor is streamed twice through skinny MFMA products (scores,
// xbar), and only xbar [T, H, d] meets W_v. The backward mirrors it.
#include <algorithm>

#include "agg.h"
#include "gemm.h"
#include "kernels.h"
#include "tile.h"

namespace orbit {
namespace {

// 8 consecutive elements (16-byte aligned) widened to float
ORBIT_DEV void agg_ld8(const bf16* p, float* f) {
  const bf16x8 v = *reinterpret_cast<const bf16x8*>(p);
#pragma unroll
  for (int u = 0; u < 8; ++u) f[u] = (float)v[u];
}
ORBIT_DEV void agg_ld8(const float* p, float* f) {
  const f32x4 a = *reinterpret_cast<const f32x4*>(p), b = *reinterpret_cast<const f32x4*>(p + 4);
#pragma unroll
  for (int u = 0; u < 4; ++u) { f[u] = a[u]; f[4 + u] = b[u]; }
}

// Weighted column sums out[j] = sum_i c_ij W[i][j] over the d rows of a [d, A]
// weight, with c_ij = x[i] (query projection) or dU[i][j / dh] (query
// gradient). Phase 1: one block per slice of kGvRows rows; a thread takes 8
// consecutive columns (16-byte row reads). When a row has fewer than 2048
// columns the block's threads form several row groups that take alternate
// rows of the slice and add their sums through LDS in a fixed order; one
// float32 partial per (slice, column). Phase 2 sums the slices in order
// (deterministic).
constexpr int kGvRows = 64;

template <typename T, bool DQ>
__global__ void __launch_bounds__(256) agg_gemv_part(const T* __restrict__ W, const T* __restrict__ x,
                                                     const float* __restrict__ dU, float* __restrict__ part, int d,
                                                     int A, int H, int dh) {
  __shared__ float red[256 * 8];
  const int cg = A / 8;                      // column groups of 8
  const int rg = cg >= 256 ? 1 : 256 / cg;   // row groups
  const int i0 = blockIdx.x * kGvRows, i1 = min(d, i0 + kGvRows);
  const int t = threadIdx.x;
  const int r = rg == 1 ? 0 : t / cg;
  for (int base = 0; base < cg; base += 256) {
    const int g = rg == 1 ? base + t : t % cg;
    const bool act = g < cg && r < rg;
    float acc[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) acc[u] = 0.f;
    if (act) {
      const int j = g * 8, h = j / dh;
      int i = i0 + r;
      // 8 rows' loads in flight at a time
      for (; i + 7 * rg < i1; i += 8 * rg) {
        float w[8][8], c[8];
#pragma unroll
        for (int k = 0; k < 8; ++k) {
          agg_ld8(W + (int64_t)(i + k * rg) * A + j, w[k]);
          c[k] = DQ ? dU[(int64_t)(i + k * rg) * H + h] : to_f(x[i + k * rg]);
        }
#pragma unroll
        for (int k = 0; k < 8; ++k)
#pragma unroll
          for (int u = 0; u < 8; ++u) acc[u] += c[k] * w[k][u];
      }
      for (; i < i1; i += rg) {
        float w[8];
        agg_ld8(W + (int64_t)i * A + j, w);
        const float c = DQ ? dU[(int64_t)i * H + h] : to_f(x[i]);
#pragma unroll
        for (int u = 0; u < 8; ++u) acc[u] += c * w[u];
      }
    }
    if (rg > 1) {
      // one pass only (cg < 256): row groups 1.. hand their sums to group 0
      if (act && r > 0)
#pragma unroll
        for (int u = 0; u < 8; ++u) red[(r * cg + g) * 8 + u] = acc[u];
      __syncthreads();
      if (act && r == 0)
        for (int rr = 1; rr < rg; ++rr)
#pragma unroll
          for (int u = 0; u < 8; ++u) acc[u] += red[(rr * cg + g) * 8 + u];
    }
    if (act && r == 0) {
      float* o = part + (int64_t)blockIdx.x * A + g * 8;
      *reinterpret_cast<f32x4*>(o) = f32x4{acc[0], acc[1], acc[2], acc[3]};
      *reinterpret_cast<f32x4*>(o + 4) = f32x4{acc[4], acc[5], acc[6], acc[7]};
    }
  }
}

// out[j] = sum over slices of part[slice][j] (+ bias[j]): a block takes 16
// columns; its 16 thread groups sum every 16th slice, and the 16 group sums
// are added in order (deterministic)
template <typename T>
__global__ void __launch_bounds__(256) agg_gemv_final(const float* __restrict__ part, int slices, int A,
                                                      const T* __restrict__ bias, float* __restrict__ out) {
  __shared__ float red[16][17];
  const int c = threadIdx.x & 15, sg = threadIdx.x >> 4;
  const int j = blockIdx.x * 16 + c;
  float s = 0.f;
  if (j < A)
    for (int k = sg; k < slices; k += 16) s += part[(int64_t)k * A + j];
  red[sg][c] = s;
  __syncthreads();
  if (sg == 0 && j < A) {
    float t = 0.f;
    for (int g = 0; g < 16; ++g) t += red[g][c];
    out[j] = bias ? t + to_f(bias[j]) : t;
  }
}

// Ut[h][i] = sum_c w_k[i][h*dh + c] q[h*dh + c]. One wave per row i: each
// lane forms the dot products of 8-column chunks (16-byte reads of the row),
// and lane h adds the dh / 8 chunks of head h in order. A row is taken in
// passes of whole heads, at most kFoldMaxChunks chunks each.
constexpr int kFoldMaxChunks = 1024;
template <typename T>
__global__ void __launch_bounds__(256) agg_fold_key(const T* __restrict__ wk, const float* __restrict__ q,
                                                    T* __restrict__ Ut, int d, int H, int dh) {
  __shared__ float part[4][kFoldMaxChunks];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int i = blockIdx.x * 4 + wave;
  const int per = dh / 8, hp = kFoldMaxChunks / per;  // chunks per head, heads per pass
  const T* row = wk + (int64_t)i * H * dh;
  for (int h0 = 0; h0 < H; h0 += hp) {
    const int nh = min(hp, H - h0), c0 = h0 * per;
    if (i < d) {
      for (int ch = lane; ch < nh * per; ch += 64) {
        float w[8], qq[8];
        agg_ld8(row + (c0 + ch) * 8, w);
        agg_ld8(q + (c0 + ch) * 8, qq);
        float s = 0.f;
#pragma unroll
        for (int u = 0; u < 8; ++u) s += w[u] * qq[u];
        part[wave][ch] = s;
      }
    }
    __syncthreads();
    if (i < d && lane < nh) {
      float s = 0.f;
      for (int k = 0; k < per; ++k) s += part[wave][lane * per + k];
      Ut[(int64_t)(h0 + lane) * d + i] = from_f<T>(s);
    }
    __syncthreads();
  }
}

// softmax over v of S[(t*V + v)*H + h]: a32[t][h][v] (float32) and
// ab[t][h][0..Vp) (dtype, zero padded). One wave per token: the token's V x H
// scores are one contiguous block; lane l takes head l % H and variables
// l / H, l / H + 64 / H, ...; the per-head max and sum combine the lanes of one
// head in a fixed butterfly order. H divides 64.
template <typename T>
__global__ void __launch_bounds__(256) agg_softmax(const float* __restrict__ S, float* __restrict__ a32,
                                                   T* __restrict__ ab, int64_t T_, int V, int Vp, int H) {
  const int lane = threadIdx.x & 63;
  const int64_t t = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= T_) return;
  const int h = lane % H, step = 64 / H;
  const float* st = S + t * V * H;
  float m = -INFINITY;
  for (int v = lane / H; v < V; v += step) m = fmaxf(m, st[v * H + h]);
  for (int o = H; o < 64; o <<= 1) m = fmaxf(m, __shfl_xor(m, o, 64));
  float z = 0.f;
  for (int v = lane / H; v < V; v += step) z += __expf(st[v * H + h] - m);
  for (int o = H; o < 64; o <<= 1) z += __shfl_xor(z, o, 64);
  const float inv = 1.f / z;
  float* ao = a32 + (t * H + h) * V;
  T* bo = ab + (t * H + h) * Vp;
  for (int v = lane / H; v < Vp; v += step) {
    const float p = v < V ? __expf(st[v * H + h] - m) * inv : 0.f;
    if (v < V) ao[v] = p;
    bo[v] = from_f<T>(p);
  }
}

// xbar[t][h][c] = sum_v a[t][h][v] x[t][v][c] (bf16) as one streaming pass over
// the token tensor: a wave per (token, 512 columns), 8 columns per lane read as
// 16-byte row segments (a wave reads 1 KB of a row per load); two variables
// per step, interleaved into bf16 pairs and multiplied by the head's weight
// pair (wave-uniform, a scalar operand) with dot2, float32 accumulation in v
// order. ab is zero-padded to an even count, so an odd last variable pairs
// with a zero weight.
template <int H>
__global__ void __launch_bounds__(256) agg_xbar(const bf16* __restrict__ ab, const bf16* __restrict__ tok,
                                                bf16* __restrict__ xbar, int64_t T_, int V, int Vp, int d) {
  typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
  typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
  const int lane = threadIdx.x & 63;
  const int nch = (d + 511) / 512;
  const int item = __builtin_amdgcn_readfirstlane((int)blockIdx.x * 4 + (int)(threadIdx.x >> 6));
  if ((int64_t)item >= T_ * nch) return;
  const int t = __builtin_amdgcn_readfirstlane(item / nch);
  const int c0 = (item - t * nch) * 512 + lane * 8;
  // the token's V rows as one buffer: loads past the last row read zeros
  const __amdgpu_buffer_rsrc_t rx = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<bf16*>(tok + (int64_t)t * V * d), 0, V * d * 2, 0x00020000);
  const unsigned* A = reinterpret_cast<const unsigned*>(ab + (int64_t)t * H * Vp);
  const int hp = Vp / 2;
  const unsigned voff = (unsigned)c0 * 2;
  const unsigned row = (unsigned)d * 2;
  float acc[H][8];
#pragma unroll
  for (int h = 0; h < H; ++h)
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[h][j] = 0.f;
#pragma unroll 2
  for (int v = 0; v < V; v += 2) {
    // non-temporal loads (cache policy bit 1): the tokens are read once here
    const u32x4 x0 = __builtin_amdgcn_raw_buffer_load_b128(rx, voff, (unsigned)v * row, 2);
    const u32x4 x1 = __builtin_amdgcn_raw_buffer_load_b128(rx, voff, (unsigned)(v + 1) * row, 2);
    unsigned p[8];
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      p[2 * w] = __builtin_amdgcn_perm(x1[w], x0[w], 0x05040100u);
      p[2 * w + 1] = __builtin_amdgcn_perm(x1[w], x0[w], 0x07060302u);
    }
#pragma unroll
    for (int h = 0; h < H; ++h) {
      const bf16x2 a2 = __builtin_bit_cast(bf16x2, A[h * hp + v / 2]);
#pragma unroll
      for (int j = 0; j < 8; ++j)
        acc[h][j] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, p[j]), a2, acc[h][j], false);
    }
  }
  if (c0 >= d) return;
#pragma unroll
  for (int h = 0; h < H; ++h) st128(xbar + ((int64_t)t * H + h) * d + c0, pack(acc[h], (bf16*)nullptr));
}

// Dot products of each token's V rows with H weight rows over the embedding,
// out[t][v][h] = alpha * sum_c w_t[h][c] x[t][v][c] (float32, element
// (t, v, h) at out[t * o_t + v * o_v + h * o_h]): the scores (w = the folded
// query keys u, shared by every token) and their backward (w_t = dxbar of
// token t). A block per token; its four waves take a quarter of the embedding
// each and run 16x16x32 bf16 MFMAs, heads as rows and 16 variables per tile
// as columns; the token rows are loaded straight into MFMA fragments (loads
// past the last variable read zeros; default cache policy, since a load
// covers half of each row's 128-byte line and its partner the other half),
// and the quarters' sums are added in order through LDS.
template <int H, int NT>
__global__ void __launch_bounds__(256) agg_rowdot(const bf16* __restrict__ tok, const bf16* __restrict__ w,
                                                  int64_t w_tstride, float* __restrict__ out, int64_t o_t, int o_v,
                                                  int o_h, float alpha, int V, int d) {
  static_assert(H == 8 || H == 16, "heads");
  typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
  const int t = blockIdx.x;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  // a 64-deep K step: lane group g = lane / 16 holds k = 16 g .. 16 g + 15 of
  // its row (two 16-byte loads; each row's 128 bytes come in one pair), the
  // first half for the step's first product, the second for its second
  const int lr = lane & 15, lk = (lane >> 4) * 16;
  const int q = d / 4, kb = wave * q;
  const __amdgpu_buffer_rsrc_t rx = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<bf16*>(tok + (int64_t)t * V * d), 0, V * d * 2, 0x00020000);
  unsigned vo[NT];
#pragma unroll
  for (int n = 0; n < NT; ++n) vo[n] = (unsigned)((n * 16 + lr) * d + kb + lk) * 2u;
  // heads past H (H = 8) are zero rows of the A fragment: their lanes load
  // row 0 and mask it, so the loop carries no branch
  const unsigned amask = lr < H ? ~0u : 0u;
  const bf16* wp = w + t * w_tstride + (int64_t)(lr < H ? lr : 0) * d + kb + lk;
  f32x4 acc[NT];
#pragma unroll
  for (int n = 0; n < NT; ++n) acc[n] = f32x4{0.f, 0.f, 0.f, 0.f};
  struct Step { u32x4 a[2], b[NT][2]; };
  auto load = [&](Step& f, int k) {
    f.a[0] = *reinterpret_cast<const u32x4*>(wp + k);
    f.a[1] = *reinterpret_cast<const u32x4*>(wp + k + 8);
#pragma unroll
    for (int n = 0; n < NT; ++n) {
      f.b[n][0] = __builtin_amdgcn_raw_buffer_load_b128(rx, vo[n] + (unsigned)k * 2u, 0, 0);
      f.b[n][1] = __builtin_amdgcn_raw_buffer_load_b128(rx, vo[n] + (unsigned)k * 2u + 16u, 0, 0);
    }
  };
  auto mma = [&](const Step& f) {
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const bf16x8 a = __builtin_bit_cast(bf16x8, f.a[u] & amask);
#pragma unroll
      for (int n = 0; n < NT; ++n)
        acc[n] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, __builtin_bit_cast(bf16x8, f.b[n][u]), acc[n], 0, 0, 0);
    }
  };
  // two steps per iteration, the next step's loads in flight during the
  // current step's products. Each token starts its sweep at its own step
  // (and wraps), so the blocks in flight do not all read the same column
  // offsets of their rows at once; the summation order is fixed per token.
  const int S = q / 64, rot = t % S;
  auto kof = [&](int i) { const int j = i + rot; return (j < S ? j : j - S) * 64; };
  Step f0, f1;
  load(f0, kof(0));
  int i = 0;
  for (; i + 1 < S; i += 2) {
    load(f1, kof(i + 1));
    mma(f0);
    if (i + 2 < S) load(f0, kof(i + 2));
    mma(f1);
  }
  if (i < S) mma(f0);
  __shared__ f32x4 part[3][NT][64];
  if (wave > 0) {
#pragma unroll
    for (int n = 0; n < NT; ++n) part[wave - 1][n][lane] = acc[n];
  }
  __syncthreads();
  if (wave != 0) return;
#pragma unroll
  for (int w2 = 0; w2 < 3; ++w2)
#pragma unroll
    for (int n = 0; n < NT; ++n) acc[n] += part[w2][n][lane];
  // lane l holds heads 4 (l / 16) .. + 3 of variable column l % 16
#pragma unroll
  for (int n = 0; n < NT; ++n) {
    const int v = n * 16 + lr;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int h = (lane >> 4) * 4 + r;
      if (h < H && v < V) out[t * o_t + (int64_t)v * o_v + (int64_t)h * o_h] = alpha * acc[n][r];
    }
  }
}

// dxbar[t][h][c] = sum_j dzh[t][h*DH + j] w_v[c][h*DH + j] (bf16): the value
// path's input gradient, a reduction over only head_dim whose output has the
// size of patches x heads x embedding. A block takes head h, 256 columns and
// a range of patch rows, walked in chunks of 32 rows. Each wave keeps its 64
// columns of W_v^h as MFMA fragments for the whole range; a chunk's dzh rows
// (32 x DH) are copied once into LDS (two buffers, one barrier per chunk) and
// read by all four waves; the 32x32x16 products' results go out through a
// per-wave LDS stage as 16-byte row pieces (128 contiguous bytes per row).
template <int DH>
__global__ void __launch_bounds__(256) agg_value_dx(const bf16* __restrict__ dzh, const bf16* __restrict__ wv,
                                                    bf16* __restrict__ dxbar, int T_, int H, int d, int rows) {
  constexpr int KS = DH / 16;
  constexpr int AP = DH + 8;  // LDS row pitch of the dzh chunk (elements)
  __shared__ __attribute__((aligned(16))) bf16 abuf[2][32 * AP];
  __shared__ __attribute__((aligned(16))) float stage[4][32][68];
  const int A = H * DH;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int lr = lane & 31, lg = lane >> 5;
  const int h = blockIdx.y;
  const int c0 = blockIdx.x * 256 + wave * 64;
  // the wave's 64 columns of W_v^h: two 32-column fragments per 16-deep step
  bf16x8 bf[2][KS];
#pragma unroll
  for (int n = 0; n < 2; ++n) {
    const bf16* wrow = wv + (int64_t)(c0 + n * 32 + lr) * A + h * DH + 8 * lg;
#pragma unroll
    for (int kk = 0; kk < KS; ++kk) bf[n][kk] = *reinterpret_cast<const bf16x8*>(wrow + 16 * kk);
  }
  const int tbeg = blockIdx.z * rows, tend = min(T_, tbeg + rows);
  // chunk copy: 32 rows x DH / 8 pieces of 16 bytes over 256 threads, loaded
  // into registers at the top of an iteration and written to LDS at its end
  constexpr int PIECES = 32 * DH / 8, PPT = PIECES / 256;
  static_assert(PIECES % 256 == 0, "whole pieces per thread");
  bf16x8 pre[PPT];
  auto load = [&](int t0) {
#pragma unroll
    for (int i = 0; i < PPT; ++i) {
      const int pc = tid + i * 256, r = pc / (DH / 8), cc = (pc % (DH / 8)) * 8;
      const int t = min(t0 + r, T_ - 1);  // rows past the last patch repeat it (never stored)
      pre[i] = *reinterpret_cast<const bf16x8*>(dzh + (int64_t)t * A + h * DH + cc);
    }
  };
  auto store = [&](bf16* dst) {
#pragma unroll
    for (int i = 0; i < PPT; ++i) {
      const int pc = tid + i * 256, r = pc / (DH / 8), cc = (pc % (DH / 8)) * 8;
      *reinterpret_cast<bf16x8*>(dst + r * AP + cc) = pre[i];
    }
  };
  if (tbeg < tend) {
    load(tbeg);
    store(abuf[0]);
  }
  __syncthreads();
  int cur = 0;
  for (int t0 = tbeg; t0 < tend; t0 += 32, cur ^= 1) {
    const bool more = t0 + 32 < tend;
    if (more) load(t0 + 32);
    const bf16* as = abuf[cur] + lr * AP + 8 * lg;
    f32x16 acc[2];
#pragma unroll
    for (int n = 0; n < 2; ++n)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[n][v] = 0.f;
#pragma unroll
    for (int kk = 0; kk < KS; ++kk) {
      const bf16x8 af = *reinterpret_cast<const bf16x8*>(as + 16 * kk);
#pragma unroll
      for (int n = 0; n < 2; ++n) acc[n] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af, bf[n][kk], acc[n], 0, 0, 0);
    }
    // acc[n][v]: chunk row 8 (v / 4) + 4 lg + v % 4, column 32 n + lr
#pragma unroll
    for (int n = 0; n < 2; ++n)
#pragma unroll
      for (int v = 0; v < 16; ++v) stage[wave][(v >> 2) * 8 + lg * 4 + (v & 3)][n * 32 + lr] = acc[n][v];
    __builtin_amdgcn_wave_barrier();
    // 8 lanes per row, 8 columns each: 8 rows per pass
#pragma unroll
    for (int it = 0; it < 4; ++it) {
      const int rl = it * 8 + (lane >> 3), cl = (lane & 7) * 8;
      const int t = t0 + rl;
      const f32x4 lo = *reinterpret_cast<const f32x4*>(&stage[wave][rl][cl]);
      const f32x4 hi = *reinterpret_cast<const f32x4*>(&stage[wave][rl][cl + 4]);
      float o[8] = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
      if (t < tend) st128(dxbar + ((int64_t)t * H + h) * d + c0 + cl, pack(o, (bf16*)nullptr));
    }
    if (more) store(abuf[cur ^ 1]);
    // the next chunk's rows are in LDS, and every wave is done with this one
    __syncthreads();
  }
}

// softmax backward per (t, h): ds = a (da - sum a da) * scale.
// ac[(t*V + v)*2H + h] = a, ac[(t*V + v)*2H + H + h] = ds   (dtype); one wave per
// token, lanes as in agg_softmax
template <typename T>
__global__ void __launch_bounds__(256) agg_softmax_bwd(const float* __restrict__ a32, const float* __restrict__ da,
                                                       T* __restrict__ ac, int64_t T_, int V, int H, float scale) {
  const int lane = threadIdx.x & 63;
  const int64_t t = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= T_) return;
  const int h = lane % H, step = 64 / H;
  const float* a = a32 + (t * H + h) * V;
  const float* g = da + (t * H + h) * V;
  float dot = 0.f;
  for (int v = lane / H; v < V; v += step) dot += a[v] * g[v];
  for (int o = H; o < 64; o <<= 1) dot += __shfl_xor(dot, o, 64);
  T* o = ac + t * V * 2 * H;
  for (int v = lane / H; v < V; v += step) {
    const float av = a[v];
    o[(int64_t)v * 2 * H + h] = from_f<T>(av);
    o[(int64_t)v * 2 * H + H + h] = from_f<T>(av * (g[v] - dot) * scale);
  }
}

// dW_k[i][j] = dU[i][h(j)] q[j];  dW_q[i][j] = q0[i] dq[j]
// (4 consecutive columns per thread, 16-byte accesses)
template <typename T>
__global__ void __launch_bounds__(256) agg_outer(const float* __restrict__ dU, const float* __restrict__ q,
                                                 const T* __restrict__ q0, const float* __restrict__ dq,
                                                 float* __restrict__ dwk, float* __restrict__ dwq, int d, int H,
                                                 int dh, int accumulate) {
  const int A = H * dh, c4 = A / 4;
  const int64_t total = (int64_t)d * c4;
  for (int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x; e < total; e += (int64_t)gridDim.x * 256) {
    const int i = (int)(e / c4), j = (int)(e % c4) * 4;
    const float u = dU[(int64_t)i * H + j / dh], q0i = to_f(q0[i]);
    const f32x4 qv = *reinterpret_cast<const f32x4*>(q + j), dqv = *reinterpret_cast<const f32x4*>(dq + j);
    f32x4* pk = reinterpret_cast<f32x4*>(dwk + (int64_t)i * A + j);
    f32x4* pq = reinterpret_cast<f32x4*>(dwq + (int64_t)i * A + j);
    f32x4 vk, vq;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      vk[k] = u * qv[k];
      vq[k] = q0i * dqv[k];
    }
    if (accumulate) {
      const f32x4 ok = *pk, oq = *pq;
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        vk[k] = ok[k] + vk[k];
        vq[k] = oq[k] + vq[k];
      }
    }
    *pk = vk;
    *pq = vq;
  }
}

// dq0[i] = sum_j w_q[i][j] dq[j]; db_q = dq; db_k = 0 (one wave per row i,
// 8 columns per lane at a time)
template <typename T>
__global__ void __launch_bounds__(256) agg_query_bwd(const T* __restrict__ wq, const float* __restrict__ dq,
                                                     float* dq0, float* dbq, float* dbk, int d, int A,
                                                     int accumulate) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int i = blockIdx.x * 4 + wave;
  if (i < d) {
    const T* row = wq + (int64_t)i * A;
    float s = 0.f;
    for (int ch = lane; ch < A / 8; ch += 64) {
      float w[8], g[8];
      agg_ld8(row + ch * 8, w);
      agg_ld8(dq + ch * 8, g);
#pragma unroll
      for (int u = 0; u < 8; ++u) s += w[u] * g[u];
    }
    s = wave_sum(s);
    if (lane == 0) dq0[i] = accumulate ? dq0[i] + s : s;
  }
  if (blockIdx.x == 0) {
    for (int j = threadIdx.x; j < A; j += 256) {
      dbq[j] = accumulate ? dbq[j] + dq[j] : dq[j];
      if (!accumulate) dbk[j] = 0.f;
    }
  }
}

// dtok_t [V, d] = [a^T | ds] [V, 2H] . [dxbar_t ; U^T] [2H, d] for bf16, one
// block per (token, 512 columns): the 2H x 512 right-hand slab is staged in LDS
// as stored (rows contiguous) and read through transposing LDS reads; the
// left-hand rows (2H contiguous values per variable) are MFMA fragments read
// straight from HBM. MT = ceil(V / 32) row tiles, KS = 2H / 16 K-steps. Each
// wave produces 64 columns at a time and writes them, rounded to bf16, through
// a private LDS area, so that every lane stores 16 contiguous bytes (a wave
// covers 8 rows x 128 bytes per store).
constexpr int kDtokCols = 512;
template <int MT, int KS>
__global__ void __launch_bounds__(256) agg_dtok(const bf16* __restrict__ ac, const bf16* __restrict__ dxbar,
                                                const bf16* __restrict__ Ut, bf16* __restrict__ dtok, int V, int d,
                                                int H) {
  using Stage = GemmStageMN<kDtokCols, 16 * KS, 256>;
  constexpr int P = Stage::PITCH;
  constexpr int EP = 64 + 8;  // staging pitch (bf16; results are rounded before staging)
  __shared__ __attribute__((aligned(16))) bf16 Bs[16 * KS * P];
  __shared__ __attribute__((aligned(16))) bf16 ew_all[4][32 * EP];
  const int tid = threadIdx.x, lane = tid & 63, g = lane >> 5, wave = tid >> 6;
  const int64_t t = blockIdx.y;
  const int c0 = blockIdx.x * kDtokCols;
  // stage rows k < H from dxbar_t, rows k >= H from U^T (zero past column d)
  constexpr int RC = kDtokCols / 8;
  for (int c = tid; c < 16 * KS * RC; c += 256) {
    const int k = c / RC, cc = c % RC;
    const int col = c0 + cc * 8;
    U128 v = zero128();
    if (col < d) v = ld128(k < H ? dxbar + (t * H + k) * d + col : Ut + (int64_t)(k - H) * d + col);
    st128(Bs + k * P + cc * 8, v);
  }
  Frag<bf16> af[MT][KS];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    const int v = mt * 32 + (lane & 31);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      if (v < V) ld_frag(af[mt][ks], ac + (t * V + v) * (2 * H) + ks * 16 + g * 8);
      else {
        float z[8] = {0, 0, 0, 0, 0, 0, 0, 0};
        frag_from(af[mt][ks], z);
      }
    }
  }
  __syncthreads();
  bf16* out = dtok + t * V * d;
  bf16* ew = ew_all[wave];
#pragma unroll 1
  for (int j = 0; j < kDtokCols / 256; ++j) {
    const int n0 = wave * (kDtokCols / 4) + j * 64;
    f32x16 acc[MT][2];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int i = 0; i < 16; ++i) acc[mt][h][i] = 0.f;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        Frag<bf16> bfr;
        Stage::frag(bfr, Bs, n0 + h * 32, ks, lane);
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) mma16(acc[mt][h], af[mt][ks], bfr);
      }
    }
    const int cl = (lane & 7) * 8;  // read-back: 8 lanes per row, 8 rows per pass
    const int col = c0 + n0 + cl;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
#pragma unroll
      for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int i = 0; i < 16; ++i)
          ew[((i >> 2) * 8 + g * 4 + (i & 3)) * EP + h * 32 + (lane & 31)] = (bf16)acc[mt][h][i];
      __builtin_amdgcn_wave_barrier();
#pragma unroll
      for (int pass = 0; pass < 4; ++pass) {
        const int r = pass * 8 + (lane >> 3);
        const int v = mt * 32 + r;
        const bf16x8 o = *reinterpret_cast<const bf16x8*>(ew + r * EP + cl);
        if (v < V && col < d) *reinterpret_cast<bf16x8*>(out + (int64_t)v * d + col) = o;
      }
      __builtin_amdgcn_wave_barrier();
    }
  }
}

unsigned g1(int64_t n) { return (unsigned)std::max<int64_t>(1, cdiv(n, 256)); }

// out = (weighted column sums of W, see agg_gemv_part) + bias; part holds
// cdiv(d, kGvRows) x A floats
template <typename T, bool DQ>
orbit_status gemv_cols(const char* name, const void* W, const void* x, const float* dU, const void* bias, float* out,
                       float* part, int d, int A, int H, int dh, hipStream_t s) {
  const int slices = (int)cdiv(d, kGvRows);
  KernelInfo k1{name, 2.0 * d * A, (double)d * A * sizeof(T)};
  ORBIT_TRY(launch(k1, agg_gemv_part<T, DQ>, dim3((unsigned)slices), dim3(256), 0, s, static_cast<const T*>(W),
                   static_cast<const T*>(x), dU, part, d, A, H, dh));
  KernelInfo k2{"agg_gemv_final", 0.0, (double)slices * A * 4};
  return launch(k2, agg_gemv_final<T>, dim3((unsigned)cdiv(A, 16)), dim3(256), 0, s, (const float*)part, slices, A,
                static_cast<const T*>(bias), out);
}
size_t gemv_part_bytes(int d, int A) { return (size_t)cdiv(d, kGvRows) * A * sizeof(float); }

struct Sizes {
  int64_t T;
  int V, Vp, d, H, dh, A, L, B;
};
Sizes sizes(const orbit_agg_desc& a) {
  Sizes s;
  s.B = a.B; s.L = a.L; s.T = (int64_t)a.B * a.L; s.V = a.V; s.Vp = (a.V + 7) / 8 * 8;
  s.d = a.d; s.H = a.heads; s.dh = a.head_dim; s.A = a.heads * a.head_dim;
  return s;
}
size_t esz(orbit_dtype dt) { return dt == ORBIT_BF16 ? 2 : 4; }

// saved layout: q f32 [A] | Ut [H, d] | a32 [T, H, V] | xbar [T, H, d] | zh [T, A]
struct Saved {
  float* q; void* Ut; float* a32; void* xbar; void* zh;
};
Saved carve_saved(const Sizes& z, orbit_dtype dt, void* base, size_t* used) {
  Carver c(base);
  Saved s;
  s.q = c.take<float>(z.A);
  s.Ut = c.take<char>((size_t)z.H * z.d * esz(dt));
  s.a32 = c.take<float>((size_t)z.T * z.H * z.V);
  s.xbar = c.take<char>((size_t)z.T * z.H * z.d * esz(dt));
  s.zh = c.take<char>((size_t)z.T * z.A * esz(dt));
  if (used) *used = c.used();
  return s;
}

Gemm base_gemm(orbit_dtype dt) {
  Gemm g;
  g.dtype = dt;
  return g;
}

// agg_rowdot's domain: bf16, 8 or 16 heads, at most 96 variables, an
// embedding of whole 256-column quarters and 16-byte aligned rows
bool rowdot_ok(orbit_dtype dt, const Sizes& z, const void* tok, const void* w) {
  return dt == ORBIT_BF16 && (z.H == 8 || z.H == 16) && z.V <= 96 && z.d % 256 == 0 &&
         (int64_t)z.V * z.d * 2 < ((int64_t)1 << 31) && (reinterpret_cast<uintptr_t>(tok) & 15) == 0 &&
         (reinterpret_cast<uintptr_t>(w) & 15) == 0;
}

// out[t * o_t + v * o_v + h * o_h] = alpha * x_{t,v} . w_{t,h} over all tokens
orbit_status rowdot(const char* name, const Sizes& z, const void* tok, const void* w, int64_t w_tstride, float* out,
                    int64_t o_t, int o_v, int o_h, float alpha, hipStream_t s) {
  const int nt = (int)cdiv(z.V, 16);
  KernelInfo k{name, 2.0 * z.T * z.V * (double)z.H * z.d,
               (double)z.T * z.V * z.d * 2.0 + (w_tstride ? (double)z.T * z.H * z.d * 2.0 : 0.0) +
                   4.0 * z.T * z.V * z.H};
  const dim3 grid((unsigned)z.T);
  const bf16* tp = static_cast<const bf16*>(tok);
  const bf16* wp = static_cast<const bf16*>(w);
#define RD(HH, N) \
  if (z.H == HH && nt == N) \
  return launch(k, agg_rowdot<HH, N>, grid, dim3(256), 0, s, tp, wp, w_tstride, out, o_t, o_v, o_h, \
                alpha, z.V, z.d)
  RD(8, 1); RD(8, 2); RD(8, 3); RD(8, 4); RD(8, 5); RD(8, 6);
  RD(16, 1); RD(16, 2); RD(16, 3); RD(16, 4); RD(16, 5); RD(16, 6);
#undef RD
  set_error("%s: %d heads x %d variables outside the row-dot kernel's range", name, z.H, z.V);
  return ORBIT_E_UNSUPPORTED;
}

}  // namespace

size_t agg_saved_bytes(const orbit_agg_desc& a) {
  size_t u = 0;
  carve_saved(sizes(a), (orbit_dtype)a.dtype, nullptr, &u);
  return u;
}

// forward workspace: S f32 [T*V, H] | ab [T, H, Vp] | query partials | gemm split-K
// backward workspace: dzh [T, A] | dxbar [T, H, d] | da f32 [T, H, V] | ac [T*V, 2H] | dU f32 [d, H]
//                     | dq f32 [A] | query-gradient partials | colsum | gemm split-K
static size_t gemm_ws_max(const Sizes& z, orbit_dtype dt) {
  // split-K partials of every product of the forward and backward passes
  const int T = (int)z.T, TV = (int)(z.T * z.V);
  const int sh[][6] = {
      // M, N, K, A K-major, B K-major, batch
      {TV, z.H, z.d, 1, 1, 1},    {z.H, z.d, z.V, 1, 0, T},   {T, z.dh, z.d, 1, 0, z.H},
      {T, z.d, z.A, 1, 0, 1},     {z.A, z.d, T, 0, 0, 1},     {T, z.A, z.d, 1, 1, 1},
      {z.d, z.dh, T, 0, 0, z.H},  {T, z.d, z.dh, 1, 1, z.H},  {z.H, z.V, z.d, 1, 1, T},
      {z.d, z.H, TV, 0, 0, 1}};
  size_t m = 0;
  for (const auto& x : sh) {
    Gemm g = base_gemm(dt);
    g.M = x[0]; g.N = x[1]; g.K = x[2]; g.a_kmajor = x[3]; g.b_kmajor = x[4]; g.batch = x[5];
    m = std::max(m, gemm_workspace_bytes(g));
  }
  return m;
}

size_t agg_workspace_bytes(const orbit_agg_desc& a) {
  const Sizes z = sizes(a);
  const orbit_dtype dt = (orbit_dtype)a.dtype;
  Carver f(nullptr);
  f.take<float>((size_t)z.T * z.V * z.H);
  f.take<char>((size_t)z.T * z.H * z.Vp * esz(dt));
  f.take<char>(gemv_part_bytes(z.d, z.A));
  size_t fwd = f.used();
  Carver b(nullptr);
  b.take<char>((size_t)z.T * z.A * esz(dt));
  b.take<char>((size_t)z.T * z.H * z.d * esz(dt));
  b.take<float>((size_t)z.T * z.H * z.V);
  b.take<char>((size_t)z.T * z.V * 2 * z.H * esz(dt));
  b.take<float>((size_t)z.d * z.H);
  b.take<float>((size_t)z.A);
  b.take<char>(gemv_part_bytes(z.d, z.A));
  b.take<char>(std::max(colsum_workspace_bytes((int)z.T, std::max(z.d, z.A)),
                        colsum_workspace_bytes(z.B, z.L * z.d)));
  size_t bwd = b.used();
  return std::max(fwd, bwd) + gemm_ws_max(z, dt);
}

orbit_status agg_forward(const orbit_agg_desc& a, const void* tok, const orbit_agg_params& p, void* z_out,
                         void* saved, void* ws, size_t ws_bytes, hipStream_t s) {
  const Sizes z = sizes(a);
  const orbit_dtype dt = (orbit_dtype)a.dtype;
  const Saved sv = carve_saved(z, dt, saved, nullptr);
  Carver w(ws);
  float* S = w.take<float>((size_t)z.T * z.V * z.H);
  void* ab = w.take<char>((size_t)z.T * z.H * z.Vp * esz(dt));
  float* gvp = w.take<float>(gemv_part_bytes(z.d, z.A) / sizeof(float));
  void* gws = w.take<char>(0);
  const size_t gws_bytes = ws_bytes - w.used();
  const int64_t TV = z.T * z.V;

  // 1. q = q0 W_q + b_q;  Ut[h] = W_k^h q_h
  KernelInfo ku{"agg_fold_key", 2.0 * z.d * z.A, (double)z.d * z.A * esz(dt)};
  if (dt == ORBIT_BF16) {
    ORBIT_TRY((gemv_cols<bf16, false>("agg_query", p.w_q, p.q0, nullptr, p.b_q, sv.q, gvp, z.d, z.A, z.H, z.dh, s)));
    ORBIT_TRY(launch(ku, agg_fold_key<bf16>, dim3((unsigned)cdiv(z.d, 4)), dim3(256), 0, s, (const bf16*)p.w_k,
                     (const float*)sv.q, (bf16*)sv.Ut, z.d, z.H, z.dh));
  } else {
    ORBIT_TRY((gemv_cols<float, false>("agg_query", p.w_q, p.q0, nullptr, p.b_q, sv.q, gvp, z.d, z.A, z.H, z.dh, s)));
    ORBIT_TRY(launch(ku, agg_fold_key<float>, dim3((unsigned)cdiv(z.d, 4)), dim3(256), 0, s,
                     (const float*)p.w_k, (const float*)sv.q, (float*)sv.Ut, z.d, z.H, z.dh));
  }
  // 2. scores S[t*V+v][h] = x_{t,v} . u_h / sqrt(dh)
  if (rowdot_ok(dt, z, tok, sv.Ut)) {
    ORBIT_TRY(rowdot("agg_scores", z, tok, sv.Ut, 0, S, (int64_t)z.V * z.H, z.H, 1, 1.f / sqrtf((float)z.dh), s));
  } else {
    Gemm g = base_gemm(dt);
    g.tag = "agg_scores";
    g.A = tok; g.lda = z.d; g.a_kmajor = true;
    g.B = sv.Ut; g.ldb = z.d; g.b_kmajor = true;
    g.C = S; g.ldc = z.H; g.out_f32 = true;
    g.M = (int)TV; g.N = z.H; g.K = z.d;
    g.alpha = 1.f / sqrtf((float)z.dh);
    g.stream = true;  // the token tensor is read once here
    ORBIT_TRY(gemm(g, gws, gws_bytes, s));
  }
  // 3. softmax over variables
  KernelInfo ks{"agg_softmax", 0.0, (double)TV * z.H * 8};
  if (dt == ORBIT_BF16)
    ORBIT_TRY(launch(ks, agg_softmax<bf16>, dim3((unsigned)cdiv(z.T, 4)), dim3(256), 0, s, (const float*)S, sv.a32,
                     (bf16*)ab, z.T, z.V, z.Vp, z.H));
  else
    ORBIT_TRY(launch(ks, agg_softmax<float>, dim3((unsigned)cdiv(z.T, 4)), dim3(256), 0, s, (const float*)S, sv.a32,
                     (float*)ab, z.T, z.V, z.Vp, z.H));
  // 4. xbar_t = a_t [H, V] X_t [V, d]   (batched over tokens)
  if (dt == ORBIT_BF16 && (z.H == 8 || z.H == 16)) {
    const int64_t items = z.T * cdiv(z.d, 512);
    KernelInfo kx{"agg_xbar", 2.0 * z.T * z.H * (double)z.V * z.d,
                  (double)z.T * (z.V + z.H) * z.d * 2.0};
    const dim3 grid((unsigned)cdiv(items, 4));
    if (z.H == 8)
      ORBIT_TRY(launch(kx, agg_xbar<8>, grid, dim3(256), 0, s, (const bf16*)ab, (const bf16*)tok, (bf16*)sv.xbar,
                       z.T, z.V, z.Vp, z.d));
    else
      ORBIT_TRY(launch(kx, agg_xbar<16>, grid, dim3(256), 0, s, (const bf16*)ab, (const bf16*)tok, (bf16*)sv.xbar,
                       z.T, z.V, z.Vp, z.d));
  } else {
    Gemm g = base_gemm(dt);
    g.tag = "agg_xbar";
    g.A = ab; g.lda = z.Vp; g.a_kmajor = true; g.sA = (int64_t)z.H * z.Vp;
    g.B = tok; g.ldb = z.d; g.b_kmajor = false; g.sB = (int64_t)z.V * z.d;
    g.C = sv.xbar; g.ldc = z.d; g.sC = (int64_t)z.H * z.d;
    g.M = z.H; g.N = z.d; g.K = z.V; g.batch = (int)z.T;
    ORBIT_TRY(gemm(g, gws, gws_bytes, s));
  }
  // 5. zh_h = xbar_h W_v^h + b_v^h   (batched over heads)
  {
    Gemm g = base_gemm(dt);
    g.tag = "agg_value";
    g.A = sv.xbar; g.lda = (int64_t)z.H * z.d; g.a_kmajor = true; g.sA = z.d;
    g.B = p.w_v; g.ldb = z.A; g.b_kmajor = false; g.sB = z.dh;
    g.C = sv.zh; g.ldc = z.A; g.sC = z.dh;
    g.bias = p.b_v; g.sBias = z.dh;
    g.M = (int)z.T; g.N = z.dh; g.K = z.d; g.batch = z.H;
    ORBIT_TRY(gemm(g, gws, gws_bytes, s));
  }
  // 6. z = zh W_o + b_o + pos[l]
  {
    Gemm g = base_gemm(dt);
    g.tag = "agg_out";
    g.A = sv.zh; g.lda = z.A; g.a_kmajor = true;
    g.B = p.w_o; g.ldb = z.d; g.b_kmajor = false;
    g.C = z_out; g.ldc = z.d;
    g.bias = p.b_o;
    if (p.pos) { g.res = p.pos; g.ldr = z.d; g.res_row_mod = z.L; }
    g.M = (int)z.T; g.N = z.d; g.K = z.A;
    ORBIT_TRY(gemm(g, gws, gws_bytes, s));
  }
  return ORBIT_OK;
}

orbit_status agg_backward(const orbit_agg_desc& a, const void* tok, const orbit_agg_params& p, const void* saved,
                          const void* dz, void* dtok, const orbit_agg_grads& gr, int accumulate, void* ws,
                          size_t ws_bytes, hipStream_t s) {
  const Sizes z = sizes(a);
  const orbit_dtype dt = (orbit_dtype)a.dtype;
  const Saved sv = carve_saved(z, dt, const_cast<void*>(saved), nullptr);
  Carver w(ws);
  void* dzh = w.take<char>((size_t)z.T * z.A * esz(dt));
  void* dxbar = w.take<char>((size_t)z.T * z.H * z.d * esz(dt));
  float* da = w.take<float>((size_t)z.T * z.H * z.V);
  void* ac = w.take<char>((size_t)z.T * z.V * 2 * z.H * esz(dt));
  float* dU = w.take<float>((size_t)z.d * z.H);
  float* dq = w.take<float>((size_t)z.A);
  float* gvp = w.take<float>(gemv_part_bytes(z.d, z.A) / sizeof(float));
  void* cws = w.take<char>(std::max(colsum_workspace_bytes((int)z.T, std::max(z.d, z.A)),
                                    colsum_workspace_bytes(z.B, z.L * z.d)));
  void* gws = w.take<char>(0);
  const size_t gws_bytes = ws_bytes - w.used();
  const int64_t TV = z.T * z.V;
  const float scale = 1.f / sqrtf((float)z.dh);

  // output projection: dpos, db_o, dW_o, dzh
  if (gr.pos) ORBIT_TRY(colsum(dt, dz, (int64_t)z.L * z.d, z.B, z.L * z.d, nullptr, 0, nullptr, nullptr, gr.pos,
                               nullptr, accumulate, cws, s));
  {
    // db_o is the column sum of dz, the weight-gradient product's B operand:
    // taken from that product where its kernel forms it
    Gemm g = base_gemm(dt);
    g.tag = "agg_out_dw";
    g.A = sv.zh; g.lda = z.A; g.a_kmajor = false;
    g.B = dz; g.ldb = z.d; g.b_kmajor = false;
    g.C = gr.w_o; g.ldc = z.d; g.out_f32 = true; g.accumulate = accumulate != 0;
    g.M = z.A; g.N = z.d; g.K = (int)z.T;
    g.bsum_max_parts = colsum_chunks((int)z.T);
    const int parts = gr.b_o ? gemm_bsum_parts(g) : 0;
    const bool fused = parts > 0 && parts <= colsum_chunks((int)z.T);
    if (fused) g.bsum = static_cast<float*>(cws);
    else
      ORBIT_TRY(colsum(dt, dz, z.d, (int)z.T, z.d, nullptr, 0, nullptr, nullptr, gr.b_o, nullptr, accumulate, cws, s));
    ORBIT_TRY(gemm(g, gws, gws_bytes, s));
    if (fused) {
      ColFinal f;
      f.add(static_cast<const float*>(cws), z.d, parts, z.d, gr.b_o);
      ORBIT_TRY(f.run(accumulate, s));
    }
  }
  {
    Gemm g = base_gemm(dt);
    g.tag = "agg_out_dx";
    g.A = dz; g.lda = z.d; g.a_kmajor = true;
    g.B = p.w_o; g.ldb = z.d; g.b_kmajor = true;
    g.C = dzh; g.ldc = z.A;
    g.M = (int)z.T; g.N = z.A; g.K = z.d;
    ORBIT_TRY(gemm(g, gws, gws_bytes, s));
  }
  // value path: db_v, dW_v^h = xbar_h^T dzh_h, dxbar_h = dzh_h W_v^h^T
  ORBIT_TRY(colsum(dt, dzh, z.A, (int)z.T, z.A, nullptr, 0, nullptr, nullptr, gr.b_v, nullptr, accumulate, cws, s));
  {
    Gemm g = base_gemm(dt);
    g.tag = "agg_value_dw";
    g.A = sv.xbar; g.lda = (int64_t)z.H * z.d; g.a_kmajor = false; g.sA = z.d;
    g.B = dzh; g.ldb = z.A; g.b_kmajor = false; g.sB = z.dh;
    g.C = gr.w_v; g.ldc = z.A; g.sC = z.dh; g.out_f32 = true; g.accumulate = accumulate != 0;
    g.M = z.d; g.N = z.dh; g.K = (int)z.T; g.batch = z.H;
    ORBIT_TRY(gemm(g, gws, gws_bytes, s));
  }
  if (dt == ORBIT_BF16 && (z.dh == 64 || z.dh == 128) && z.d % 256 == 0 && z.A % 8 == 0 &&
      (reinterpret_cast<uintptr_t>(p.w_v) & 15) == 0) {
    // row ranges: enough blocks for two per CU, whole 32-row chunks
    const int64_t cols = (int64_t)(z.d / 256) * z.H;
    const int64_t ranges = std::max<int64_t>(1, std::min<int64_t>(cdiv(z.T, 32), cdiv(512, cols)));
    const int rows = (int)(cdiv(cdiv(z.T, ranges), 32) * 32);
    KernelInfo kv{"agg_value_dx", 2.0 * z.T * z.H * (double)z.dh * z.d,
                  (double)z.T * z.H * z.d * 2.0 + (double)z.d * z.A * 2.0 + (double)z.T * z.A * 2.0};
    const dim3 grid((unsigned)(z.d / 256), (unsigned)z.H, (unsigned)cdiv(z.T, rows));
    if (z.dh == 64)
      ORBIT_TRY(launch(kv, agg_value_dx<64>, grid, dim3(256), 0, s, (const bf16*)dzh, (const bf16*)p.w_v,
                       (bf16*)dxbar, (int)z.T, z.H, z.d, rows));
    else
      ORBIT_TRY(launch(kv, agg_value_dx<128>, grid, dim3(256), 0, s, (const bf16*)dzh, (const bf16*)p.w_v,
                       (bf16*)dxbar, (int)z.T, z.H, z.d, rows));
  } else {
    Gemm g = base_gemm(dt);
    g.tag = "agg_value_dx";
    g.A = dzh; g.lda = z.A; g.a_kmajor = true; g.sA = z.dh;
    g.B = p.w_v; g.ldb = z.A; g.b_kmajor = true; g.sB = z.dh;
    g.C = dxbar; g.ldc = (int64_t)z.H * z.d; g.sC = z.d;
    g.M = (int)z.T; g.N = z.d; g.K = z.dh; g.batch = z.H;
    ORBIT_TRY(gemm(g, gws, gws_bytes, s));
  }
  // da_t [H, V] = dxbar_t [H, d] X_t^T
  if (rowdot_ok(dt, z, tok, dxbar)) {
    ORBIT_TRY(rowdot("agg_da", z, tok, dxbar, (int64_t)z.H * z.d, da, (int64_t)z.H * z.V, 1, z.V, 1.f, s));
  } else {
    Gemm g = base_gemm(dt);
    g.tag = "agg_da";
    g.A = dxbar; g.lda = z.d; g.a_kmajor = true; g.sA = (int64_t)z.H * z.d;
    g.B = tok; g.ldb = z.d; g.b_kmajor = true; g.sB = (int64_t)z.V * z.d;
    g.C = da; g.ldc = z.V; g.sC = (int64_t)z.H * z.V; g.out_f32 = true;
    g.M = z.H; g.N = z.V; g.K = z.d; g.batch = (int)z.T;
    ORBIT_TRY(gemm(g, gws, gws_bytes, s));
  }
  // softmax backward -> ac = [a | ds] per (t, v) row
  KernelInfo ksb{"agg_softmax_bwd", 0.0, (double)TV * z.H * (8 + 4 * esz(dt))};
  if (dt == ORBIT_BF16)
    ORBIT_TRY(launch(ksb, agg_softmax_bwd<bf16>, dim3((unsigned)cdiv(z.T, 4)), dim3(256), 0, s, (const float*)sv.a32,
                     (const float*)da, (bf16*)ac, z.T, z.V, z.H, scale));
  else
    ORBIT_TRY(launch(ksb, agg_softmax_bwd<float>, dim3((unsigned)cdiv(z.T, 4)), dim3(256), 0, s, (const float*)sv.a32,
                     (const float*)da, (float*)ac, z.T, z.V, z.H, scale));
  // dU [d, H] = X^T ds  (reduction over all T*V token rows)
  {
    Gemm g = base_gemm(dt);
    g.tag = "agg_du";
    g.A = tok; g.lda = z.d; g.a_kmajor = false;
    g.B = static_cast<const char*>(ac) + z.H * esz(dt); g.ldb = 2 * z.H; g.b_kmajor = false;
    g.C = dU; g.ldc = z.H; g.out_f32 = true;
    g.M = z.d; g.N = z.H; g.K = (int)TV;
    ORBIT_TRY(gemm(g, gws, gws_bytes, s));
  }
  // query path
  KernelInfo kou{"agg_outer", 2.0 * z.d * z.A, 8.0 * z.d * z.A};
  KernelInfo kqb{"agg_query_bwd", 2.0 * z.d * z.A, (double)z.d * z.A * esz(dt)};
  if (dt == ORBIT_BF16) {
    ORBIT_TRY((gemv_cols<bf16, true>("agg_dq", p.w_k, nullptr, dU, nullptr, dq, gvp, z.d, z.A, z.H, z.dh, s)));
    ORBIT_TRY(launch(kou, agg_outer<bf16>, dim3((unsigned)std::min<int64_t>(g1((int64_t)z.d * z.A / 4), 8192)),
                     dim3(256), 0, s, (const float*)dU, (const float*)sv.q, (const bf16*)p.q0, (const float*)dq,
                     gr.w_k, gr.w_q, z.d, z.H, z.dh, accumulate));
    ORBIT_TRY(launch(kqb, agg_query_bwd<bf16>, dim3((unsigned)cdiv(z.d, 4)), dim3(256), 0, s, (const bf16*)p.w_q,
                     (const float*)dq, gr.q0, gr.b_q, gr.b_k, z.d, z.A, accumulate));
  } else {
    ORBIT_TRY((gemv_cols<float, true>("agg_dq", p.w_k, nullptr, dU, nullptr, dq, gvp, z.d, z.A, z.H, z.dh, s)));
    ORBIT_TRY(launch(kou, agg_outer<float>, dim3((unsigned)std::min<int64_t>(g1((int64_t)z.d * z.A / 4), 8192)),
                     dim3(256), 0, s, (const float*)dU, (const float*)sv.q, (const float*)p.q0, (const float*)dq,
                     gr.w_k, gr.w_q, z.d, z.H, z.dh, accumulate));
    ORBIT_TRY(launch(kqb, agg_query_bwd<float>, dim3((unsigned)cdiv(z.d, 4)), dim3(256), 0, s,
                     (const float*)p.w_q, (const float*)dq, gr.q0, gr.b_q, gr.b_k, z.d, z.A, accumulate));
  }
  // dtok_t [V, d] = [a^T | ds] [V, 2H] . [dxbar_t ; U^T] [2H, d]   (batched over tokens)
  if (dt == ORBIT_BF16 && z.V <= 96 && (z.H == 8 || z.H == 16 || z.H == 32)) {
    KernelInfo kd{"agg_dtok", 2.0 * z.T * z.V * (double)z.d * 2 * z.H,
                  (double)z.T * (z.V + z.H) * z.d * 2.0};
    const dim3 grid((unsigned)cdiv(z.d, kDtokCols), (unsigned)z.T);
    const int mt = (int)cdiv(z.V, 32), ks = 2 * z.H / 16;
    const bf16* acp = static_cast<const bf16*>(ac);
    const bf16* dxp = static_cast<const bf16*>(dxbar);
    const bf16* up = static_cast<const bf16*>(sv.Ut);
    bf16* dp = static_cast<bf16*>(dtok);
#define DTOK(M, K) \
  if (mt == M && ks == K) return launch(kd, agg_dtok<M, K>, grid, dim3(256), 0, s, acp, dxp, up, dp, z.V, z.d, z.H)
    DTOK(1, 1); DTOK(2, 1); DTOK(3, 1);
    DTOK(1, 2); DTOK(2, 2); DTOK(3, 2);
    DTOK(1, 4); DTOK(2, 4); DTOK(3, 4);
#undef DTOK
  }
  {
    Gemm g = base_gemm(dt);
    g.tag = "agg_dtok";
    g.A = ac; g.lda = 2 * z.H; g.a_kmajor = true; g.sA = (int64_t)z.V * 2 * z.H;
    g.B = dxbar; g.ldb = z.d; g.b_kmajor = false; g.sB = (int64_t)z.H * z.d;
    g.B2 = sv.Ut; g.k_split = z.H; g.sB2 = 0;
    g.C = dtok; g.ldc = z.d; g.sC = (int64_t)z.V * z.d;
    g.M = z.V; g.N = z.d; g.K = 2 * z.H; g.batch = (int)z.T;
    ORBIT_TRY(gemm(g, gws, gws_bytes, s));
  }
  return ORBIT_OK;
}

}  // namespace orbit
