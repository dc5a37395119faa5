// Per-variable patch tokenisation: tok[b,l,v,:] = P[b,v,l,:] W_pe[v] + b_pe[v]
// + ve[v] with 4x4 patches (16 pixels), and its parameter gradients.
//
// Both directions are bound by HBM traffic on tok / dtok (one token row of d
// elements per patch and variable); the 16-deep products are done in float32
// vector ALU with the weight slice of a thread held in registers and the
// block's pixels staged in LDS.
#include <algorithm>

#include "kernels.h"
#include "tile.h"

namespace orbit {
namespace {

constexpr int kPP = 16;             // pixels per 4x4 patch
constexpr int kPatchesPerBlock = 64;

template <typename T> ORBIT_DEV void ld8f(const T* p, float* f) {
  if constexpr (sizeof(T) == 2) unpack(ld128(p), f, (bf16*)nullptr);
  else {
    unpack(ld128(p), f, (float*)nullptr);
    unpack(ld128(p + 4), f + 4, (float*)nullptr);
  }
}
template <typename T> ORBIT_DEV void st8f(T* p, const float* f) {
  if constexpr (sizeof(T) == 2) st128(p, pack(f, (bf16*)nullptr));
  else {
    st128(p, pack(f, (float*)nullptr));
    st128(p + 4, pack(f + 4, (float*)nullptr));
  }
}

// block: (patch group of 64, v, b); thread: 8 output columns of some patches
template <typename T>
__global__ void __launch_bounds__(256) patch_fwd_kernel(const float* __restrict__ img, const T* __restrict__ w,
                                                        const T* __restrict__ bias, const T* __restrict__ ve,
                                                        T* __restrict__ tok, int V, int Hg, int Wg, int d) {
  __shared__ float px[kPatchesPerBlock][kPP];
  const int v = blockIdx.y, b = blockIdx.z;
  const int nw = Wg / 4, L = (Hg / 4) * nw;
  const int l0 = blockIdx.x * kPatchesPerBlock;
  const float* im = img + ((int64_t)b * V + v) * Hg * Wg;
  for (int idx = threadIdx.x; idx < kPatchesPerBlock * kPP; idx += 256) {
    const int pl = idx / kPP, c = idx % kPP;
    const int l = l0 + pl;
    float val = 0.f;
    if (l < L) {
      const int ph = l / nw, pw = l % nw;
      val = im[(int64_t)(ph * 4 + c / 4) * Wg + pw * 4 + (c % 4)];
    }
    px[pl][c] = val;
  }
  __syncthreads();
  const int ech = d / 8;
  const int lanes = ech >= 256 ? 1 : 256 / ech;   // patch lanes per block
  const int ec_first = threadIdx.x % (ech >= 256 ? 256 : ech);
  const int plane = threadIdx.x / (ech >= 256 ? 256 : ech);
  if (plane >= lanes) return;
  for (int ec = ec_first; ec < ech; ec += 256) {
    const int e0 = ec * 8;
    float wr[kPP][8], add[8];
#pragma unroll
    for (int c = 0; c < kPP; ++c) ld8f(w + ((int64_t)v * kPP + c) * d + e0, wr[c]);
    ld8f(bias + (int64_t)v * d + e0, add);
    if (ve) {
      float t[8];
      ld8f(ve + (int64_t)v * d + e0, t);
#pragma unroll
      for (int i = 0; i < 8; ++i) add[i] += t[i];
    }
    for (int pl = plane; pl < kPatchesPerBlock; pl += lanes) {
      const int l = l0 + pl;
      if (l >= L) break;
      float o[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) o[i] = add[i];
#pragma unroll
      for (int c = 0; c < kPP; ++c) {
        const float p = px[pl][c];
#pragma unroll
        for (int i = 0; i < 8; ++i) o[i] += p * wr[c][i];
      }
      st8f(tok + (((int64_t)b * L + l) * V + v) * d + e0, o);
    }
  }
}

// partial gradients over a chunk of patches (all samples flattened, n = B*L):
// part[chunk][lane][v][17][d]: rows 0..15 = dW rows, row 16 = db
constexpr int kBwdPatchesPerChunk = 1024;

template <typename T>
__global__ void __launch_bounds__(256) patch_bwd_partial(const float* __restrict__ img, const T* __restrict__ dtok,
                                                         float* __restrict__ part, int B, int V, int Hg, int Wg,
                                                         int d) {
  __shared__ float px[kPatchesPerBlock][kPP];
  const int v = blockIdx.y, chunk = blockIdx.x;
  const int nw = Wg / 4, L = (Hg / 4) * nw;
  const int64_t n = (int64_t)B * L;
  const int ech = d / 8;
  const int per = ech >= 256 ? 256 : ech;
  const int lanes = ech >= 256 ? 1 : 256 / ech;  // 1, 2, 4 ... patch lanes
  const int ec_first = threadIdx.x % per, plane = threadIdx.x / per;
  for (int ecb = 0; ecb < ech; ecb += 256) {
    const int ec = ecb + ec_first;
    float acc[17][8];
#pragma unroll
    for (int r = 0; r < 17; ++r)
#pragma unroll
      for (int i = 0; i < 8; ++i) acc[r][i] = 0.f;
    for (int g0 = chunk * kBwdPatchesPerChunk; g0 < min<int64_t>(n, (int64_t)(chunk + 1) * kBwdPatchesPerChunk);
         g0 += kPatchesPerBlock) {
      __syncthreads();
      for (int idx = threadIdx.x; idx < kPatchesPerBlock * kPP; idx += 256) {
        const int pl = idx / kPP, c = idx % kPP;
        const int64_t gi = g0 + pl;
        float val = 0.f;
        if (gi < n) {
          const int b = (int)(gi / L), l = (int)(gi % L);
          const int ph = l / nw, pw = l % nw;
          val = img[(((int64_t)b * V + v) * Hg + ph * 4 + c / 4) * Wg + pw * 4 + (c % 4)];
        }
        px[pl][c] = val;
      }
      __syncthreads();
      if (plane < lanes && ec < ech) {
        for (int pl = plane; pl < kPatchesPerBlock; pl += lanes) {
          const int64_t gi = g0 + pl;
          if (gi >= n) break;
          float g8[8];
          ld8f(dtok + (gi * V + v) * d + ec * 8, g8);
#pragma unroll
          for (int c = 0; c < kPP; ++c) {
            const float p = px[pl][c];
#pragma unroll
            for (int i = 0; i < 8; ++i) acc[c][i] += p * g8[i];
          }
#pragma unroll
          for (int i = 0; i < 8; ++i) acc[16][i] += g8[i];
        }
      }
    }
    // one partial per (chunk, patch lane); the final pass sums them in order
    if (plane < lanes && ec < ech)
#pragma unroll
      for (int r = 0; r < 17; ++r)
        st8f(part + ((((int64_t)chunk * lanes + plane) * V + v) * 17 + r) * d + ec * 8, acc[r]);
  }
}

// bf16 pixels as two MFMA operands: x ~ hi + lo with hi = bf16(x) and
// lo = bf16(x - hi) (relative error ~2^-16, far below the bf16 output's)
ORBIT_DEV void split_hi_lo(const float* x, Frag<bf16>& hi, Frag<bf16>& lo) {
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const bf16 h = (bf16)x[j];
    hi.v[j] = h;
    lo.v[j] = (bf16)(x[j] - (float)h);
  }
}

// bf16 forward on MFMA: a block takes kPfTok tokens (32 per wave) of one
// variable and kPfCols columns. Left operand: the token's 16 pixels (hi and lo
// parts, two products); right operand: the W_pe[v] column slice staged in LDS
// as stored and read through transposing reads. Each wave writes 64 columns
// at a time through a private LDS area (16 contiguous bytes per lane) with the
// bias and variable embedding added.
constexpr int kPfCols = 512, kPfTok = 128;

__global__ void __launch_bounds__(256) patch_fwd_mfma(const float* __restrict__ img, const bf16* __restrict__ w,
                                                      const bf16* __restrict__ bias, const bf16* __restrict__ ve,
                                                      bf16* __restrict__ tok, int V, int Hg, int Wg, int d,
                                                      int64_t ntok) {
  using Stage = GemmStageMN<kPfCols, 16, 256>;
  constexpr int P = Stage::PITCH, EP = 64 + 4;
  __shared__ __attribute__((aligned(16))) bf16 Ws[16 * P];
  __shared__ __attribute__((aligned(16))) float ew_all[4][32 * EP];
  const int tid = threadIdx.x, lane = tid & 63, g = lane >> 5, wave = tid >> 6;
  const int v = blockIdx.y, c0 = blockIdx.x * kPfCols;
  const int64_t t0 = (int64_t)blockIdx.z * kPfTok + wave * 32;
  const int nw = Wg / 4, L = (Hg / 4) * nw;
  {
    Stage st;
    st.load(w + (int64_t)v * 16 * d, nullptr, 0, d, c0, d, 0, 16, tid);
    st.store(Ws, tid);
  }
  // pixels 8g .. 8g+7 of this lane's token: image rows 2g, 2g + 1 of the patch
  Frag<bf16> ahi, alo;
  {
    float x[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    const int64_t t = t0 + (lane & 31);
    if (t < ntok) {
      const int b = (int)(t / L), l = (int)(t % L);
      const int ph = l / nw, pw = l % nw;
      const float* row = img + (((int64_t)b * V + v) * Hg + ph * 4 + 2 * g) * Wg + pw * 4;
      const f32x4 r0 = *reinterpret_cast<const f32x4*>(row);
      const f32x4 r1 = *reinterpret_cast<const f32x4*>(row + Wg);
#pragma unroll
      for (int q = 0; q < 4; ++q) { x[q] = r0[q]; x[4 + q] = r1[q]; }
    }
    split_hi_lo(x, ahi, alo);
  }
  __syncthreads();
  float* ew = ew_all[wave];
  const int cl = (lane & 7) * 8;
#pragma unroll 1
  for (int pp = 0; pp < kPfCols / 64; ++pp) {
    const int col = c0 + pp * 64 + cl;
    if (c0 + pp * 64 >= d) break;
    f32x16 acc[2];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
#pragma unroll
      for (int i = 0; i < 16; ++i) acc[h][i] = 0.f;
      Frag<bf16> bfr;
      Stage::frag(bfr, Ws, pp * 64 + h * 32, 0, lane);
      mma16(acc[h], ahi, bfr);
      mma16(acc[h], alo, bfr);
    }
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int i = 0; i < 16; ++i) ew[((i >> 2) * 8 + g * 4 + (i & 3)) * EP + h * 32 + (lane & 31)] = acc[h][i];
    __builtin_amdgcn_wave_barrier();
    float add[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    if (col < d) {
      ld8f(bias + (int64_t)v * d + col, add);
      if (ve) {
        float e[8];
        ld8f(ve + (int64_t)v * d + col, e);
#pragma unroll
        for (int i = 0; i < 8; ++i) add[i] += e[i];
      }
    }
#pragma unroll
    for (int pass = 0; pass < 4; ++pass) {
      const int r = pass * 8 + (lane >> 3);
      const int64_t t = t0 + r;
      const f32x4 lo = *reinterpret_cast<const f32x4*>(ew + r * EP + cl);
      const f32x4 hi = *reinterpret_cast<const f32x4*>(ew + r * EP + cl + 4);
      if (t < ntok && col < d) {
        float o[8];
#pragma unroll
        for (int q = 0; q < 4; ++q) { o[q] = lo[q] + add[q]; o[4 + q] = hi[q] + add[4 + q]; }
        st8f(tok + (t * V + v) * d + col, o);
      }
    }
    __builtin_amdgcn_wave_barrier();
  }
}

// bf16: dW_pe[v] = sum_t P[t,v]^T dtok[t,v,:] on MFMA. A block takes 256
// columns of one variable over a slice of kPbTokens tokens, kPbStep tokens per
// stage (two 16-deep K-steps). Left operand rows: the 16 pixels (hi and lo
// parts, two products) plus a row of ones whose product is the bias gradient;
// the stage's pixels are gathered into LDS pixel-major. Right operand: the
// dtok rows of the stage, staged in LDS as stored and read through
// transposing reads. Partials per token slice in the layout patch_bwd_final
// sums.
constexpr int kPbCols = 256;
constexpr int kPbTokens = 1024;
constexpr int kPbStep = 32;

__global__ void __launch_bounds__(256) patch_bwd_mfma(const float* __restrict__ img, const bf16* __restrict__ dtok,
                                                      float* __restrict__ part, int V, int Hg, int Wg, int d,
                                                      int64_t ntok) {
  using Stage = GemmStageMN<kPbCols, kPbStep, 256>;
  constexpr int P = Stage::PITCH, XP = kPbStep + 4;
  __shared__ __attribute__((aligned(16))) bf16 Bs[2][kPbStep * P];
  __shared__ __attribute__((aligned(16))) float Px[2][16 * XP];
  const int tid = threadIdx.x, lane = tid & 63, g = lane >> 5, wave = tid >> 6;
  const int v = blockIdx.y, c0 = blockIdx.x * kPbCols;
  const int64_t t_begin = (int64_t)blockIdx.z * kPbTokens;
  const int64_t t_end = std::min<int64_t>(ntok, t_begin + kPbTokens);
  const int nw = Wg / 4, L = (Hg / 4) * nw;
  const int p = lane & 31;  // operand row: pixel (0..15), ones (16), zero
  f32x16 acc_hi[2], acc_lo[2];
#pragma unroll
  for (int j = 0; j < 2; ++j)
#pragma unroll
    for (int i = 0; i < 16; ++i) acc_hi[j][i] = acc_lo[j][i] = 0.f;
  Stage st;
  const bf16* X = dtok + (int64_t)v * d;
  const int64_t ld = (int64_t)V * d;
  // pixel gather: threads 0..127 take token tid % 32 and image row tid / 32 of its patch
  f32x4 px;
  auto gather = [&](int64_t ts) {
    px = f32x4{0.f, 0.f, 0.f, 0.f};
    const int64_t t = ts + (tid & 31);
    if (tid < 128 && t < t_end) {
      const int b = (int)(t / L), l = (int)(t % L);
      const int ph = l / nw, pw = l % nw;
      px = *reinterpret_cast<const f32x4*>(img + (((int64_t)b * V + v) * Hg + ph * 4 + (tid >> 5)) * Wg + pw * 4);
    }
  };
  auto put = [&](float* S) {
    if (tid < 128) {
#pragma unroll
      for (int e = 0; e < 4; ++e) S[((tid >> 5) * 4 + e) * XP + (tid & 31)] = px[e];
    }
  };
  // token indices of the slice are below 2^31 (checked by the caller)
  st.load(X, nullptr, 0, ld, c0, d, (int)t_begin, (int)t_end, tid);
  gather(t_begin);
  st.store(Bs[0], tid);
  put(Px[0]);
  __syncthreads();
  const int nsteps = (int)((t_end - t_begin + kPbStep - 1) / kPbStep);
  for (int it = 0; it < nsteps; ++it) {
    const int cur = it & 1;
    const int64_t t0 = t_begin + (int64_t)it * kPbStep;
    if (it + 1 < nsteps) {
      st.load(X, nullptr, 0, ld, c0, d, (int)(t0 + kPbStep), (int)t_end, tid);
      gather(t0 + kPbStep);
    }
#pragma unroll
    for (int kk = 0; kk < kPbStep / 16; ++kk) {
      float x[8] = {0, 0, 0, 0, 0, 0, 0, 0};
      if (p < 16) {
        const f32x4 a = *reinterpret_cast<const f32x4*>(Px[cur] + p * XP + kk * 16 + 8 * g);
        const f32x4 b = *reinterpret_cast<const f32x4*>(Px[cur] + p * XP + kk * 16 + 8 * g + 4);
#pragma unroll
        for (int q = 0; q < 4; ++q) { x[q] = a[q]; x[4 + q] = b[q]; }
      } else if (p == 16) {
#pragma unroll
        for (int j = 0; j < 8; ++j) x[j] = t0 + kk * 16 + 8 * g + j < t_end ? 1.f : 0.f;
      }
      Frag<bf16> ahi, alo;
      split_hi_lo(x, ahi, alo);
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        Frag<bf16> bfr;
        Stage::frag(bfr, Bs[cur], wave * 64 + j * 32, kk, lane);
        mma16(acc_hi[j], ahi, bfr);
        mma16(acc_lo[j], alo, bfr);
      }
    }
    if (it + 1 < nsteps) {
      st.store(Bs[cur ^ 1], tid);
      put(Px[cur ^ 1]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int c = c0 + wave * 64 + j * 32 + (lane & 31);
    if (c < d) {
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int r = (i >> 2) * 8 + g * 4 + (i & 3);
        if (r <= 16)
          part[(((int64_t)blockIdx.z * V + v) * 17 + r) * d + c] = acc_hi[j][i] + acc_lo[j][i];
      }
    }
  }
}

__global__ void __launch_bounds__(256) patch_bwd_final(const float* __restrict__ part, int chunks, int V, int d,
                                                       float* dw, float* db, float* dve, int accumulate) {
  const int64_t per = (int64_t)V * 17 * d;
  for (int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x; e < per; e += (int64_t)gridDim.x * 256) {
    float s = 0.f;
    for (int k = 0; k < chunks; ++k) s += part[(int64_t)k * per + e];
    const int64_t v = e / (17 * d), rem = e % (17 * d);
    const int r = (int)(rem / d), c = (int)(rem % d);
    if (r < 16) {
      float* o = dw + (v * 16 + r) * d + c;
      *o = accumulate ? *o + s : s;
    } else {
      float* o = db + v * d + c;
      *o = accumulate ? *o + s : s;
      if (dve) {
        float* o2 = dve + v * d + c;
        *o2 = accumulate ? *o2 + s : s;
      }
    }
  }
}

}  // namespace

orbit_status patch_embed_fwd(orbit_dtype dt, const float* img, const void* w, const void* b, const void* ve,
                             void* tok, int B, int V, int Hg, int Wg, int p, int d, hipStream_t s) {
  (void)p;
  const int L = (Hg / 4) * (Wg / 4);
  dim3 grid((unsigned)cdiv(L, kPatchesPerBlock), V, B);
  const double toks = (double)B * L * V;
  KernelInfo ki{dt == ORBIT_BF16 ? "patch_fwd_kernel<bf16>" : "patch_fwd_kernel<f32>", toks * d * 2 * kPP,
                toks * (kPP * 4.0 + d * (dt == ORBIT_BF16 ? 2.0 : 4.0))};
  if (dt == ORBIT_BF16) {
    const int64_t ntok = (int64_t)B * L;
    KernelInfo km{"patch_fwd_mfma", toks * d * 2 * kPP * 2, toks * (kPP * 4.0 + d * 2.0)};
    return launch(km, patch_fwd_mfma, dim3((unsigned)cdiv(d, kPfCols), V, (unsigned)cdiv(ntok, kPfTok)), dim3(256),
                  0, s, img, (const bf16*)w, (const bf16*)b, (const bf16*)ve, (bf16*)tok, V, Hg, Wg, d, ntok);
  }
  return launch(ki, patch_fwd_kernel<float>, grid, dim3(256), 0, s, img, (const float*)w, (const float*)b,
                (const float*)ve, (float*)tok, V, Hg, Wg, d);
}

size_t patch_embed_bwd_workspace_bytes(int B, int V, int Hg, int Wg, int p, int d) {
  (void)p;
  const int64_t n = (int64_t)B * (Hg / 4) * (Wg / 4);
  const int lanes = d / 8 >= 256 ? 1 : 256 / (d / 8);
  // partials of the float32 path (chunks x lanes) or of the bf16 path (token slices)
  const int64_t slices = std::max<int64_t>(cdiv(n, kBwdPatchesPerChunk) * lanes, cdiv(n, kPbTokens));
  return align_up((size_t)slices * V * 17 * (size_t)d * sizeof(float));
}

orbit_status patch_embed_bwd(orbit_dtype dt, const float* img, const void* dtok, float* dw, float* db, float* dve,
                             int accumulate, int B, int V, int Hg, int Wg, int p, int d, void* ws, hipStream_t s) {
  (void)p;
  const int64_t n = (int64_t)B * (Hg / 4) * (Wg / 4);
  const int chunks = (int)cdiv(n, kBwdPatchesPerChunk);
  const int lanes = d / 8 >= 256 ? 1 : 256 / (d / 8);
  float* part = static_cast<float*>(ws);
  dim3 grid(chunks, V);
  const double toks = (double)n * V;
  KernelInfo ki{dt == ORBIT_BF16 ? "patch_bwd_partial<bf16>" : "patch_bwd_partial<f32>", toks * d * 2 * 17,
                toks * (kPP * 4.0 + d * (dt == ORBIT_BF16 ? 2.0 : 4.0))};
  if (dt == ORBIT_BF16) {
    const int slices = (int)cdiv(n, kPbTokens);
    KernelInfo km{"patch_bwd_mfma", toks * d * 2 * 17, toks * (kPP * 4.0 + d * 2.0)};
    ORBIT_TRY(launch(km, patch_bwd_mfma, dim3((unsigned)cdiv(d, kPbCols), V, slices), dim3(256), 0, s, img,
                     (const bf16*)dtok, part, V, Hg, Wg, d, n));
    const int64_t per = (int64_t)V * 17 * d;
    KernelInfo kf{"patch_bwd_final", 0.0, (double)slices * per * 4};
    return launch(kf, patch_bwd_final, dim3((unsigned)std::min<int64_t>(cdiv(per, 256), 4096)), dim3(256), 0, s,
                  (const float*)part, slices, V, d, dw, db, dve, accumulate);
  } else {
    ORBIT_TRY(launch(ki, patch_bwd_partial<float>, grid, dim3(256), 0, s, img, (const float*)dtok, part, B, V,
                     Hg, Wg, d));
  }
  const int64_t per = (int64_t)V * 17 * d;
  KernelInfo kf{"patch_bwd_final", 0.0, (double)chunks * lanes * per * 4};
  return launch(kf, patch_bwd_final, dim3((unsigned)std::min<int64_t>(cdiv(per, 256), 4096)), dim3(256), 0, s,
                (const float*)part, chunks * lanes, V, d, dw, db, dve, accumulate);
}

}  // namespace orbit
