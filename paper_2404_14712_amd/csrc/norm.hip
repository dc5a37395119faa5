// LayerNorm (pre-LN, final LN and the per-head QK-LayerNorm) forward and
// backward, deterministic column reductions (bias and LayerNorm-parameter
// gradients) and small elementwise helpers. All HBM-bound: rows are read as
// 16-byte vectors by consecutive lanes; statistics are float32 wave/block
// reductions.
#include <algorithm>

#include "kernels.h"

namespace orbit {
namespace {

template <typename T> ORBIT_DEV void load8(const T* p, float* f);
template <> ORBIT_DEV void load8<bf16>(const bf16* p, float* f) { unpack(ld128(p), f, (bf16*)nullptr); }
template <> ORBIT_DEV void load8<float>(const float* p, float* f) {
  unpack(ld128(p), f, (float*)nullptr);
  unpack(ld128(p + 4), f + 4, (float*)nullptr);
}
template <typename T> ORBIT_DEV void store8(T* p, const float* f);
template <> ORBIT_DEV void store8<bf16>(bf16* p, const float* f) { st128(p, pack(f, (bf16*)nullptr)); }
template <> ORBIT_DEV void store8<float>(float* p, const float* f) {
  st128(p, pack(f, (float*)nullptr));
  st128(p + 4, pack(f + 4, (float*)nullptr));
}

// sum over a 256-thread block; `red` is 4 floats of LDS; ends with a barrier
ORBIT_DEV float block_sum256(float v, float* red) {
  v = wave_sum(v);
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) red[w] = v;
  __syncthreads();
  const float r = (red[0] + red[1]) + (red[2] + red[3]);
  __syncthreads();
  return r;
}

template <typename T, int NCH>
__global__ void __launch_bounds__(256) ln_fwd_kernel(const T* __restrict__ x, int64_t ldx,
                                                     const T* __restrict__ g, const T* __restrict__ b,
                                                     T* __restrict__ y, int64_t ldy, float* mean,
                                                     float* rstd, int n, float eps) {
  __shared__ float red[4];
  const int64_t row = blockIdx.x;
  const T* xr = x + row * ldx;
  float v[NCH][8];
  float s = 0.f;
#pragma unroll
  for (int c = 0; c < NCH; ++c) {
    const int idx = (threadIdx.x + c * 256) * 8;
    if (idx < n) {
      load8(xr + idx, v[c]);
#pragma unroll
      for (int i = 0; i < 8; ++i) s += v[c][i];
    }
  }
  const float mu = block_sum256(s, red) / (float)n;
  float q = 0.f;
#pragma unroll
  for (int c = 0; c < NCH; ++c) {
    const int idx = (threadIdx.x + c * 256) * 8;
    if (idx < n) {
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const float t = v[c][i] - mu;
        q += t * t;
      }
    }
  }
  const float r = rsqrtf(block_sum256(q, red) / (float)n + eps);
  T* yr = y + row * ldy;
#pragma unroll
  for (int c = 0; c < NCH; ++c) {
    const int idx = (threadIdx.x + c * 256) * 8;
    if (idx < n) {
      float gg[8], bb[8], o[8];
      load8(g + idx, gg);
      load8(b + idx, bb);
#pragma unroll
      for (int i = 0; i < 8; ++i) o[i] = (v[c][i] - mu) * r * gg[i] + bb[i];
      store8(yr + idx, o);
    }
  }
  if (threadIdx.x == 0) {
    if (mean) mean[row] = mu;
    if (rstd) rstd[row] = r;
  }
}

// Rows of up to 4096 elements: one wave per row (4 rows per block), lane l
// taking the 16-byte chunks l, l + 64, ...; statistics by wave reductions.
template <typename T, int PER>
__global__ void __launch_bounds__(256) ln_fwd_wave(const T* __restrict__ x, int64_t ldx, const T* __restrict__ g,
                                                   const T* __restrict__ b, T* __restrict__ y, int64_t ldy,
                                                   float* mean, float* rstd, int rows, int n, float eps) {
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= rows) return;
  const T* xr = x + row * ldx;
  float v[PER][8];
  float s = 0.f;
#pragma unroll
  for (int c = 0; c < PER; ++c) {
    const int idx = (lane + c * 64) * 8;
    if (idx < n) {
      load8(xr + idx, v[c]);
#pragma unroll
      for (int i = 0; i < 8; ++i) s += v[c][i];
    }
  }
  const float mu = wave_sum(s) / (float)n;
  float q = 0.f;
#pragma unroll
  for (int c = 0; c < PER; ++c)
    if ((lane + c * 64) * 8 < n)
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const float t = v[c][i] - mu;
        q += t * t;
      }
  const float r = rsqrtf(wave_sum(q) / (float)n + eps);
  T* yr = y + row * ldy;
#pragma unroll
  for (int c = 0; c < PER; ++c) {
    const int idx = (lane + c * 64) * 8;
    if (idx < n) {
      float gg[8], bb[8], o[8];
      load8(g + idx, gg);
      load8(b + idx, bb);
#pragma unroll
      for (int i = 0; i < 8; ++i) o[i] = (v[c][i] - mu) * r * gg[i] + bb[i];
      store8(yr + idx, o);
    }
  }
  if (lane == 0) {
    if (mean) mean[row] = mu;
    if (rstd) rstd[row] = r;
  }
}

// ---- column sums ------------------------------------------------------------
// Phase 1: a grid of (column block, row chunk) blocks, 1024 threads each: 64
// lanes x 8 consecutive columns, 16 row lanes striding over the chunk with 4
// rows in flight; the 16 row lanes are combined in LDS in a fixed order and
// the chunk's partial row is stored. Phase 2 sums the chunk partials of any
// number of outputs in a fixed order (per backward call, one launch for the
// outputs with many partials and one for those with few).
constexpr int kCsCols = 512;      // columns per block (64 lanes x 8)
constexpr int kCsRowLanes = 16;   // row lanes per block
constexpr int kCsMaxChunks = 32;
constexpr int kCsThinRows = 8;     // at most this many rows: colsum_thin_kernel

int cs_rows_per_chunk(int rows) {
  return (int)std::max<int64_t>(64, cdiv(cdiv(rows, kCsMaxChunks), 16) * 16);
}

struct CsJobK {
  const void* src; int64_t ld; int64_t sbatch;   // batch b: src + b * sbatch
  const void* x; int64_t ldx; int64_t sxbatch;
  const float* mean; const float* rstd;
  float* part; int64_t spart;                     // [batch][chunks (x2 for LN)][n]
  int n, cb0, batch;
};
struct CsArgs {
  CsJobK job[kColMaxJobs];
  int njobs, rows, rpc, chunks;
};

template <typename T>
__global__ void __launch_bounds__(1024) colsum_partials_kernel(CsArgs a) {
  __shared__ float red[2][kCsRowLanes][kCsCols + 4];
  int j = 0;
  while (j + 1 < a.njobs && (int)blockIdx.x >= a.job[j + 1].cb0) ++j;
  const CsJobK& J = a.job[j];
  const int cb = (int)blockIdx.x - J.cb0;
  const int bz = blockIdx.z;
  if (bz >= J.batch) return;
  const bool ln = J.x != nullptr;
  const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
  const int c0 = cb * kCsCols + tx * 8;
  const int chunk = blockIdx.y;
  const int r0 = chunk * a.rpc, r1 = min(a.rows, r0 + a.rpc);
  const T* src = static_cast<const T*>(J.src) + bz * J.sbatch;
  const T* xs = ln ? static_cast<const T*>(J.x) + bz * J.sxbatch : nullptr;
  float s[8], sx[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) s[i] = sx[i] = 0.f;
  if (c0 < J.n) {
    for (int rb = r0 + ty; rb < r1; rb += 4 * kCsRowLanes) {
      float d[4][8], xv[4][8];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int r = rb + u * kCsRowLanes;
        if (r < r1) {
          load8(src + (int64_t)r * J.ld + c0, d[u]);
          if (ln) load8(xs + (int64_t)r * J.ldx + c0, xv[u]);
        }
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int r = rb + u * kCsRowLanes;
        if (r < r1) {
#pragma unroll
          for (int i = 0; i < 8; ++i) s[i] += d[u][i];
          if (ln) {
            const float mu = J.mean[(int64_t)bz * a.rows + r], rs = J.rstd[(int64_t)bz * a.rows + r];
#pragma unroll
            for (int i = 0; i < 8; ++i) sx[i] += d[u][i] * ((xv[u][i] - mu) * rs);
          }
        }
      }
    }
  }
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    red[0][ty][tx * 8 + i] = s[i];
    red[1][ty][tx * 8 + i] = sx[i];
  }
  __syncthreads();
  // threads 0..511: the sum of column c; 512..1023: the x-weighted sum
  const int which = threadIdx.x / kCsCols, cc = threadIdx.x % kCsCols;
  const int c = cb * kCsCols + cc;
  if (c < J.n && (which == 0 || ln)) {
    float t = 0.f;
#pragma unroll
    for (int q = 0; q < kCsRowLanes; ++q) t += red[which][q][cc];
    J.part[bz * J.spart + ((int64_t)which * a.chunks + chunk) * J.n + c] = t;
  }
}

// Column sums of a few rows (the batch sum of a per-position gradient): one
// thread per 8 consecutive columns adds the rows in order and writes (or adds
// to) the output directly, with no partials.
template <typename T>
__global__ void __launch_bounds__(256) colsum_thin_kernel(const T* src, int64_t ld, int rows, int64_t n,
                                                          float* out, int accumulate) {
  const int64_t c = ((int64_t)blockIdx.x * 256 + threadIdx.x) * 8;
  if (c >= n) return;
  float s[8], d[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) s[i] = 0.f;
  for (int r = 0; r < rows; ++r) {
    load8(src + (int64_t)r * ld + c, d);
#pragma unroll
    for (int i = 0; i < 8; ++i) s[i] += d[i];
  }
  float4* o = reinterpret_cast<float4*>(out + c);
  float4 lo = make_float4(s[0], s[1], s[2], s[3]), hi = make_float4(s[4], s[5], s[6], s[7]);
  if (accumulate) {
    const float4 a0 = o[0], a1 = o[1];
    lo = make_float4(a0.x + lo.x, a0.y + lo.y, a0.z + lo.z, a0.w + lo.w);
    hi = make_float4(a1.x + hi.x, a1.y + hi.y, a1.z + hi.z, a1.w + hi.w);
  }
  o[0] = lo;
  o[1] = hi;
}

struct CsFinalK {
  const float* part; int64_t ldp;   // partial k of element e at part[k * ldp + e]
  float* out;
  int chunks, n, cb0;
};
struct CsFinalArgs {
  CsFinalK item[kColMaxFinal];
  int nitems, accumulate;
};

// EL = 256 / CL elements x CL chunk lanes per block; each lane sums a fixed
// strided subset of the chunks (8 loads in flight), the CL lane sums are
// combined in order. CL = 16 for many chunks, 1 for a few.
template <int CL>
__global__ void __launch_bounds__(256) colsum_final_kernel(CsFinalArgs a) {
  constexpr int EL = 256 / CL;
  __shared__ float red[CL][EL + 1];
  int j = 0;
  while (j + 1 < a.nitems && (int)blockIdx.x >= a.item[j + 1].cb0) ++j;
  const CsFinalK& I = a.item[j];
  const int el = threadIdx.x % EL, q = threadIdx.x / EL;
  const int64_t e = (int64_t)((int)blockIdx.x - I.cb0) * EL + el;
  float s = 0.f;
  if (e < I.n) {
#pragma unroll 8
    for (int k = q; k < I.chunks; k += CL) s += I.part[(int64_t)k * I.ldp + e];
  }
  if constexpr (CL == 1) {
    if (e < I.n) I.out[e] = a.accumulate ? I.out[e] + s : s;
  } else {
    red[q][el] = s;
    __syncthreads();
    if (q == 0 && e < I.n) {
      float t = 0.f;
#pragma unroll
      for (int k = 0; k < CL; ++k) t += red[k][el];
      I.out[e] = a.accumulate ? I.out[e] + t : t;
    }
  }
}

// ---- LayerNorm backward fused with its column sums ---------------------------
// A block takes a chunk of rpb rows. Besides dx it stores one partial row per
// column sum over the chunk: of dy (the shift's gradient), of dy * xhat (the
// gain's) and, with OSUM, of the output dx (the bias gradient of the layer
// whose output the residual stream carries into this LayerNorm). The
// partials are added in a fixed order afterwards, so the sums never re-read
// dy, x or dx. The block's G groups of TPR threads (TPR a multiple of 64 up
// to 512, 8 NCH TPR >= n) take the chunk's rows in turn: group q rows r0 + q,
// r0 + q + G, ...; thread t of a group owns the NCH 8-column pieces starting
// at 8(t + c TPR). A group loads RB rows at once (dy, x and the residual
// gradient all in flight together) and forms their statistics with one
// block barrier; every group runs the same number of batches, so the
// barriers line up.
struct LnColArgs {
  const void *dy, *x, *g, *dres;
  void* dx;
  const float *mean, *rstd;
  int64_t lddy, ldx, lddx;
  float* part;  // sum k (0: dy, 1: dy * xhat, 2: dx) of chunk c at part[(k * chunks + c) * n]
  int rows, n, tpr, rpb;
};

// 8 values of T as loaded (bf16 stays packed: 4 registers instead of 8)
template <typename T>
struct Raw8 {
  U128 v[sizeof(T) / 2];
  ORBIT_DEV void load(const T* p) {
#pragma unroll
    for (int i = 0; i < (int)(sizeof(T) / 2); ++i) v[i] = ld128(p + i * (8 / (sizeof(T) / 2)));
  }
  ORBIT_DEV void zero() {
#pragma unroll
    for (int i = 0; i < (int)(sizeof(T) / 2); ++i) v[i] = zero128();
  }
  ORBIT_DEV void get(float* f) const {
#pragma unroll
    for (int i = 0; i < (int)(sizeof(T) / 2); ++i) unpack(v[i], f + i * (8 / (sizeof(T) / 2)), (T*)nullptr);
  }
};

template <typename T, int NCH>
constexpr int ln_cols_rb() { return NCH == 2 ? 2 : 1; }

// one batch of RB rows of a group: their positions, statistics and data
template <typename T, int NCH, int RB>
struct LnBatch {
  int64_t r[RB];
  bool rv[RB];
  float mu[RB], rs[RB];
  Raw8<T> d[RB][NCH], x[RB][NCH], e[RB][NCH];
};

template <typename T, int NCH, bool OSUM>
__global__ void __launch_bounds__(512) ln_bwd_cols_kernel(LnColArgs a) {
  constexpr int RB = ln_cols_rb<T, NCH>();
  using Batch = LnBatch<T, NCH, RB>;
  __shared__ float red[2][8][RB][2];
  const int tpr = a.tpr, G = (int)blockDim.x / tpr, wpg = tpr >> 6;
  const int q = (int)threadIdx.x / tpr, t = (int)threadIdx.x % tpr;
  const int wave = (int)threadIdx.x >> 6, lane = (int)threadIdx.x & 63;
  const int n = a.n, chunks = (int)gridDim.x;
  const int r0 = (int)blockIdx.x * a.rpb, r1 = min(a.rows, r0 + a.rpb);
  const T* dy = static_cast<const T*>(a.dy);
  const T* x = static_cast<const T*>(a.x);
  const T* dres = static_cast<const T*>(a.dres);
  const T* gp = static_cast<const T*>(a.g);
  T* dx = static_cast<T*>(a.dx);
  int col[NCH];
  bool on[NCH];
#pragma unroll
  for (int c = 0; c < NCH; ++c) {
    col[c] = 8 * (t + c * tpr);
    on[c] = col[c] < n;
  }
  float cs[NCH][8], cx[NCH][8], co[NCH][8];
#pragma unroll
  for (int c = 0; c < NCH; ++c)
#pragma unroll
    for (int i = 0; i < 8; ++i) cs[c][i] = cx[c][i] = co[c][i] = 0.f;
  const float inv_n = 1.f / (float)n;
  const int steps = (a.rpb + G - 1) / G;  // rows per group
  // batch `it` (rows it .. it + RB - 1 of this group): the next batch is
  // fetched before the current one is reduced, so loads stay in flight
  auto fetch = [&](int it, Batch& B) {
#pragma unroll
    for (int b = 0; b < RB; ++b) {
      B.r[b] = r0 + q + (int64_t)(it + b) * G;
      B.rv[b] = it + b < steps && B.r[b] < r1;
      B.mu[b] = B.rv[b] ? a.mean[B.r[b]] : 0.f;
      B.rs[b] = B.rv[b] ? a.rstd[B.r[b]] : 0.f;
#pragma unroll
      for (int c = 0; c < NCH; ++c) {
        if (B.rv[b] && on[c]) {
          B.d[b][c].load(dy + B.r[b] * a.lddy + col[c]);
          B.x[b][c].load(x + B.r[b] * a.ldx + col[c]);
          if (dres) B.e[b][c].load(dres + B.r[b] * a.lddx + col[c]);
          else B.e[b][c].zero();
        } else {
          B.d[b][c].zero();
          B.x[b][c].zero();
          B.e[b][c].zero();
        }
      }
    }
  };
  // bf16 rows hold the next batch in registers as well (float32 rows and
  // the widest rows with three sums would spill)
  constexpr bool DB = sizeof(T) == 2 && !(NCH == 4 && OSUM);
  Batch cur;
  if (DB) fetch(0, cur);
  int par = 0;
  for (int it = 0; it < steps; it += RB, par ^= 1) {
    Batch nxt;
    if (DB) fetch(it + RB, nxt);
    else fetch(it, cur);
    float s1[RB], s2[RB];
#pragma unroll
    for (int b = 0; b < RB; ++b) {
      s1[b] = s2[b] = 0.f;
#pragma unroll
      for (int c = 0; c < NCH; ++c) {
        if (cur.rv[b] && on[c]) {
          Raw8<T> gr;
          gr.load(gp + col[c]);
          float d8[8], x8[8], g8[8];
          cur.d[b][c].get(d8);
          cur.x[b][c].get(x8);
          gr.get(g8);
#pragma unroll
          for (int i = 0; i < 8; ++i) {
            const float gh = d8[i] * g8[i];
            s1[b] += gh;
            s2[b] += gh * ((x8[i] - cur.mu[b]) * cur.rs[b]);
          }
        }
      }
      s1[b] = wave_sum(s1[b]);
      s2[b] = wave_sum(s2[b]);
    }
    if (wpg > 1) {
      // the group's wave sums, added in wave order
      if (lane == 0) {
#pragma unroll
        for (int b = 0; b < RB; ++b) {
          red[par][wave][b][0] = s1[b];
          red[par][wave][b][1] = s2[b];
        }
      }
      __syncthreads();
#pragma unroll
      for (int b = 0; b < RB; ++b) {
        s1[b] = s2[b] = 0.f;
        for (int w = q * wpg; w < (q + 1) * wpg; ++w) {
          s1[b] += red[par][w][b][0];
          s2[b] += red[par][w][b][1];
        }
      }
    }
#pragma unroll
    for (int b = 0; b < RB; ++b) {
      const float m1 = s1[b] * inv_n, m2 = s2[b] * inv_n;
#pragma unroll
      for (int c = 0; c < NCH; ++c) {
        if (cur.rv[b] && on[c]) {
          float d8[8], x8[8], g8[8], e8[8], o[8];
          Raw8<T> gr;
          gr.load(gp + col[c]);
          cur.d[b][c].get(d8);
          cur.x[b][c].get(x8);
          cur.e[b][c].get(e8);
          gr.get(g8);
#pragma unroll
          for (int i = 0; i < 8; ++i) {
            x8[i] = (x8[i] - cur.mu[b]) * cur.rs[b];
            o[i] = cur.rs[b] * (d8[i] * g8[i] - m1 - x8[i] * m2) + e8[i];
          }
          store8(dx + cur.r[b] * a.lddx + col[c], o);
#pragma unroll
          for (int i = 0; i < 8; ++i) {
            cs[c][i] += d8[i];
            cx[c][i] += d8[i] * x8[i];
            if (OSUM) co[c][i] += o[i];
          }
        }
      }
    }
    if (DB) cur = nxt;
  }
  // the groups' sums of the chunk, added in group order through LDS (rows of
  // up to 8192 elements, where a block holds more than one group), then one
  // partial row per sum
  __shared__ float comb[NCH == 2 ? 512 * 16 : 1];
#pragma unroll
  for (int k = 0; k < (OSUM ? 3 : 2); ++k) {
    float (*v)[8] = k == 0 ? cs : k == 1 ? cx : co;
    if (NCH == 2 && G > 1) {
      __syncthreads();
#pragma unroll
      for (int c = 0; c < NCH; ++c)
#pragma unroll
        for (int i = 0; i < 8; ++i) comb[threadIdx.x * 16 + c * 8 + i] = v[c][i];
      __syncthreads();
      if (q == 0) {
        for (int gq = 1; gq < G; ++gq)
#pragma unroll
          for (int c = 0; c < NCH; ++c)
#pragma unroll
            for (int i = 0; i < 8; ++i) v[c][i] += comb[(gq * tpr + t) * 16 + c * 8 + i];
      }
    }
    if (q != 0) continue;
#pragma unroll
    for (int c = 0; c < NCH; ++c)
      if (on[c]) store8(a.part + ((int64_t)k * chunks + blockIdx.x) * n + col[c], v[c]);
  }
}

// ---- QK-LayerNorm -------------------------------------------------------------
template <typename T, int DH>
__global__ void __launch_bounds__(256) qkln_fwd_kernel(const T* __restrict__ src, int64_t lds,
                                                       T* __restrict__ dst, int64_t ldd,
                                                       const T* __restrict__ qg, const T* __restrict__ qb,
                                                       const T* __restrict__ kg, const T* __restrict__ kb,
                                                       float* mean, float* rstd, int T_, int H, int A,
                                                       float eps) {
  // a row's DH / 8 chunks of 8 values on G = the next power of two lanes
  // (lanes past the last chunk hold zeros; head_dim 192 runs 24 of 32)
  constexpr int CH = DH / 8, G = pow2_ceil(CH);
  const int li = threadIdx.x % G;
  const bool lv = li < CH;
  // row (t, j): head slot j < 2H of token t (q heads, then k heads), at
  // column j * DH of the token's [q | k] columns; rows < 2^31 (host check)
  const unsigned row = blockIdx.x * (256u / G) + threadIdx.x / G;
  const unsigned nr = 2u * H;
  const bool valid = row < (unsigned)T_ * nr;
  const unsigned t = valid ? row / nr : 0u;
  const unsigned j = valid ? row - t * nr : 0u;
  const int sidx = (int)j >= H;
  float v[8];
  if (valid && lv) load8(src + (int64_t)t * lds + j * DH + li * 8, v);
  else
#pragma unroll
    for (int i = 0; i < 8; ++i) v[i] = 0.f;
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < 8; ++i) s += v[i];
#pragma unroll
  for (int o = G / 2; o >= 1; o >>= 1) s += __shfl_xor(s, o, 64);
  const float mu = s / (float)DH;
  float q = 0.f;
#pragma unroll
  for (int i = 0; i < 8; ++i) q += lv ? (v[i] - mu) * (v[i] - mu) : 0.f;
#pragma unroll
  for (int o = G / 2; o >= 1; o >>= 1) q += __shfl_xor(q, o, 64);
  const float r = rsqrtf(q / (float)DH + eps);
  if (!valid || !lv) return;
  float gg[8], bb[8], y[8];
  load8((sidx ? kg : qg) + li * 8, gg);
  load8((sidx ? kb : qb) + li * 8, bb);
#pragma unroll
  for (int i = 0; i < 8; ++i) y[i] = (v[i] - mu) * r * gg[i] + bb[i];
  store8(dst + (int64_t)t * ldd + j * DH + li * 8, y);
  if (li == 0) {
    mean[row] = mu;
    rstd[row] = r;
  }
}

constexpr int kQkBwdBlocks = 512;

template <typename T, int DH>
__global__ void __launch_bounds__(256) qkln_bwd_kernel(T* d, int64_t ldd, const T* __restrict__ src,
                                                       int64_t lds, const float* __restrict__ mean,
                                                       const float* __restrict__ rstd,
                                                       const T* __restrict__ qg, const T* __restrict__ kg,
                                                       int T_, int H, int A, float* __restrict__ part) {
  constexpr int CH = DH / 8, G = pow2_ceil(CH);  // as in the forward
  constexpr int NG = 256 / G;  // row groups per block
  __shared__ float sm[NG][4][DH];
  const int li = threadIdx.x % G, grp = threadIdx.x / G;
  const bool lv = li < CH;
  float ag[2][8], ab[2][8];
#pragma unroll
  for (int s = 0; s < 2; ++s)
#pragma unroll
    for (int i = 0; i < 8; ++i) ag[s][i] = ab[s][i] = 0.f;
  float gq[8], gk[8];
  if (lv) {
    load8(qg + li * 8, gq);
    load8(kg + li * 8, gk);
  } else {
#pragma unroll
    for (int i = 0; i < 8; ++i) gq[i] = gk[i] = 0.f;
  }
  // rows (t, j) as in the forward; a row group walks rows base, base +
  // stride, ... keeping (t, j) by carries (one division at the start)
  const unsigned nr = 2u * H;
  const unsigned nrows = (unsigned)T_ * nr;
  // every row group of every block runs the same number of iterations
  // (shuffles); each iteration takes kQkRows rows, whose loads were issued
  // during the previous iteration (packed, as loaded)
  constexpr int kQkRows = 4;
  const unsigned stride = gridDim.x * (unsigned)NG;
  const unsigned iters = (nrows + stride * kQkRows - 1) / (stride * kQkRows);
  const unsigned st = stride / nr, sj = stride - st * nr;
  unsigned row = blockIdx.x * (unsigned)NG + grp;
  unsigned tc = row / nr, jc = row - tc * nr;
  struct Batch {
    Raw8<T> dy[kQkRows], xv[kQkRows];
    int64_t off_d[kQkRows];
    bool k[kQkRows], valid[kQkRows];
    float mu[kQkRows], r[kQkRows];
  };
  auto fetch = [&](Batch& B) {
#pragma unroll
    for (int u = 0; u < kQkRows; ++u) {
      B.valid[u] = row < nrows;
      B.k[u] = (int)jc >= H;
      B.off_d[u] = (int64_t)tc * ldd + jc * DH + li * 8;
      const int64_t off_s = (int64_t)tc * lds + jc * DH + li * 8;
      const unsigned rcur = row;
      row += stride;
      jc += sj;
      tc += st;
      if (jc >= nr) { jc -= nr; ++tc; }
      if (B.valid[u] && lv) {
        B.dy[u].load(d + B.off_d[u]);
        B.xv[u].load(src + off_s);
      } else {
        B.dy[u].zero();
        B.xv[u].zero();
      }
      B.mu[u] = B.valid[u] ? mean[rcur] : 0.f;
      B.r[u] = B.valid[u] ? rstd[rcur] : 0.f;
    }
  };
  Batch cur;
  if (iters > 0) fetch(cur);
  for (unsigned it = 0; it < iters; ++it) {
    Batch nxt;
    if (it + 1 < iters) fetch(nxt);
#pragma unroll
    for (int u = 0; u < kQkRows; ++u) {
      float dy[8], xv[8], xh[8], gh[8];
      cur.dy[u].get(dy);
      cur.xv[u].get(xv);
      float s1 = 0.f, s2 = 0.f;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        xh[i] = (xv[i] - cur.mu[u]) * cur.r[u];
        gh[i] = dy[i] * (cur.k[u] ? gk[i] : gq[i]);
        s1 += gh[i];
        s2 += gh[i] * xh[i];
      }
#pragma unroll
      for (int o = G / 2; o >= 1; o >>= 1) {
        s1 += __shfl_xor(s1, o, 64);
        s2 += __shfl_xor(s2, o, 64);
      }
      if (cur.valid[u] && lv) {
        const float m1 = s1 / (float)DH, m2 = s2 / (float)DH;
        float o8[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) o8[i] = cur.r[u] * (gh[i] - m1 - xh[i] * m2);
        store8(d + cur.off_d[u], o8);
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          if (cur.k[u]) { ag[1][i] += dy[i] * xh[i]; ab[1][i] += dy[i]; }
          else          { ag[0][i] += dy[i] * xh[i]; ab[0][i] += dy[i]; }
        }
      }
    }
    cur = nxt;
  }
  if (lv) {
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      sm[grp][0][li * 8 + i] = ag[0][i];
      sm[grp][1][li * 8 + i] = ab[0][i];
      sm[grp][2][li * 8 + i] = ag[1][i];
      sm[grp][3][li * 8 + i] = ab[1][i];
    }
  }
  __syncthreads();
  for (int e = threadIdx.x; e < 4 * DH; e += 256) {
    const int which = e / DH, c = e % DH;
    float s = 0.f;
    for (int g2 = 0; g2 < NG; ++g2) s += sm[g2][which][c];
    part[(int64_t)blockIdx.x * 4 * DH + e] = s;
  }
}

// ---- elementwise --------------------------------------------------------------
template <typename T>
__global__ void __launch_bounds__(256) cast_kernel(const float* __restrict__ src, T* __restrict__ dst, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256)
    dst[i] = from_f<T>(src[i]);
}

__global__ void __launch_bounds__(256) axpy_kernel(const float* __restrict__ src, float* dst, int64_t n, int acc) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256)
    dst[i] = acc ? dst[i] + src[i] : src[i];
}

__global__ void __launch_bounds__(256) fill_kernel(float* dst, int64_t n, float v) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256) dst[i] = v;
}

unsigned grid1d(int64_t n) { return (unsigned)std::max<int64_t>(1, std::min<int64_t>(cdiv(n, 256), 16384)); }

template <typename T, int NCH>
orbit_status ln_fwd_t(const void* x, int64_t ldx, const void* g, const void* b, void* y, int64_t ldy,
                      float* mean, float* rstd, int rows, int n, float eps, hipStream_t s) {
  KernelInfo ki{sizeof(T) == 2 ? "ln_fwd_kernel<bf16>" : "ln_fwd_kernel<f32>", 8.0 * rows * n,
                2.0 * rows * n * sizeof(T)};
  return launch(ki, ln_fwd_kernel<T, NCH>, dim3(rows), dim3(256), 0, s, (const T*)x, ldx, (const T*)g,
                (const T*)b, (T*)y, ldy, mean, rstd, n, eps);
}

template <typename T>
orbit_status ln_fwd_dispatch(const void* x, int64_t ldx, const void* g, const void* b, void* y, int64_t ldy,
                             float* mean, float* rstd, int rows, int n, float eps, hipStream_t s) {
  if (n <= 4096) {
    KernelInfo ki{sizeof(T) == 2 ? "ln_fwd_wave<bf16>" : "ln_fwd_wave<f32>", 8.0 * rows * n,
                  2.0 * rows * n * sizeof(T)};
    const int per = (int)cdiv(n, 512);
    const dim3 grid((unsigned)cdiv(rows, 4));
#define LNF(P) if (per <= P) return launch(ki, ln_fwd_wave<T, P>, grid, dim3(256), 0, s, (const T*)x, ldx, (const T*)g, \
                                           (const T*)b, (T*)y, ldy, mean, rstd, rows, n, eps)
    LNF(1); LNF(2); LNF(4); LNF(8);
#undef LNF
  }
  const int nch = (int)cdiv(n, 2048);
  if (nch <= 1) return ln_fwd_t<T, 1>(x, ldx, g, b, y, ldy, mean, rstd, rows, n, eps, s);
  if (nch <= 2) return ln_fwd_t<T, 2>(x, ldx, g, b, y, ldy, mean, rstd, rows, n, eps, s);
  if (nch <= 4) return ln_fwd_t<T, 4>(x, ldx, g, b, y, ldy, mean, rstd, rows, n, eps, s);
  if (nch <= 8) return ln_fwd_t<T, 8>(x, ldx, g, b, y, ldy, mean, rstd, rows, n, eps, s);
  set_error("layernorm: row length %d exceeds 16384", n);
  return ORBIT_E_UNSUPPORTED;
}

template <typename T, int DH>
orbit_status qk_fwd_t(const void* src, int64_t lds, void* dst, int64_t ldd, const void* qg, const void* qb,
                      const void* kg, const void* kb, float* mean, float* rstd, int T_, int H, float eps,
                      hipStream_t s) {
  constexpr int G = pow2_ceil(DH / 8);
  const int64_t rows = (int64_t)T_ * 2 * H;
  KernelInfo ki{sizeof(T) == 2 ? "qkln_fwd_kernel<bf16>" : "qkln_fwd_kernel<f32>", 8.0 * rows * DH,
                2.0 * rows * DH * sizeof(T)};
  return launch(ki, qkln_fwd_kernel<T, DH>, dim3((unsigned)cdiv(rows, 256 / G)), dim3(256), 0, s,
                (const T*)src, lds, (T*)dst, ldd, (const T*)qg, (const T*)qb, (const T*)kg, (const T*)kb, mean,
                rstd, T_, H, H * DH, eps);
}

template <typename T, int DH>
orbit_status qk_bwd_t(void* d, int64_t ldd, const void* src, int64_t lds, const float* mean, const float* rstd,
                      const void* qg, const void* kg, float* dqg, float* dqb, float* dkg, float* dkb,
                      int accumulate, int T_, int H, void* ws, ColFinal* fin, hipStream_t s) {
  const int64_t rows = (int64_t)T_ * 2 * H;
  const int blocks = (int)std::min<int64_t>(kQkBwdBlocks, cdiv(rows, 256 / pow2_ceil(DH / 8)));
  float* part = static_cast<float*>(ws);
  KernelInfo ki{sizeof(T) == 2 ? "qkln_bwd_kernel<bf16>" : "qkln_bwd_kernel<f32>", 12.0 * rows * DH,
                3.0 * rows * DH * sizeof(T)};
  ORBIT_TRY(launch(ki, qkln_bwd_kernel<T, DH>, dim3(blocks), dim3(256), 0, s, (T*)d, ldd, (const T*)src, lds,
                   mean, rstd, (const T*)qg, (const T*)kg, T_, H, H * DH, part));
  ColFinal own;
  ColFinal& f = fin ? *fin : own;
  float* outs[4] = {dqg, dqb, dkg, dkb};
  for (int k = 0; k < 4; ++k) f.add(part + k * DH, 4 * DH, blocks, DH, outs[k]);
  return fin ? ORBIT_OK : own.run(accumulate, s);
}

}  // namespace

orbit_status layernorm_fwd(orbit_dtype dt, const void* x, int64_t ldx, const void* g, const void* b, void* y,
                           int64_t ldy, float* mean, float* rstd, int rows, int n, float eps, hipStream_t s) {
  if (dt == ORBIT_BF16) return ln_fwd_dispatch<bf16>(x, ldx, g, b, y, ldy, mean, rstd, rows, n, eps, s);
  return ln_fwd_dispatch<float>(x, ldx, g, b, y, ldy, mean, rstd, rows, n, eps, s);
}

// ---- column sums: host side ------------------------------------------------
int colsum_chunks(int rows) { return rows > 0 ? (int)cdiv(rows, cs_rows_per_chunk(rows)) : 0; }

size_t colsum_part_bytes(int rows, int n, bool ln, int batch) {
  return align_up((size_t)batch * (ln ? 2 : 1) * colsum_chunks(rows) * (size_t)n * sizeof(float));
}

orbit_status colsum_partials(orbit_dtype dt, ColJob* jobs, int njobs, int rows, hipStream_t s) {
  if (njobs <= 0 || rows <= 0) return ORBIT_OK;
  if (njobs > kColMaxJobs) {
    set_error("colsum: %d jobs exceed the limit of %d", njobs, kColMaxJobs);
    return ORBIT_E_ARG;
  }
  CsArgs a{};
  a.njobs = njobs;
  a.rows = rows;
  a.rpc = cs_rows_per_chunk(rows);
  a.chunks = (int)cdiv(rows, a.rpc);
  int cb = 0, maxb = 1;
  double bytes = 0;
  for (int j = 0; j < njobs; ++j) {
    const ColJob& J = jobs[j];
    const int batch = std::max(1, J.batch);
    CsJobK& K = a.job[j];
    K.src = J.src; K.ld = J.ld; K.sbatch = J.sbatch;
    K.x = J.x; K.ldx = J.ldx; K.sxbatch = J.sxbatch; K.mean = J.mean; K.rstd = J.rstd;
    K.part = J.part; K.spart = (int64_t)(J.x ? 2 : 1) * a.chunks * J.n;
    K.n = J.n; K.cb0 = cb; K.batch = batch;
    cb += (int)cdiv(J.n, kCsCols);
    maxb = std::max(maxb, batch);
    bytes += (J.x ? 2.0 : 1.0) * batch * rows * (double)J.n * (dt == ORBIT_BF16 ? 2 : 4);
  }
  const dim3 grid((unsigned)cb, (unsigned)a.chunks, (unsigned)maxb);
  KernelInfo ki{dt == ORBIT_BF16 ? "colsum_partials<bf16>" : "colsum_partials<f32>", 0.0, bytes};
  if (dt == ORBIT_BF16) return launch(ki, colsum_partials_kernel<bf16>, grid, dim3(1024), 0, s, a);
  return launch(ki, colsum_partials_kernel<float>, grid, dim3(1024), 0, s, a);
}

void ColFinal::add(const float* part, int64_t ldp, int chunks, int n, float* out) {
  if (!out || n <= 0) return;
  Item it{part, ldp, out, chunks, n};
  items.push_back(it);
}

void ColFinal::add_job(const ColJob& J, int rows) {
  const int ch = colsum_chunks(rows);
  const int batch = std::max(1, J.batch);
  for (int b = 0; b < batch; ++b) {
    const float* p = J.part + (int64_t)b * (J.x ? 2 : 1) * ch * J.n;
    add(p, J.n, ch, J.n, J.out_sum ? J.out_sum + (int64_t)b * J.sout : nullptr);
    if (J.x) add(p + (int64_t)ch * J.n, J.n, ch, J.n, J.out_xsum ? J.out_xsum + (int64_t)b * J.sout : nullptr);
  }
}

orbit_status ColFinal::run(int accumulate, hipStream_t s) {
  // items are independent (each writes its own output), so a launch takes up
  // to kColMaxFinal items of one kind (many or few chunks) in any order
  for (int pass = 0; pass < 2; ++pass) {
    const bool many = pass == 0;
    const int el = many ? 16 : 256;
    size_t i = 0;
    for (;;) {
      CsFinalArgs a{};
      a.accumulate = accumulate;
      int64_t cb = 0;
      double bytes = 0;
      for (; i < items.size() && a.nitems < kColMaxFinal; ++i) {
        if ((items[i].chunks > 8) != many) continue;
        const Item& it = items[i];
        CsFinalK& K = a.item[a.nitems++];
        K.part = it.part; K.ldp = it.ldp; K.out = it.out; K.chunks = it.chunks; K.n = it.n; K.cb0 = (int)cb;
        cb += cdiv(it.n, el);
        bytes += 4.0 * it.chunks * it.n;
      }
      if (a.nitems == 0) break;
      KernelInfo kf{"colsum_final", 0.0, bytes};
      if (many) {
        ORBIT_TRY(launch(kf, colsum_final_kernel<16>, dim3((unsigned)cb), dim3(256), 0, s, a));
      } else {
        ORBIT_TRY(launch(kf, colsum_final_kernel<1>, dim3((unsigned)cb), dim3(256), 0, s, a));
      }
    }
  }
  items.clear();
  return ORBIT_OK;
}

size_t colsum_workspace_bytes(int rows, int n) { return colsum_part_bytes(rows, n, true, 1); }

orbit_status colsum(orbit_dtype dt, const void* dy, int64_t lddy, int rows, int n, const void* x, int64_t ldx,
                    const float* mean, const float* rstd, float* out_sum, float* out_xsum, int accumulate,
                    void* ws, hipStream_t s) {
  if (rows <= 0 || n <= 0) return ORBIT_OK;
  if (rows <= kCsThinRows && !x && n % 8 == 0 && lddy % 8 == 0 && (reinterpret_cast<uintptr_t>(out_sum) & 15) == 0 &&
      (reinterpret_cast<uintptr_t>(dy) & 15) == 0) {
    if (!out_sum) return ORBIT_OK;
    const dim3 grid((unsigned)cdiv((int64_t)n, 8 * 256));
    KernelInfo ki{dt == ORBIT_BF16 ? "colsum_thin<bf16>" : "colsum_thin<f32>", 0.0,
                  (double)rows * n * (dt == ORBIT_BF16 ? 2 : 4) + (accumulate ? 8.0 : 4.0) * n};
    if (dt == ORBIT_BF16)
      return launch(ki, colsum_thin_kernel<bf16>, grid, dim3(256), 0, s, static_cast<const bf16*>(dy), lddy, rows,
                    (int64_t)n, out_sum, accumulate);
    return launch(ki, colsum_thin_kernel<float>, grid, dim3(256), 0, s, static_cast<const float*>(dy), lddy, rows,
                  (int64_t)n, out_sum, accumulate);
  }
  ColJob J{};
  J.src = dy; J.ld = lddy; J.n = n;
  J.x = x; J.ldx = ldx; J.mean = mean; J.rstd = rstd;
  J.out_sum = out_sum; J.out_xsum = x ? out_xsum : nullptr;
  J.part = static_cast<float*>(ws);
  ORBIT_TRY(colsum_partials(dt, &J, 1, rows, s));
  ColFinal f;
  f.add_job(J, rows);
  return f.run(accumulate, s);
}

// ---- LayerNorm backward with its column sums: host side ---------------------
int ln_cols_nch(int n) { return n <= 8192 ? 2 : 4; }
int ln_cols_tpr(int n) { return (int)(cdiv(cdiv(n, 8 * ln_cols_nch(n)), 64) * 64); }
// rows per chunk: 16, or 8 where 16-row chunks would leave CUs without a block
int ln_cols_rpb(int rows) { return cdiv(rows, 16) >= 256 ? 16 : 8; }

size_t ln_bwd_cols_part_bytes(int rows, int n, bool osum) {
  return align_up((size_t)(osum ? 3 : 2) * cdiv(rows, ln_cols_rpb(rows)) * (size_t)n * sizeof(float));
}

orbit_status layernorm_bwd_cols(orbit_dtype dt, const void* dy, int64_t lddy, const void* x, int64_t ldx,
                                const float* mean, const float* rstd, const void* g, const void* dres, void* dx,
                                int64_t lddx, int rows, int n, float* part, float* out_b, float* out_g,
                                float* out_o, ColFinal& fin, hipStream_t s) {
  if (rows <= 0 || n <= 0) return ORBIT_OK;
  if (n % 8 != 0 || n > 16384) {
    set_error("layernorm_bwd_cols: row length %d must be a multiple of 8 and at most 16384", n);
    return ORBIT_E_UNSUPPORTED;
  }
  LnColArgs a{};
  a.dy = dy; a.x = x; a.g = g; a.dres = dres; a.dx = dx; a.mean = mean; a.rstd = rstd;
  a.lddy = lddy; a.ldx = ldx; a.lddx = lddx; a.part = part; a.rows = rows; a.n = n;
  a.tpr = ln_cols_tpr(n);
  a.rpb = ln_cols_rpb(rows);
  const int G = 512 / a.tpr;
  const int chunks = (int)cdiv(rows, a.rpb);
  const bool osum = out_o != nullptr;
  const double e = dt == ORBIT_BF16 ? 2.0 : 4.0;
  KernelInfo ki{dt == ORBIT_BF16 ? "ln_bwd_cols<bf16>" : "ln_bwd_cols<f32>", 14.0 * rows * n,
                (dres ? 4.0 : 3.0) * rows * n * e + (osum ? 3.0 : 2.0) * chunks * n * 4.0};
  const dim3 grid((unsigned)chunks), block((unsigned)(G * a.tpr));
#define LNC(TT, C, O) ORBIT_TRY(launch(ki, ln_bwd_cols_kernel<TT, C, O>, grid, block, 0, s, a))
  const bool wide = ln_cols_nch(n) == 4;
  if (dt == ORBIT_BF16) {
    if (wide) { if (osum) LNC(bf16, 4, true); else LNC(bf16, 4, false); }
    else { if (osum) LNC(bf16, 2, true); else LNC(bf16, 2, false); }
  } else {
    if (wide) { if (osum) LNC(float, 4, true); else LNC(float, 4, false); }
    else { if (osum) LNC(float, 2, true); else LNC(float, 2, false); }
  }
#undef LNC
  fin.add(part, n, chunks, n, out_b);
  fin.add(part + (int64_t)chunks * n, n, chunks, n, out_g);
  if (osum) fin.add(part + (int64_t)2 * chunks * n, n, chunks, n, out_o);
  return ORBIT_OK;
}

orbit_status colsum_f32(const float* dy, int64_t lddy, int rows, int n, float* out_sum, int accumulate, void* ws,
                        hipStream_t s) {
  return colsum(ORBIT_F32, dy, lddy, rows, n, nullptr, 0, nullptr, nullptr, out_sum, nullptr, accumulate, ws, s);
}

orbit_status qk_norm_fwd(orbit_dtype dt, const void* src, int64_t lds, void* dst, int64_t ldd, const void* qg,
                         const void* qb, const void* kg, const void* kb, float* mean, float* rstd, int T_, int H,
                         int dh, float eps, hipStream_t s) {
  if ((int64_t)T_ * 2 * H >= ((int64_t)1 << 31)) {
    set_error("qk_norm: %d tokens x %d heads exceed 2^31 head rows", T_, H);
    return ORBIT_E_UNSUPPORTED;
  }
#define QKF(TT, D) return qk_fwd_t<TT, D>(src, lds, dst, ldd, qg, qb, kg, kb, mean, rstd, T_, H, eps, s)
  if (dt == ORBIT_BF16) {
    if (dh == 32) QKF(bf16, 32);
    if (dh == 64) QKF(bf16, 64);
    if (dh == 128) QKF(bf16, 128);
    if (dh == 192) QKF(bf16, 192);
    if (dh == 256) QKF(bf16, 256);
  } else {
    if (dh == 32) QKF(float, 32);
    if (dh == 64) QKF(float, 64);
    if (dh == 128) QKF(float, 128);
  }
#undef QKF
  set_error("qk_norm: head_dim %d unsupported", dh);
  return ORBIT_E_UNSUPPORTED;
}

size_t qk_norm_bwd_workspace_bytes(int dh) { return align_up((size_t)kQkBwdBlocks * 4 * dh * sizeof(float)); }

orbit_status qk_norm_bwd(orbit_dtype dt, void* d, int64_t ldd, const void* src, int64_t lds, const float* mean,
                         const float* rstd, const void* qg, const void* kg, float* dqg, float* dqb, float* dkg,
                         float* dkb, int accumulate, int T_, int H, int dh, void* ws, ColFinal* fin,
                         hipStream_t s) {
  if ((int64_t)T_ * 2 * H >= ((int64_t)1 << 31)) {
    set_error("qk_norm: %d tokens x %d heads exceed 2^31 head rows", T_, H);
    return ORBIT_E_UNSUPPORTED;
  }
#define QKB(TT, D) \
  return qk_bwd_t<TT, D>(d, ldd, src, lds, mean, rstd, qg, kg, dqg, dqb, dkg, dkb, accumulate, T_, H, ws, fin, s)
  if (dt == ORBIT_BF16) {
    if (dh == 32) QKB(bf16, 32);
    if (dh == 64) QKB(bf16, 64);
    if (dh == 128) QKB(bf16, 128);
    if (dh == 192) QKB(bf16, 192);
    if (dh == 256) QKB(bf16, 256);
  } else {
    if (dh == 32) QKB(float, 32);
    if (dh == 64) QKB(float, 64);
    if (dh == 128) QKB(float, 128);
  }
#undef QKB
  set_error("qk_norm: head_dim %d unsupported", dh);
  return ORBIT_E_UNSUPPORTED;
}

orbit_status cast_from_f32(orbit_dtype dt, const float* src, void* dst, int64_t n, hipStream_t s) {
  KernelInfo ki{"cast_kernel", 0.0, (4.0 + (dt == ORBIT_BF16 ? 2 : 4)) * n};
  if (dt == ORBIT_BF16) return launch(ki, cast_kernel<bf16>, dim3(grid1d(n)), dim3(256), 0, s, src, (bf16*)dst, n);
  return launch(ki, cast_kernel<float>, dim3(grid1d(n)), dim3(256), 0, s, src, (float*)dst, n);
}

orbit_status axpy_f32(const float* src, float* dst, int64_t n, int accumulate, hipStream_t s) {
  KernelInfo ki{"axpy_kernel", 0.0, 12.0 * n};
  return launch(ki, axpy_kernel, dim3(grid1d(n)), dim3(256), 0, s, src, dst, n, accumulate);
}

orbit_status fill_f32(float* dst, int64_t n, float v, hipStream_t s) {
  KernelInfo ki{"fill_kernel", 0.0, 4.0 * n};
  return launch(ki, fill_kernel, dim3(grid1d(n)), dim3(256), 0, s, dst, n, v);
}

}  // namespace orbit
