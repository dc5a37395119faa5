// Fused multi-head self-attention O = softmax(q k^T / sqrt(dh)) v (no mask),
// forward with an online softmax held in registers and backward in the
// two-kernel deterministic form (K/V-major kernel for dK, dV; Q-major kernel
// for dQ; no atomics), on 32x32x16 MFMA tiles.
//
// Layout trick: the forward computes S^T = K Q^T, so each lane owns one query
// (accumulator column) and the probabilities P^T come out of the accumulator
// already in the B-operand layout of O^T = V^T P^T; V is staged transposed in
// LDS so its fragments are two 8-byte reads. The backward uses the same idea
// in both orientations (see the per-kernel comments).
#include <algorithm>
#include <type_traits>

#include "kernels.h"
#include "tile.h"

namespace orbit {
namespace {

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.69314718055994531f;

struct FwdArgs {
  const void *q, *k, *v;
  void* o;
  float* lse;
  float* o32;  // optional float32 copy of O (consistent softmax-backward row sums)
  int64_t ldq, ldk, ldv, ldo, ldo32;
  int H, L;
  float sl2;  // log2(e) / sqrt(dh)
  // key split (ns > 1): block column = split * query tiles + query tile; the
  // float32 partials go to `part` ([ns][rows][dh] outputs, then [ns][rows]
  // reference maxima and [ns][rows] row sums; rows = B H L, (sample, head,
  // query) order) and attn_fwd_merge finishes O, o32 and lse
  int B = 0, ns = 1;
  float* part = nullptr;
};

// lane l: fragment slot j (0..7) of lane group g = l/32 in a 16-deep K step of
// an accumulator-derived operand covers index (j/4)*8 + g*4 + j%4 of the step.
// read that fragment from a transposed LDS row: two runs of 4.
template <typename T>
ORBIT_DEV void ld_frag_acc_order(Frag<T>& f, const T* row, int kstep, int g) {
  ld_frag2(f, row + kstep * 16 + g * 4, row + kstep * 16 + 8 + g * 4);
}

// fragment of 8 values of an accumulator (registers base..base+7) as T
template <typename T>
ORBIT_DEV void acc_frag(Frag<T>& f, const f32x16& a, int base) {
  float t[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) t[j] = a[base + j];
  frag_from(f, t);
}

// store 4 consecutive floats as T
template <typename T>
ORBIT_DEV void st4(T* p, float a, float b, float c, float d) {
  if constexpr (sizeof(T) == 2) {
    bf16x4 v = {(bf16)a, (bf16)b, (bf16)c, (bf16)d};
    *reinterpret_cast<bf16x4*>(p) = v;
  } else {
    f32x4 v = {a, b, c, d};
    *reinterpret_cast<f32x4*>(p) = v;
  }
}

// ---------------------------------------------------------------------------
// forward: 4 waves x 32 queries per block, 64-key tiles
// ---------------------------------------------------------------------------
template <typename T, int DH>
__global__ void __launch_bounds__(256) attn_fwd_kernel(FwdArgs a) {
  constexpr int KT = 64;
  constexpr int E = 16 / (int)sizeof(T);
  using LK = TileLoader<T, KT, DH, 256, true>;    // K rows  [kv][c]
  using LV = TileLoader<T, DH, KT, 256, false>;   // V^T     [c][kv]
  constexpr int KP = LK::PITCH, VP = LV::PITCH;
  __shared__ __attribute__((aligned(16))) T ks[2][KT * KP];
  __shared__ __attribute__((aligned(16))) T vs[2][DH * VP];

  const int tid = threadIdx.x, lane = tid & 63, g = lane >> 5, wave = tid >> 6;
  const int h = blockIdx.y, b = blockIdx.z;
  const int L = a.L;
  const int64_t row0 = (int64_t)b * L;
  const T* Q = static_cast<const T*>(a.q) + row0 * a.ldq + h * DH;
  const T* K = static_cast<const T*>(a.k) + row0 * a.ldk + h * DH;
  const T* V = static_cast<const T*>(a.v) + row0 * a.ldv + h * DH;

  const int qi = blockIdx.x * 128 + wave * 32 + (lane & 31);
  Frag<T> qf[DH / 16];
#pragma unroll
  for (int kk = 0; kk < DH / 16; ++kk) {
    if (qi < L) ld_frag(qf[kk], Q + (int64_t)qi * a.ldq + kk * 16 + g * 8);
    else {
      float z[8] = {0, 0, 0, 0, 0, 0, 0, 0};
      frag_from(qf[kk], z);
    }
  }

  f32x16 o[DH / 32];
#pragma unroll
  for (int c = 0; c < DH / 32; ++c)
#pragma unroll
    for (int v = 0; v < 16; ++v) o[c][v] = 0.f;
  float m = -INFINITY, lsum = 0.f;

  LK lk;
  LV lv;
  const int nt = (L + KT - 1) / KT;
  lk.load(K, nullptr, 0, a.ldk, 0, L, 0, DH, tid);
  lv.load(V, nullptr, 0, a.ldv, 0, DH, 0, L, tid);
  lk.store(ks[0], tid);
  lv.store(vs[0], tid);
  __syncthreads();

  for (int jt = 0; jt < nt; ++jt) {
    const int cur = jt & 1;
    if (jt + 1 < nt) {
      const int j0 = (jt + 1) * KT;
      lk.load(K, nullptr, 0, a.ldk, j0, L, 0, DH, tid);
      lv.load(V + (int64_t)j0 * a.ldv, nullptr, 0, a.ldv, 0, DH, 0, L - j0, tid);
    }
    const T* Ks = ks[cur];
    const T* Vs = vs[cur];
    // S^T[kv][q] for 64 keys: two 32-row tiles
    f32x16 s[2];
#pragma unroll
    for (int mt = 0; mt < 2; ++mt) {
#pragma unroll
      for (int v = 0; v < 16; ++v) s[mt][v] = 0.f;
#pragma unroll
      for (int kk = 0; kk < DH / 16; ++kk) {
        Frag<T> kf;
        ld_frag(kf, Ks + (mt * 32 + (lane & 31)) * KP + kk * 16 + g * 8);
        mma16(s[mt], kf, qf[kk]);
      }
    }
    // online softmax over this tile (log2 domain); lane owns query qi and,
    // with its partner lane l ^ 32, the running max m and sum of that query
    const int jbase = jt * KT;
    if (jbase + KT > L) {
#pragma unroll
      for (int mt = 0; mt < 2; ++mt)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int kv = jbase + mt * 32 + (v >> 2) * 8 + g * 4 + (v & 3);
          if (kv >= L) s[mt][v] = -INFINITY;
        }
    }
    float mloc = -INFINITY;
#pragma unroll
    for (int mt = 0; mt < 2; ++mt)
#pragma unroll
      for (int v = 0; v < 16; ++v) mloc = fmaxf(mloc, s[mt][v]);
    mloc = fmaxf(mloc, __shfl_xor(mloc, 32, 64));
    const float mnew = fmaxf(m, mloc * a.sl2);
    // rescale O and the sum only when some query's maximum moved
    if (__ballot(mnew > m) != 0) {
      const float alpha = __builtin_amdgcn_exp2f(m - mnew);
      lsum *= alpha;
#pragma unroll
      for (int c = 0; c < DH / 32; ++c)
#pragma unroll
        for (int v = 0; v < 16; ++v) o[c][v] *= alpha;
      m = mnew;
    }
    float ps = 0.f;
#pragma unroll
    for (int mt = 0; mt < 2; ++mt)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const float p = __builtin_amdgcn_exp2f(fmaf(s[mt][v], a.sl2, -m));
        s[mt][v] = p;
        ps += p;
      }
    lsum += ps;
    // O^T[c][q] += V^T[c][kv] P^T[kv][q]
#pragma unroll
    for (int kk = 0; kk < KT / 16; ++kk) {
      Frag<T> pf;
      acc_frag(pf, s[kk >> 1], (kk & 1) * 8);
#pragma unroll
      for (int c = 0; c < DH / 32; ++c) {
        Frag<T> vf;
        ld_frag_acc_order(vf, Vs + (c * 32 + (lane & 31)) * VP, kk, g);
        mma16(o[c], vf, pf);
      }
    }
    if (jt + 1 < nt) {
      lk.store(ks[cur ^ 1], tid);
      lv.store(vs[cur ^ 1], tid);
    }
    __syncthreads();
  }

  const float ltot = lsum + __shfl_xor(lsum, 32, 64);
  if (qi < L) {
    const float inv = 1.f / ltot;
    T* O = static_cast<T*>(a.o) + (row0 + qi) * a.ldo + h * DH;
#pragma unroll
    for (int c = 0; c < DH / 32; ++c)
#pragma unroll
      for (int r4 = 0; r4 < 4; ++r4) {
        const int col = c * 32 + r4 * 8 + g * 4;
        st4(O + col, o[c][r4 * 4] * inv, o[c][r4 * 4 + 1] * inv, o[c][r4 * 4 + 2] * inv,
            o[c][r4 * 4 + 3] * inv);
      }
    if (a.o32) {
      float* O32 = a.o32 + (row0 + qi) * a.ldo32 + h * DH;
#pragma unroll
      for (int c = 0; c < DH / 32; ++c)
#pragma unroll
        for (int r4 = 0; r4 < 4; ++r4) {
          const int col = c * 32 + r4 * 8 + g * 4;
          st4(O32 + col, o[c][r4 * 4] * inv, o[c][r4 * 4 + 1] * inv, o[c][r4 * 4 + 2] * inv,
              o[c][r4 * 4 + 3] * inv);
        }
    }
    if (g == 0) a.lse[((int64_t)b * a.H + h) * L + qi] = (m + __log2f(ltot)) * kLn2;
  }
  (void)E;
}

// ---------------------------------------------------------------------------
// backward preprocess: D[b,h,i] = sum_c dO[i,c] O[i,c]
// ---------------------------------------------------------------------------
template <typename T, typename OT, int DH>
__global__ void __launch_bounds__(256) attn_bwd_pre(const OT* __restrict__ o, int64_t ldo, const T* __restrict__ dO,
                                                    int64_t lddo, float* __restrict__ D, int B, int H, int L) {
  // a row's DH / 8 chunks on the next power of two lanes (head_dim 192: 24 of 32)
  constexpr int CH = DH / 8, G = pow2_ceil(CH);
  const int li = threadIdx.x % G;
  // row (t, h), 32-bit (the host keeps B * L * H below 2^31)
  const unsigned row = blockIdx.x * (256u / G) + threadIdx.x / G;
  const bool valid = row < (unsigned)B * L * H;
  const unsigned t = valid ? row / (unsigned)H : 0u;
  const int h = (int)(row - t * (unsigned)H);
  float s = 0.f;
  if (valid && li < CH) {
    float a8[8], b8[8];
    const OT* op = o + (int64_t)t * ldo + h * DH + li * 8;
    const T* dp = dO + (int64_t)t * lddo + h * DH + li * 8;
    unpack(ld128(op), a8, (OT*)nullptr);
    unpack(ld128(dp), b8, (T*)nullptr);
    if constexpr (sizeof(OT) == 4) unpack(ld128(op + 4), a8 + 4, (OT*)nullptr);
    if constexpr (sizeof(T) == 4) unpack(ld128(dp + 4), b8 + 4, (T*)nullptr);
#pragma unroll
    for (int i = 0; i < 8; ++i) s += a8[i] * b8[i];
  }
#pragma unroll
  for (int off = G / 2; off >= 1; off >>= 1) s += __shfl_xor(s, off, 64);
  if (valid && li == 0) {
    const unsigned bb = t / (unsigned)L, l = t - bb * (unsigned)L;
    D[((int64_t)bb * H + h) * L + l] = s;
  }
}

struct BwdArgs {
  const void *q, *k, *v, *dO;
  const float *lse, *D;
  const float *qsum, *ksum;  // per (sample, head, feature) sums of q and k over the sequence
  void *dq, *dk, *dv;
  int64_t ldq, ldk, ldv, lddo, ldg;
  int H, L;
  float sl2, scale;  // log2(e)/sqrt(dh), 1/sqrt(dh)
  // sweep split (ns > 1): block column = split * tiles + tile; each split
  // writes float32 partial sums to `part` (rows = B H L) and a merge kernel
  // finishes the gradients
  int B = 0, ns = 1;
  float* part = nullptr;
};

// Stage a 32-row x DH tile X[r][c] (rows r0.., valid < rlim) into LDS twice:
// row-major Xs[r][c] (pitch DH+E) and transposed Xt[c][r] (pitch 32+E).
template <typename T, int DH, int NT>
struct DualStage {
  static constexpr int E = 16 / (int)sizeof(T);
  static constexpr int RP = DH + E, TP = 32 + E;
  static constexpr int NU = (32 / 4) * (DH / E);  // units of 4 rows x E columns
  static constexpr int PER = (NU + NT - 1) / NT;
  U128 r[PER * 4];
  ORBIT_DEV void load(const T* X, int64_t ld, int r0, int rlim, int tid) {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int u = tid + i * NT;
      const int rg = u / (DH / E), cc = u % (DH / E);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int rr = r0 + rg * 4 + j;
        r[i * 4 + j] = (u < NU && rr < rlim) ? ld128(X + (int64_t)rr * ld + cc * E) : zero128();
      }
    }
  }
  // Xt gets X - mean[column] when mean is given
  ORBIT_DEV void store(T* Xs, T* Xt, int tid, const float* mean) const {
    using TL = TileLoader<T, DH, 32, NT, false>;
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int u = tid + i * NT;
      if (u >= NU) continue;
      const int rg = u / (DH / E), cc = u % (DH / E);
#pragma unroll
      for (int j = 0; j < 4; ++j) st128(Xs + (rg * 4 + j) * RP + cc * E, r[i * 4 + j]);
      if (mean) TL::store_transposed_sub(Xt + (cc * E) * TP + rg * 4, &r[i * 4], mean + cc * E);
      else TL::store_transposed(Xt + (cc * E) * TP + rg * 4, &r[i * 4]);
    }
  }
};

// ---------------------------------------------------------------------------
// backward, K/V-major: each wave owns 32 keys (K, V fragments in registers)
// and sweeps all queries in tiles of 32:
//   S = Q K^T (lane <-> key column), P = exp(S/sqrt(dh) - lse), dP = dO V^T,
//   dS = P (dP - D);  dV^T += dO^T P,  dK^T += Q^T dS  (P, dS feed the MFMA
//   B operand straight from the accumulator; dO^T, Q^T are staged transposed).
// ---------------------------------------------------------------------------
template <typename T, int DH>
__global__ void __launch_bounds__(256) attn_bwd_dkdv(BwdArgs a) {
  using DS = DualStage<T, DH, 256>;
  constexpr int RP = DS::RP, TP = DS::TP;
  __shared__ __attribute__((aligned(16))) T qs[32 * RP];
  __shared__ __attribute__((aligned(16))) T qt[DH * TP];
  __shared__ __attribute__((aligned(16))) T ds_[32 * RP];
  __shared__ __attribute__((aligned(16))) T dt[DH * TP];
  __shared__ float lse_s[32], d_s[32];
  __shared__ float qbar[DH];

  const int tid = threadIdx.x, lane = tid & 63, g = lane >> 5, wave = tid >> 6;
  const int h = blockIdx.y, b = blockIdx.z;
  const int L = a.L;
  const int64_t row0 = (int64_t)b * L;
  if (tid < DH) qbar[tid] = a.qsum[((int64_t)b * a.H + h) * DH + tid] / (float)L;
  const T* Q = static_cast<const T*>(a.q) + row0 * a.ldq + h * DH;
  const T* K = static_cast<const T*>(a.k) + row0 * a.ldk + h * DH;
  const T* V = static_cast<const T*>(a.v) + row0 * a.ldv + h * DH;
  const T* dO = static_cast<const T*>(a.dO) + row0 * a.lddo + h * DH;
  const float* lse = a.lse + ((int64_t)b * a.H + h) * L;
  const float* Dv = a.D + ((int64_t)b * a.H + h) * L;

  const int kv = blockIdx.x * 128 + wave * 32 + (lane & 31);
  Frag<T> kf[DH / 16], vf[DH / 16];
#pragma unroll
  for (int kk = 0; kk < DH / 16; ++kk) {
    if (kv < L) {
      ld_frag(kf[kk], K + (int64_t)kv * a.ldk + kk * 16 + g * 8);
      ld_frag(vf[kk], V + (int64_t)kv * a.ldv + kk * 16 + g * 8);
    } else {
      float z[8] = {0, 0, 0, 0, 0, 0, 0, 0};
      frag_from(kf[kk], z);
      frag_from(vf[kk], z);
    }
  }
  f32x16 dvt[DH / 32], dkt[DH / 32];
#pragma unroll
  for (int c = 0; c < DH / 32; ++c)
#pragma unroll
    for (int v = 0; v < 16; ++v) dvt[c][v] = dkt[c][v] = 0.f;

  // dK_j = sum_i dS_ij q_i = sum_i dS_ij (q_i - qbar) + qbar sum_i dS_ij: the
  // product runs on centred queries (small when the queries are alike) and
  // the rank-one remainder is added in float32 from the exact column sums.
  float cs = 0.f;
  DS sq, sd;
  const int nq = (L + 31) / 32;
  // the next query tile (and its softmax statistics) is loaded while the
  // current one is multiplied
  sq.load(Q, a.ldq, 0, L, tid);
  sd.load(dO, a.lddo, 0, L, tid);
  float lse_n = 0.f, d_n = 0.f;
  if (tid < 32) {
    lse_n = tid < L ? lse[tid] * kLog2e : INFINITY;
    d_n = tid < L ? Dv[tid] : 0.f;
  }
  for (int it = 0; it < nq; ++it) {
    __syncthreads();  // previous tile fully consumed (and qbar visible)
    sq.store(qs, qt, tid, qbar);
    sd.store(ds_, dt, tid, nullptr);
    if (tid < 32) {
      lse_s[tid] = lse_n;
      d_s[tid] = d_n;
    }
    __syncthreads();
    if (it + 1 < nq) {
      const int q1 = (it + 1) * 32;
      sq.load(Q, a.ldq, q1, L, tid);
      sd.load(dO, a.lddo, q1, L, tid);
      if (tid < 32) {
        lse_n = q1 + tid < L ? lse[q1 + tid] * kLog2e : INFINITY;
        d_n = q1 + tid < L ? Dv[q1 + tid] : 0.f;
      }
    }

    f32x16 s, dp;
#pragma unroll
    for (int v = 0; v < 16; ++v) s[v] = dp[v] = 0.f;
#pragma unroll
    for (int kk = 0; kk < DH / 16; ++kk) {
      Frag<T> af;
      ld_frag(af, qs + (lane & 31) * RP + kk * 16 + g * 8);
      mma16(s, af, kf[kk]);
      ld_frag(af, ds_ + (lane & 31) * RP + kk * 16 + g * 8);
      mma16(dp, af, vf[kk]);
    }
    // rows: query 8*(v/4) + 4g + v%4 of the tile; column: this lane's key
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int qr = (v >> 2) * 8 + g * 4 + (v & 3);
      const float p = __builtin_amdgcn_exp2f(fmaf(s[v], a.sl2, -lse_s[qr]));
      s[v] = p;
      dp[v] = p * (dp[v] - d_s[qr]);
      cs += dp[v];
    }
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      Frag<T> pf, sf;
      acc_frag(pf, s, kk * 8);
      acc_frag(sf, dp, kk * 8);
#pragma unroll
      for (int c = 0; c < DH / 32; ++c) {
        Frag<T> af;
        ld_frag_acc_order(af, dt + (c * 32 + (lane & 31)) * TP, kk, g);
        mma16(dvt[c], af, pf);
        ld_frag_acc_order(af, qt + (c * 32 + (lane & 31)) * TP, kk, g);
        mma16(dkt[c], af, sf);
      }
    }
  }

  cs += __shfl_xor(cs, 32, 64);
  if (kv < L) {
    T* dK = static_cast<T*>(a.dk) + (row0 + kv) * a.ldg + h * DH;
    T* dV = static_cast<T*>(a.dv) + (row0 + kv) * a.ldg + h * DH;
#pragma unroll
    for (int c = 0; c < DH / 32; ++c)
#pragma unroll
      for (int r4 = 0; r4 < 4; ++r4) {
        const int col = c * 32 + r4 * 8 + g * 4;
        st4(dK + col, (dkt[c][r4 * 4] + qbar[col] * cs) * a.scale, (dkt[c][r4 * 4 + 1] + qbar[col + 1] * cs) * a.scale,
            (dkt[c][r4 * 4 + 2] + qbar[col + 2] * cs) * a.scale, (dkt[c][r4 * 4 + 3] + qbar[col + 3] * cs) * a.scale);
        st4(dV + col, dvt[c][r4 * 4], dvt[c][r4 * 4 + 1], dvt[c][r4 * 4 + 2], dvt[c][r4 * 4 + 3]);
      }
  }
}

// ---------------------------------------------------------------------------
// backward, Q-major: each wave owns 32 queries (Q, dO fragments in registers)
// and sweeps all keys in tiles of 64:
//   S^T = K Q^T, P^T, dP^T = V dO^T, dS^T = P^T (dP^T - D);  dQ^T += (K - kbar)^T dS^T
// ---------------------------------------------------------------------------
template <typename T, int DH>
__global__ void __launch_bounds__(256) attn_bwd_dq(BwdArgs a) {
  constexpr int KT = 64;
  using LK = TileLoader<T, KT, DH, 256, true>;    // K, V rows [kv][c]
  using LT = TileLoader<T, DH, KT, 256, false>;   // K^T      [c][kv]
  constexpr int KP = LK::PITCH, TP = LT::PITCH;
  __shared__ __attribute__((aligned(16))) T ks[KT * KP];
  __shared__ __attribute__((aligned(16))) T vs[KT * KP];
  __shared__ __attribute__((aligned(16))) T kt[DH * TP];
  __shared__ float kbar[DH];

  const int tid = threadIdx.x, lane = tid & 63, g = lane >> 5, wave = tid >> 6;
  const int h = blockIdx.y, b = blockIdx.z;
  const int L = a.L;
  const int64_t row0 = (int64_t)b * L;
  if (tid < DH) kbar[tid] = a.ksum[((int64_t)b * a.H + h) * DH + tid] / (float)L;
  const T* Q = static_cast<const T*>(a.q) + row0 * a.ldq + h * DH;
  const T* K = static_cast<const T*>(a.k) + row0 * a.ldk + h * DH;
  const T* V = static_cast<const T*>(a.v) + row0 * a.ldv + h * DH;
  const T* dO = static_cast<const T*>(a.dO) + row0 * a.lddo + h * DH;

  const int qi = blockIdx.x * 128 + wave * 32 + (lane & 31);
  Frag<T> qf[DH / 16], of[DH / 16];
#pragma unroll
  for (int kk = 0; kk < DH / 16; ++kk) {
    if (qi < L) {
      ld_frag(qf[kk], Q + (int64_t)qi * a.ldq + kk * 16 + g * 8);
      ld_frag(of[kk], dO + (int64_t)qi * a.lddo + kk * 16 + g * 8);
    } else {
      float z[8] = {0, 0, 0, 0, 0, 0, 0, 0};
      frag_from(qf[kk], z);
      frag_from(of[kk], z);
    }
  }
  const float lse2 = qi < L ? a.lse[((int64_t)b * a.H + h) * L + qi] * kLog2e : INFINITY;
  const float Dq = qi < L ? a.D[((int64_t)b * a.H + h) * L + qi] : 0.f;

  f32x16 dqt[DH / 32];
#pragma unroll
  for (int c = 0; c < DH / 32; ++c)
#pragma unroll
    for (int v = 0; v < 16; ++v) dqt[c][v] = 0.f;

  LK lk, lvv;
  LT lt;
  const int nt = (L + KT - 1) / KT;
  lk.load(K, nullptr, 0, a.ldk, 0, L, 0, DH, tid);
  lvv.load(V, nullptr, 0, a.ldv, 0, L, 0, DH, tid);
  lt.load(K, nullptr, 0, a.ldk, 0, DH, 0, L, tid);
  for (int jt = 0; jt < nt; ++jt) {
    const int j0 = jt * KT;
    __syncthreads();  // previous tile fully consumed (and kbar visible)
    lk.store(ks, tid);
    lvv.store(vs, tid);
    // dQ_i = sum_j dS_ij k_j = sum_j dS_ij (k_j - kbar) since sum_j dS_ij = 0:
    // centred keys keep the product well conditioned when the keys are alike
    lt.store_sub(kt, tid, kbar);
    __syncthreads();
    if (jt + 1 < nt) {  // the next key tile is loaded while this one is multiplied
      const int j1 = j0 + KT;
      lk.load(K, nullptr, 0, a.ldk, j1, L, 0, DH, tid);
      lvv.load(V, nullptr, 0, a.ldv, j1, L, 0, DH, tid);
      lt.load(K + (int64_t)j1 * a.ldk, nullptr, 0, a.ldk, 0, DH, 0, L - j1, tid);
    }

    f32x16 s[2], dp[2];
#pragma unroll
    for (int mt = 0; mt < 2; ++mt) {
#pragma unroll
      for (int v = 0; v < 16; ++v) s[mt][v] = dp[mt][v] = 0.f;
#pragma unroll
      for (int kk = 0; kk < DH / 16; ++kk) {
        Frag<T> af;
        ld_frag(af, ks + (mt * 32 + (lane & 31)) * KP + kk * 16 + g * 8);
        mma16(s[mt], af, qf[kk]);
        ld_frag(af, vs + (mt * 32 + (lane & 31)) * KP + kk * 16 + g * 8);
        mma16(dp[mt], af, of[kk]);
      }
      if (j0 + KT > L) {
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int kvi = j0 + mt * 32 + (v >> 2) * 8 + g * 4 + (v & 3);
          if (kvi >= L) s[mt][v] = -INFINITY;
        }
      }
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const float p = __builtin_amdgcn_exp2f(fmaf(s[mt][v], a.sl2, -lse2));
        dp[mt][v] = p * (dp[mt][v] - Dq);
      }
    }
#pragma unroll
    for (int kk = 0; kk < KT / 16; ++kk) {
      Frag<T> sf;
      acc_frag(sf, dp[kk >> 1], (kk & 1) * 8);
#pragma unroll
      for (int c = 0; c < DH / 32; ++c) {
        Frag<T> af;
        ld_frag_acc_order(af, kt + (c * 32 + (lane & 31)) * TP, kk, g);
        mma16(dqt[c], af, sf);
      }
    }
  }

  if (qi < L) {
    T* dQ = static_cast<T*>(a.dq) + (row0 + qi) * a.ldg + h * DH;
#pragma unroll
    for (int c = 0; c < DH / 32; ++c)
#pragma unroll
      for (int r4 = 0; r4 < 4; ++r4) {
        const int col = c * 32 + r4 * 8 + g * 4;
        st4(dQ + col, dqt[c][r4 * 4] * a.scale, dqt[c][r4 * 4 + 1] * a.scale, dqt[c][r4 * 4 + 2] * a.scale,
            dqt[c][r4 * 4 + 3] * a.scale);
      }
  }
}

// ---------------------------------------------------------------------------
// bf16 kernels with transposing LDS reads (ds_read_b64_tr_b16): every tile is
// staged once, row-major, and the operands that are needed transposed (V^T in
// the forward; dO^T, Q^T and K^T in the backward) are read as MFMA fragments
// straight from that copy. Tiles are double-buffered in LDS (one barrier per
// tile) and the last, partial tile is peeled so the main loop carries no masks.
// ---------------------------------------------------------------------------
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef short s16x8 __attribute__((ext_vector_type(8)));

// A-operand fragment of a matrix stored M-contiguous in LDS (element (k, m) at
// base[k * pitch + m]): rows m = lane % 32, a 16-deep K step in accumulator
// slot order (slot j of lane group g = lane / 32 holds k = (j/4)*8 + 4g + j%4).
// Each 16-lane group reads 4 k-rows x 16 m per transposing read; two reads.
ORBIT_DEV void ld_frag_tr(Frag<bf16>& f, const bf16* base, int pitch, int lane) {
  const int G = lane >> 4, r = lane & 15;
  bf16* p0 = const_cast<bf16*>(base) + (4 * (G >> 1) + (r >> 2)) * pitch + 16 * (G & 1) + 4 * (r & 3);
  bf16* p1 = p0 + 8 * pitch;
  const s16x4 x = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4*)p0);
  const s16x4 y = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4*)p1);
  const s16x8 xy = __builtin_shufflevector(x, y, 0, 1, 2, 3, 4, 5, 6, 7);
  f.v = __builtin_bit_cast(bf16x8, xy);
}

// ROWS consecutive rows of one head's DH-column slice of a bf16 [L][ld]
// matrix, copied global -> registers -> LDS ([row][DH + 8]). The loads go
// through a buffer resource whose extent ends with row L - 1, so rows at or
// past L read as zeros without a branch; a tile's position is a scalar byte
// offset, so advancing costs no vector instructions.
template <int ROWS, int DH>
struct RowTile {
  static constexpr int CPR = DH / 8;  // 16-byte chunks per row
  static constexpr int NCH = ROWS * CPR;
  static constexpr int PER = (NCH + 255) / 256;  // chunks per thread
  // row pitch (elements): 16-byte fragment reads of 16 consecutive rows and
  // transposing reads of 4 k-rows x 64 bytes both hit 64 distinct banks
  static constexpr int PITCH = DH == 128 ? DH + 24 : DH + 8;
  static_assert(NCH % 256 == 0 || NCH % 64 == 0, "whole waves per chunk round");
  typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
  __amdgpu_buffer_rsrc_t rsrc;
  unsigned row_bytes;
  int tid_;
  unsigned voff[PER];
  unsigned lofs[PER];
  u32x4 r[PER];
  ORBIT_DEV void init(const bf16* base, int64_t ld, int L, int tid) {
    row_bytes = (unsigned)(ld * 2);
    tid_ = tid;
    const int extent = (int)(((int64_t)(L - 1) * ld + DH) * 2);
    rsrc = __builtin_amdgcn_make_buffer_rsrc(const_cast<bf16*>(base), 0, extent, 0x00020000);
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int c = tid + i * 256, row = c / CPR, col = c % CPR;
      voff[i] = (unsigned)row * row_bytes + col * 16;
      lofs[i] = (unsigned)(row * PITCH + col * 8);
    }
  }
  ORBIT_DEV void load(int row0) {
    const unsigned so = (unsigned)row0 * row_bytes;
#pragma unroll
    for (int i = 0; i < PER; ++i)
      if (NCH % 256 == 0 || tid_ + i * 256 < NCH) r[i] = __builtin_amdgcn_raw_buffer_load_b128(rsrc, voff[i], so, 0);
  }
  ORBIT_DEV void store(bf16* S) const {
#pragma unroll
    for (int i = 0; i < PER; ++i)
      if (NCH % 256 == 0 || tid_ + i * 256 < NCH) *reinterpret_cast<u32x4*>(S + lofs[i]) = r[i];
  }
};

// ROWS rows of one head's DH-column slices of two bf16 [L][ld] matrices
// (sharing a row range), copied by the buffer unit straight into LDS in the
// RowTile layout, [row][PITCH], with no staging registers: 1 KB wave copies,
// copy c of a matrix filling 16-byte chunks 64c .. 64c + 63 of its area. The
// copies are dealt round-robin over NW waves. A chunk in a row's padding or
// in the last copy's slack, and every chunk of a row at or past L, is read at
// an offset at or past the resource's extent, which the range check turns
// into zeros (the copy then writes zeros).
#define ORBIT_LDS __attribute__((address_space(3)))
template <int ROWS, int DH, int NW>
struct DmaRows {
  static constexpr int PITCH = RowTile<ROWS, DH>::PITCH;
  static constexpr int CPP = PITCH / 8;               // 16-byte chunks per LDS row
  static constexpr int NC = (ROWS * CPP + 63) / 64;   // copies per matrix
  static constexpr int BYTES = NC * 1024;             // LDS area of one matrix
  static constexpr int PW = (2 * NC + NW - 1) / NW;   // copies per wave (the last may be idle)
  static_assert(PITCH % 8 == 0, "whole chunks per row");
  // (members, not arrays: the copy's matrix depends on the wave, and an
  // array indexed by it would be kept in memory)
  __amdgpu_buffer_rsrc_t rsrc0, rsrc1;
  unsigned rb0, rb1;
  unsigned voff[PW];
  ORBIT_DEV void init(const bf16* x0, int64_t ld0, const bf16* x1, int64_t ld1, int L, int wave, int lane) {
    rb0 = (unsigned)(ld0 * 2);
    rb1 = (unsigned)(ld1 * 2);
    rsrc0 = __builtin_amdgcn_make_buffer_rsrc(const_cast<bf16*>(x0), 0, (int)(((int64_t)(L - 1) * ld0 + DH) * 2),
                                              0x00020000);
    rsrc1 = __builtin_amdgcn_make_buffer_rsrc(const_cast<bf16*>(x1), 0, (int)(((int64_t)(L - 1) * ld1 + DH) * 2),
                                              0x00020000);
#pragma unroll
    for (int i = 0; i < PW; ++i) {
      const int cp = wave + NW * i, c = cp % NC;
      const int p = c * 64 + lane, row = p / CPP, col = p % CPP;
      const bool ok = cp < 2 * NC && row < ROWS && col < DH / 8;
      voff[i] = ok ? (unsigned)row * (cp >= NC ? rb1 : rb0) + col * 16 : 0x80000000u;
    }
  }
  // copies of rows row0 .. row0 + ROWS - 1; matrix m goes to LDS byte
  // address lds + m * BYTES
  ORBIT_DEV void issue(unsigned lds, int row0, int wave) const {
#pragma unroll
    for (int i = 0; i < PW; ++i) {
      const int cp = wave + NW * i;
      if (cp < 2 * NC) {
        const bool m1 = cp >= NC;
        const int c = m1 ? cp - NC : cp;
        dma16(m1 ? rsrc1 : rsrc0, lds + (m1 ? BYTES : 0) + c * 1024, voff[i] + (unsigned)row0 * (m1 ? rb1 : rb0));
      }
    }
  }
};

// sum of the 8 values of a bf16 fragment added to acc (two per instruction)
ORBIT_DEV float frag_sum(const Frag<bf16>& f, float acc) {
  typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
  const bf16x2 one = {(__bf16)1.f, (__bf16)1.f};
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const bf16x2 pr = {f.v[2 * j], f.v[2 * j + 1]};
    acc = __builtin_amdgcn_fdot2_f32_bf16(pr, one, acc, false);
  }
  return acc;
}

// (query or key block, head, sample) of this block, arranged so that all the
// blocks of one (sample, head) run on one XCD and share its L2 for the K/V
// (or Q/dO) tiles they all stream: hardware block ids go round-robin over the
// 8 XCDs, so XCD x takes the (sample, head) pairs x, x + 8, ... in turn. Grids
// whose pair count is not a multiple of 8 keep the plain order.
ORBIT_DEV void attn_block_coords(int& xb, int& h, int& b) {
  const unsigned nx = gridDim.x, ny = gridDim.y, pairs = gridDim.y * gridDim.z;
  if (pairs % 8 == 0) {
    const unsigned lb = blockIdx.x + nx * (blockIdx.y + ny * blockIdx.z);
    const unsigned i = lb / 8, ph = (i / nx) * 8 + lb % 8;
    xb = (int)(i % nx);
    h = (int)(ph % ny);
    b = (int)(ph / ny);
  } else {
    xb = blockIdx.x;
    h = blockIdx.y;
    b = blockIdx.z;
  }
}

// Softmax reference point: scores are exponentiated as exp2(s - m) with m a
// running maximum that is raised only when a new score exceeds it by more than
// this margin (log2 units), so the output is rescaled rarely; the unnormalised
// probabilities stay below 2^margin.
constexpr float kMaxSlack = 8.f;

// four waves per SIMD for head_dim 64 (the kernel fits in 128 VGPRs)
template <int DH>
__global__ void __launch_bounds__(256, DH == 64 ? 4 : 1) attn_fwd_tr(FwdArgs a) {
  using T = bf16;
  constexpr int KT = 64;
  using TL = RowTile<KT, DH>;  // K and V rows [kv][c]
  constexpr int KP = TL::PITCH;
  __shared__ __attribute__((aligned(16))) T ks[2][KT * KP];
  __shared__ __attribute__((aligned(16))) T vs[2][KT * KP];

  const int tid = threadIdx.x, lane = tid & 63, g = lane >> 5, wave = tid >> 6;
  int xb, h, b;
  attn_block_coords(xb, h, b);
  const int L = a.L;
  const int sp = xb / ((L + 127) / 128);  // key split of this block
  xb -= sp * ((L + 127) / 128);
  const int64_t row0 = (int64_t)b * L;
  const T* Q = static_cast<const T*>(a.q) + row0 * a.ldq + h * DH;
  const T* K = static_cast<const T*>(a.k) + row0 * a.ldk + h * DH;
  const T* V = static_cast<const T*>(a.v) + row0 * a.ldv + h * DH;

  const int qi = xb * 128 + wave * 32 + (lane & 31);
  Frag<T> qf[DH / 16];
#pragma unroll
  for (int kk = 0; kk < DH / 16; ++kk) {
    if (qi < L) ld_frag(qf[kk], Q + (int64_t)qi * a.ldq + kk * 16 + g * 8);
    else {
      float z[8] = {0, 0, 0, 0, 0, 0, 0, 0};
      frag_from(qf[kk], z);
    }
  }
  f32x16 o[DH / 32];
#pragma unroll
  for (int c = 0; c < DH / 32; ++c)
#pragma unroll
    for (int v = 0; v < 16; ++v) o[c][v] = 0.f;
  float m = -INFINITY, lsum = 0.f;

  TL tk, tv;
  tk.init(K, a.ldk, L, tid);
  tv.init(V, a.ldv, L, tid);
  const int nt = (L + KT - 1) / KT;
  // this split's key tiles [t0, t1)
  const int per = (nt + a.ns - 1) / a.ns;
  const int t0 = sp * per, t1 = min(nt, t0 + per);
  tk.load(t0 * KT);
  tv.load(t0 * KT);
  tk.store(ks[0]);
  tv.store(vs[0]);
  __syncthreads();

  auto tile = [&](int jt, auto mask) {
    const int cur = (jt - t0) & 1;
    if (jt + 1 < t1) {
      tk.load((jt + 1) * KT);
      tv.load((jt + 1) * KT);
    }
    const T* Ks = ks[cur];
    const T* Vs = vs[cur];
    f32x16 s[2];
#pragma unroll
    for (int mt = 0; mt < 2; ++mt) {
#pragma unroll
      for (int v = 0; v < 16; ++v) s[mt][v] = 0.f;
#pragma unroll
      for (int kk = 0; kk < DH / 16; ++kk) {
        Frag<T> kf;
        ld_frag(kf, Ks + (mt * 32 + (lane & 31)) * KP + kk * 16 + g * 8);
        mma16(s[mt], kf, qf[kk]);
      }
    }
    if constexpr (decltype(mask)::value) {
      const int jbase = jt * KT;
#pragma unroll
      for (int mt = 0; mt < 2; ++mt)
#pragma unroll
        for (int v = 0; v < 16; ++v)
          if (jbase + mt * 32 + (v >> 2) * 8 + g * 4 + (v & 3) >= L) s[mt][v] = -INFINITY;
    }
    float mloc = -INFINITY;
#pragma unroll
    for (int mt = 0; mt < 2; ++mt)
#pragma unroll
      for (int v = 0; v < 16; ++v) mloc = fmaxf(mloc, s[mt][v]);
    mloc = fmaxf(mloc, __shfl_xor(mloc, 32, 64)) * a.sl2;
    if (__ballot(mloc > m + kMaxSlack) != 0) {
      const float mnew = fmaxf(m, mloc);
      const float alpha = __builtin_amdgcn_exp2f(m - mnew);
      lsum *= alpha;
#pragma unroll
      for (int c = 0; c < DH / 32; ++c)
#pragma unroll
        for (int v = 0; v < 16; ++v) o[c][v] *= alpha;
      m = mnew;
    }
#pragma unroll
    for (int mt = 0; mt < 2; ++mt)
#pragma unroll
      for (int v = 0; v < 16; ++v) s[mt][v] = __builtin_amdgcn_exp2f(fmaf(s[mt][v], a.sl2, -m));
    // O^T[c][q] += V^T[c][kv] P^T[kv][q]; the row sums come from the same
    // bf16 probabilities that enter the product
#pragma unroll
    for (int kk = 0; kk < KT / 16; ++kk) {
      Frag<T> pf;
      acc_frag(pf, s[kk >> 1], (kk & 1) * 8);
      lsum = frag_sum(pf, lsum);
#pragma unroll
      for (int c = 0; c < DH / 32; ++c) {
        Frag<T> vf;
        ld_frag_tr(vf, Vs + kk * 16 * KP + c * 32, KP, lane);
        mma16(o[c], vf, pf);
      }
    }
    if (jt + 1 < t1) {
      tk.store(ks[cur ^ 1]);
      tv.store(vs[cur ^ 1]);
    }
    __syncthreads();
  };
  // full tiles, then the partial last tile of the sequence if it is in range
  const int tf = min(t1, L / KT);
  for (int jt = t0; jt < tf; ++jt) tile(jt, std::false_type{});
  if (tf < t1) tile(tf, std::true_type{});

  const float ltot = lsum + __shfl_xor(lsum, 32, 64);
  if (a.ns > 1) {
    // unnormalised outputs, their reference maximum and row sum
    if (qi < L) {
      const int64_t R = (int64_t)a.B * a.H * L, r = ((int64_t)b * a.H + h) * L + qi;
      float* po = a.part + ((int64_t)sp * R + r) * DH;
#pragma unroll
      for (int c = 0; c < DH / 32; ++c)
#pragma unroll
        for (int r4 = 0; r4 < 4; ++r4)
          st4(po + c * 32 + r4 * 8 + g * 4, o[c][r4 * 4], o[c][r4 * 4 + 1], o[c][r4 * 4 + 2], o[c][r4 * 4 + 3]);
      if (g == 0) {
        float* pm = a.part + (int64_t)a.ns * R * DH;
        pm[(int64_t)sp * R + r] = m;
        pm[(int64_t)(a.ns + sp) * R + r] = ltot;
      }
    }
    return;
  }
  if (qi < L) {
    const float inv = 1.f / ltot;
    T* O = static_cast<T*>(a.o) + (row0 + qi) * a.ldo + h * DH;
#pragma unroll
    for (int c = 0; c < DH / 32; ++c)
#pragma unroll
      for (int r4 = 0; r4 < 4; ++r4) {
        const int col = c * 32 + r4 * 8 + g * 4;
        st4(O + col, o[c][r4 * 4] * inv, o[c][r4 * 4 + 1] * inv, o[c][r4 * 4 + 2] * inv, o[c][r4 * 4 + 3] * inv);
      }
    if (a.o32) {
      float* O32 = a.o32 + (row0 + qi) * a.ldo32 + h * DH;
#pragma unroll
      for (int c = 0; c < DH / 32; ++c)
#pragma unroll
        for (int r4 = 0; r4 < 4; ++r4) {
          const int col = c * 32 + r4 * 8 + g * 4;
          st4(O32 + col, o[c][r4 * 4] * inv, o[c][r4 * 4 + 1] * inv, o[c][r4 * 4 + 2] * inv,
              o[c][r4 * 4 + 3] * inv);
        }
    }
    if (g == 0) a.lse[((int64_t)b * a.H + h) * L + qi] = (m + __log2f(ltot)) * kLn2;
  }
}

// K/V-major backward (bf16): each wave owns 32 keys and sweeps 32-query tiles.
// dK_j = sum_i dS_ij q_i runs on the uncentred queries; the part of the bf16
// rounding of dS that the common query component qbar would amplify is put
// back exactly: dK_j += qbar (sum_i dS_ij - sum_i bf16(dS_ij)), both sums in
// float32, which equals the centred form sum_i bf16(dS_ij) (q_i - qbar) +
// qbar sum_i dS_ij.
// The Q and dO tiles come in by LDS copies (no staging registers), which
// leaves the registers to read each product's fragments one step ahead of
// the product that uses them.
// QG = 2 (grids of at most one block per CU): two groups of 4 waves share the
// block's 128 keys and take alternate query tiles; group 1's dK, dV partials
// are added to group 0's through LDS at the end (fixed order).
template <int DH, int QS = 1, int QG = 1>
__global__ void __launch_bounds__(256 * QG, QG == 2 ? 1 : DH == 128 ? 2 : DH == 64 ? (QS == 1 ? 3 : 2) : 1)
attn_bwd_dkdv_tr(BwdArgs a) {
  using T = bf16;
  constexpr int QT = 32 * QS;  // queries per LDS tile: QS sub-tiles of 32 per barrier
  using DT = DmaRows<QT, DH, 4>;  // Q and dO rows [q][c] of a query tile
  constexpr int RP = DT::PITCH;
  constexpr int TE = DT::BYTES / 2;  // elements of one matrix area
  // the block's V rows stay in LDS rather than in registers, which brings the
  // kernel within the register budget of three waves per SIMD at head_dim 64
  // and two at head_dim 128
  constexpr bool VLDS = DH >= 64;
  __shared__ __attribute__((aligned(16))) T tiles[QG][2][2][TE];  // [group][buffer][Q, dO]
  __shared__ __attribute__((aligned(16))) T vsh[VLDS ? 128 * RP : 8];
  __shared__ float lse_all[QG][2][QT], d_all[QG][2][QT];
  __shared__ float qbar[DH];

  const int lane = threadIdx.x & 63, g = lane >> 5;
  const int grp = QG == 1 ? 0 : __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 8);
  const int tid = threadIdx.x & 255;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  auto& lse_s = lse_all[grp];
  auto& d_s = d_all[grp];
  int xb, h, b;
  attn_block_coords(xb, h, b);
  const int L = a.L;
  const int sp = xb / ((L + 127) / 128);  // query split of this block
  xb -= sp * ((L + 127) / 128);
  const int64_t row0 = (int64_t)b * L;
  if (grp == 0 && tid < DH) qbar[tid] = a.qsum[((int64_t)b * a.H + h) * DH + tid] / (float)L;
  const T* Q = static_cast<const T*>(a.q) + row0 * a.ldq + h * DH;
  const T* K = static_cast<const T*>(a.k) + row0 * a.ldk + h * DH;
  const T* V = static_cast<const T*>(a.v) + row0 * a.ldv + h * DH;
  const T* dO = static_cast<const T*>(a.dO) + row0 * a.lddo + h * DH;
  const float* lse = a.lse + ((int64_t)b * a.H + h) * L;
  const float* Dv = a.D + ((int64_t)b * a.H + h) * L;

  const int kv = xb * 128 + wave * 32 + (lane & 31);
  Frag<T> kf[DH / 16], vf[VLDS ? 1 : DH / 16];
#pragma unroll
  for (int kk = 0; kk < DH / 16; ++kk) {
    if (kv < L) {
      ld_frag(kf[kk], K + (int64_t)kv * a.ldk + kk * 16 + g * 8);
      if constexpr (!VLDS) ld_frag(vf[kk], V + (int64_t)kv * a.ldv + kk * 16 + g * 8);
    } else {
      float z[8] = {0, 0, 0, 0, 0, 0, 0, 0};
      frag_from(kf[kk], z);
      if constexpr (!VLDS) frag_from(vf[kk], z);
    }
  }
  if (VLDS && grp == 0) {
    RowTile<128, DH> tvb;
    tvb.init(V, a.ldv, L, tid);
    tvb.load(xb * 128);
    tvb.store(vsh);
  }
  const T* vrow = vsh + (wave * 32 + (lane & 31)) * RP + g * 8;
  f32x16 dvt[DH / 32], dkt[DH / 32];
#pragma unroll
  for (int c = 0; c < DH / 32; ++c)
#pragma unroll
    for (int v = 0; v < 16; ++v) dvt[c][v] = dkt[c][v] = 0.f;

  float cs = 0.f, csr = 0.f;
  DT dma;
  dma.init(Q, a.ldq, dO, a.lddo, L, wave, lane);
  const unsigned tlds = (unsigned)(uintptr_t)(ORBIT_LDS void*)&tiles[grp][0][0][0];
  constexpr unsigned BUF = 2 * DT::BYTES;
  // this split's query tiles qt0 .. qt0 + nq - 1
  const int nqa = (L + QT - 1) / QT, qper = (nqa + a.ns - 1) / a.ns, qt0 = sp * qper;
  const int nq = max(0, min(nqa, qt0 + qper) - qt0);
  // group grp takes query tiles grp, grp + QG, ... of the range; every group
  // runs the same number of iterations (shared barriers), past its last tile
  // without work
  const int iters = (nq + QG - 1) / QG;
  {
    const int q0 = (qt0 + grp) * QT;
    dma.issue(tlds, q0, wave);
    if (tid < QT) {
      lse_s[0][tid] = q0 + tid < L ? lse[q0 + tid] * kLog2e : INFINITY;
      d_s[0][tid] = q0 + tid < L ? Dv[q0 + tid] : 0.f;
    }
  }
  wait_vmcnt<0>();
  __syncthreads();
  constexpr int KS = DH / 16, NC3 = DH / 32;
  for (int i = 0; i < iters; ++i) {
    const int it = i * QG + grp;
    const int cur = i & 1;
    float lse_n = 0.f, d_n = 0.f;
    if (it + QG < nq) {
      const int q1 = (qt0 + it + QG) * QT;
      dma.issue(tlds + (cur ^ 1) * BUF, q1, wave);
      if (tid < QT) {
        lse_n = q1 + tid < L ? lse[q1 + tid] * kLog2e : INFINITY;
        d_n = q1 + tid < L ? Dv[q1 + tid] : 0.f;
      }
    }
    if (QG == 1 || it < nq) {
      const T* Qs = &tiles[grp][cur][0][0];
      const T* Os = &tiles[grp][cur][1][0];
      // S = Q K^T and dP = dO V^T; step kk + 1's fragments are read before
      // step kk's products are issued
      f32x16 s[QS], dp[QS];
#pragma unroll
      for (int q = 0; q < QS; ++q)
#pragma unroll
        for (int v = 0; v < 16; ++v) s[q][v] = dp[q][v] = 0.f;
      // (fragments rotate through named variables: arrays indexed by the
      // buffer parity would be placed in memory before unrolling)
      Frag<T> cq[QS], co[QS], cv, nq[QS], no[QS], nv;
      auto ld1 = [&](int kk) {
#pragma unroll
        for (int q = 0; q < QS; ++q) {
          ld_frag(nq[q], Qs + (q * 32 + (lane & 31)) * RP + kk * 16 + g * 8);
          ld_frag(no[q], Os + (q * 32 + (lane & 31)) * RP + kk * 16 + g * 8);
        }
        if constexpr (VLDS) ld_frag(nv, vrow + kk * 16);
      };
      auto rot1 = [&]() {
#pragma unroll
        for (int q = 0; q < QS; ++q) {
          cq[q] = nq[q];
          co[q] = no[q];
        }
        cv = nv;
      };
      ld1(0);
      rot1();
#pragma unroll
      for (int kk = 0; kk < KS; ++kk) {
        if (kk + 1 < KS) ld1(kk + 1);
#pragma unroll
        for (int q = 0; q < QS; ++q) {
          mma16(s[q], cq[q], kf[kk]);
          if constexpr (VLDS) mma16(dp[q], co[q], cv);
          else mma16(dp[q], co[q], vf[kk]);
        }
        rot1();
      }
      // P and dS; rows: query 8*(v/4) + 4g + v%4 of the sub-tile, column:
      // this lane's key
#pragma unroll
      for (int q = 0; q < QS; ++q)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int qr = q * 32 + (v >> 2) * 8 + g * 4 + (v & 3);
          const float p = __builtin_amdgcn_exp2f(fmaf(s[q][v], a.sl2, -lse_s[cur][qr]));
          s[q][v] = p;
          dp[q][v] = p * (dp[q][v] - d_s[cur][qr]);
          cs += dp[q][v];
        }
      // dV^T += dO^T P and dK^T += Q^T dS, step n + 1's transposed fragments
      // read before step n's products
      constexpr int N3 = QS * 2 * NC3;
      Frag<T> to, tq, tno, tnq, pf, sf;
      auto ld3 = [&](int n) {
        const int q = n / (2 * NC3), kk = (n / NC3) & 1, c = n % NC3;
        const int off = (q * 32 + kk * 16) * RP + c * 32;
        ld_frag_tr(tno, Os + off, RP, lane);
        ld_frag_tr(tnq, Qs + off, RP, lane);
      };
      ld3(0);
      to = tno;
      tq = tnq;
#pragma unroll
      for (int n = 0; n < N3; ++n) {
        const int q = n / (2 * NC3), kk = (n / NC3) & 1, c = n % NC3;
        if (c == 0) {
          acc_frag(pf, s[q], kk * 8);
          acc_frag(sf, dp[q], kk * 8);
          csr = frag_sum(sf, csr);
        }
        if (n + 1 < N3) ld3(n + 1);
        mma16(dvt[c], to, pf);
        mma16(dkt[c], tq, sf);
        to = tno;
        tq = tnq;
      }
    }
    if (it + QG < nq && tid < QT) {
      lse_s[cur ^ 1][tid] = lse_n;
      d_s[cur ^ 1][tid] = d_n;
    }
    wait_vmcnt<0>();
    __syncthreads();
  }

  cs += __shfl_xor(cs, 32, 64);
  csr += __shfl_xor(csr, 32, 64);
  if constexpr (QG == 2) {
    // group 1 hands its partials to group 0 through the idle tile areas (two
    // regions of the tile buffers and the V rows: each holds 32 floats per
    // thread), dV^T first, then dK^T and the remainder sums; group 0 adds
    // them in that fixed order
    static_assert(VLDS, "the exchange uses the V-row area");
    constexpr int C = DH / 32, CPR = (C + 1) / 2, RB = CPR * 16 * 256 * 4;
    static_assert(2 * RB <= (int)sizeof(tiles) && 2 * 256 * 4 <= (int)sizeof(vsh), "exchange areas");
    float* region[3] = {reinterpret_cast<float*>(&tiles[0][0][0][0]),
                        reinterpret_cast<float*>(&tiles[0][0][0][0]) + RB / 4, reinterpret_cast<float*>(vsh)};
    auto slot = [&](int c, int v) -> float& {
      return region[c / CPR][(wave * CPR * 16 + (c % CPR) * 16 + v) * 64 + lane];
    };
    if (grp == 1) {
#pragma unroll
      for (int c = 0; c < C; ++c)
#pragma unroll
        for (int v = 0; v < 16; ++v) slot(c, v) = dvt[c][v];
    }
    __syncthreads();
    if (grp == 0) {
#pragma unroll
      for (int c = 0; c < C; ++c)
#pragma unroll
        for (int v = 0; v < 16; ++v) dvt[c][v] += slot(c, v);
    }
    __syncthreads();
    float* rs = region[2] + wave * 2 * 64 + lane;
    if (grp == 1) {
#pragma unroll
      for (int c = 0; c < C; ++c)
#pragma unroll
        for (int v = 0; v < 16; ++v) slot(c, v) = dkt[c][v];
      rs[0] = cs;
      rs[64] = csr;
    }
    __syncthreads();
    if (grp == 1) return;
#pragma unroll
    for (int c = 0; c < C; ++c)
#pragma unroll
      for (int v = 0; v < 16; ++v) dkt[c][v] += slot(c, v);
    cs += rs[0];
    csr += rs[64];
  }
  if (a.ns > 1) {
    // raw sums of this query range: dK^T, dV^T and the two remainder sums
    if (kv < L) {
      const int64_t R = (int64_t)a.B * a.H * L, r = ((int64_t)b * a.H + h) * L + kv;
      float* pk = a.part + ((int64_t)sp * R + r) * DH;
      float* pv = a.part + ((int64_t)(a.ns + sp) * R + r) * DH;
#pragma unroll
      for (int c = 0; c < DH / 32; ++c)
#pragma unroll
        for (int r4 = 0; r4 < 4; ++r4) {
          const int col = c * 32 + r4 * 8 + g * 4;
          st4(pk + col, dkt[c][r4 * 4], dkt[c][r4 * 4 + 1], dkt[c][r4 * 4 + 2], dkt[c][r4 * 4 + 3]);
          st4(pv + col, dvt[c][r4 * 4], dvt[c][r4 * 4 + 1], dvt[c][r4 * 4 + 2], dvt[c][r4 * 4 + 3]);
        }
      if (g == 0) {
        float* pc = a.part + (int64_t)2 * a.ns * R * DH;
        pc[(int64_t)sp * R + r] = cs;
        pc[(int64_t)(a.ns + sp) * R + r] = csr;
      }
    }
    return;
  }
  const float corr = cs - csr;
  if (kv < L) {
    T* dK = static_cast<T*>(a.dk) + (row0 + kv) * a.ldg + h * DH;
    T* dV = static_cast<T*>(a.dv) + (row0 + kv) * a.ldg + h * DH;
#pragma unroll
    for (int c = 0; c < DH / 32; ++c)
#pragma unroll
      for (int r4 = 0; r4 < 4; ++r4) {
        const int col = c * 32 + r4 * 8 + g * 4;
        st4(dK + col, (dkt[c][r4 * 4] + qbar[col] * corr) * a.scale,
            (dkt[c][r4 * 4 + 1] + qbar[col + 1] * corr) * a.scale,
            (dkt[c][r4 * 4 + 2] + qbar[col + 2] * corr) * a.scale,
            (dkt[c][r4 * 4 + 3] + qbar[col + 3] * corr) * a.scale);
        st4(dV + col, dvt[c][r4 * 4], dvt[c][r4 * 4 + 1], dvt[c][r4 * 4 + 2], dvt[c][r4 * 4 + 3]);
      }
  }
}

// Q-major backward (bf16): each wave owns 32 queries and sweeps 64-key tiles.
// dQ_i = sum_j dS_ij k_j = sum_j dS_ij (k_j - kbar) since sum_j dS_ij = 0; the
// product runs on the uncentred keys and kbar sum_j bf16(dS_ij) (float32) is
// subtracted, which equals the centred form sum_j bf16(dS_ij) (k_j - kbar).
// The K and V tiles come in by LDS copies (no staging registers), and each
// product's fragments are read one step ahead of the product.
// QG = 2 (grids of at most one block per CU): two groups of 4 waves share the
// block's 128 queries and take alternate key tiles; group 1's dQ partials are
// added to group 0's through LDS at the end (fixed order).
template <int DH, int QG = 1>
__global__ void __launch_bounds__(256 * QG, QG == 2 ? 1 : 1) attn_bwd_dq_tr(BwdArgs a) {
  using T = bf16;
  constexpr int KT = 64;
  using DT = DmaRows<KT, DH, 4>;  // K and V rows [kv][c] of a key tile
  constexpr int KP = DT::PITCH;
  constexpr int TE = DT::BYTES / 2;
  __shared__ __attribute__((aligned(16))) T tiles[QG][2][2][TE];  // [group][buffer][K, V]
  __shared__ float kbar[DH];

  const int lane = threadIdx.x & 63, g = lane >> 5;
  const int grp = QG == 1 ? 0 : __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 8);
  const int tid = threadIdx.x & 255;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  int xb, h, b;
  attn_block_coords(xb, h, b);
  const int L = a.L;
  const int sp = xb / ((L + 127) / 128);  // key split of this block
  xb -= sp * ((L + 127) / 128);
  const int64_t row0 = (int64_t)b * L;
  if (grp == 0 && tid < DH) kbar[tid] = a.ksum[((int64_t)b * a.H + h) * DH + tid] / (float)L;
  const T* Q = static_cast<const T*>(a.q) + row0 * a.ldq + h * DH;
  const T* K = static_cast<const T*>(a.k) + row0 * a.ldk + h * DH;
  const T* V = static_cast<const T*>(a.v) + row0 * a.ldv + h * DH;
  const T* dO = static_cast<const T*>(a.dO) + row0 * a.lddo + h * DH;

  const int qi = xb * 128 + wave * 32 + (lane & 31);
  Frag<T> qf[DH / 16], of[DH / 16];
#pragma unroll
  for (int kk = 0; kk < DH / 16; ++kk) {
    if (qi < L) {
      ld_frag(qf[kk], Q + (int64_t)qi * a.ldq + kk * 16 + g * 8);
      ld_frag(of[kk], dO + (int64_t)qi * a.lddo + kk * 16 + g * 8);
    } else {
      float z[8] = {0, 0, 0, 0, 0, 0, 0, 0};
      frag_from(qf[kk], z);
      frag_from(of[kk], z);
    }
  }
  const float lse2 = qi < L ? a.lse[((int64_t)b * a.H + h) * L + qi] * kLog2e : INFINITY;
  const float Dq = qi < L ? a.D[((int64_t)b * a.H + h) * L + qi] : 0.f;

  f32x16 dqt[DH / 32];
#pragma unroll
  for (int c = 0; c < DH / 32; ++c)
#pragma unroll
    for (int v = 0; v < 16; ++v) dqt[c][v] = 0.f;
  float rs = 0.f;

  DT dma;
  dma.init(K, a.ldk, V, a.ldv, L, wave, lane);
  const unsigned tlds = (unsigned)(uintptr_t)(ORBIT_LDS void*)&tiles[grp][0][0][0];
  constexpr unsigned BUF = 2 * DT::BYTES;
  // this split's key tiles [t0, t1)
  const int nt = (L + KT - 1) / KT, per = (nt + a.ns - 1) / a.ns;
  const int t0 = sp * per, t1 = min(nt, t0 + per);
  // group grp takes key tiles t0 + grp, t0 + grp + QG, ...; both groups run
  // the same number of iterations (shared barriers)
  dma.issue(tlds, (t0 + grp) * KT, wave);
  wait_vmcnt<0>();
  __syncthreads();

  constexpr int KS = DH / 16, NC3 = DH / 32;
  auto tile = [&](int jt, int cur, auto mask) {
    if (jt + QG < t1) dma.issue(tlds + (cur ^ 1) * BUF, (jt + QG) * KT, wave);
    const T* Ks = &tiles[grp][cur][0][0];
    const T* Vs = &tiles[grp][cur][1][0];
    f32x16 s[2], dp[2];
    // the softmax of a 32-key half; at head_dim 64 both halves' products are
    // issued before either half's softmax (the register budget allows it)
    auto soft = [&](int mt) {
      if constexpr (decltype(mask)::value) {
        const int jbase = jt * KT;
#pragma unroll
        for (int v = 0; v < 16; ++v)
          if (jbase + mt * 32 + (v >> 2) * 8 + g * 4 + (v & 3) >= L) s[mt][v] = -INFINITY;
      }
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const float p = __builtin_amdgcn_exp2f(fmaf(s[mt][v], a.sl2, -lse2));
        dp[mt][v] = p * (dp[mt][v] - Dq);
      }
    };
    constexpr bool kBoth = DH == 64;
    // S^T = K Q^T and dP^T = V dO^T over the two 32-key halves, step n + 1's
    // fragments read before step n's products
    Frag<T> ck, cv, nk, nv;
    auto ld1 = [&](int n) {
      const int mt = n / KS, kk = n % KS;
      ld_frag(nk, Ks + (mt * 32 + (lane & 31)) * KP + kk * 16 + g * 8);
      ld_frag(nv, Vs + (mt * 32 + (lane & 31)) * KP + kk * 16 + g * 8);
    };
    ld1(0);
    ck = nk;
    cv = nv;
#pragma unroll
    for (int n = 0; n < 2 * KS; ++n) {
      const int mt = n / KS, kk = n % KS;
      if (kk == 0)
#pragma unroll
        for (int v = 0; v < 16; ++v) s[mt][v] = dp[mt][v] = 0.f;
      if (n + 1 < 2 * KS) ld1(n + 1);
      mma16(s[mt], ck, qf[kk]);
      mma16(dp[mt], cv, of[kk]);
      ck = nk;
      cv = nv;
      if (!kBoth && kk == KS - 1) soft(mt);
    }
    if constexpr (kBoth) {
      soft(0);
      soft(1);
    }
    // dQ^T[c][q] += K^T[c][kv] dS^T[kv][q], step n + 1's transposed K
    // fragment read before step n's product
    constexpr int N3 = (KT / 16) * NC3;
    Frag<T> ct, nt3, sf;
    auto ld3 = [&](int n) {
      const int kk = n / NC3, c = n % NC3;
      ld_frag_tr(nt3, Ks + kk * 16 * KP + c * 32, KP, lane);
    };
    ld3(0);
    ct = nt3;
#pragma unroll
    for (int n = 0; n < N3; ++n) {
      const int kk = n / NC3, c = n % NC3;
      if (c == 0) {
        acc_frag(sf, dp[kk >> 1], (kk & 1) * 8);
        rs = frag_sum(sf, rs);
      }
      if (n + 1 < N3) ld3(n + 1);
      mma16(dqt[c], ct, sf);
      ct = nt3;
    }
    wait_vmcnt<0>();
    __syncthreads();
  };
  // full tiles of the range (the sequence's partial last tile, if any, comes last)
  const int nfs = max(0, min(t1, L / KT) - t0), nts = t1 - t0;
  if constexpr (QG == 1) {
    for (int i = 0; i < nfs; ++i) tile(t0 + i, i & 1, std::false_type{});
    if (nfs < nts) tile(t0 + nfs, nfs & 1, std::true_type{});
  } else {
    // pairs of full tiles, then at most two more tiles (one may be partial;
    // a group past its last tile only joins the barrier)
    const int pairs = nfs / QG;
    for (int i = 0; i < pairs; ++i) tile(t0 + i * QG + grp, i & 1, std::false_type{});
    for (int i = pairs; i < (nts + QG - 1) / QG; ++i) {
      const int jt = t0 + i * QG + grp;
      if (jt < t1) tile(jt, i & 1, std::true_type{});
      else __syncthreads();
    }
  }

  rs += __shfl_xor(rs, 32, 64);
  if constexpr (QG == 2) {
    // group 1's dQ^T partials and remainder sums to group 0 through the idle
    // tile buffers
    constexpr int C = DH / 32;
    static_assert(C * 16 * 256 * 4 + 256 * 4 <= (int)sizeof(tiles), "exchange areas");
    float* rq = reinterpret_cast<float*>(&tiles[0][0][0][0]) + wave * C * 16 * 64 + lane;
    float* rr = reinterpret_cast<float*>(&tiles[0][0][0][0]) + C * 16 * 256 + wave * 64 + lane;
    if (grp == 1) {
#pragma unroll
      for (int c = 0; c < C; ++c)
#pragma unroll
        for (int v = 0; v < 16; ++v) rq[(c * 16 + v) * 64] = dqt[c][v];
      rr[0] = rs;
    }
    __syncthreads();
    if (grp == 1) return;
#pragma unroll
    for (int c = 0; c < C; ++c)
#pragma unroll
      for (int v = 0; v < 16; ++v) dqt[c][v] += rq[(c * 16 + v) * 64];
    rs += rr[0];
  }
  if (a.ns > 1) {
    // raw sums of this key range: dQ^T and the remainder sum
    if (qi < L) {
      const int64_t R = (int64_t)a.B * a.H * L, r = ((int64_t)b * a.H + h) * L + qi;
      float* pq = a.part + ((int64_t)sp * R + r) * DH;
#pragma unroll
      for (int c = 0; c < DH / 32; ++c)
#pragma unroll
        for (int r4 = 0; r4 < 4; ++r4)
          st4(pq + c * 32 + r4 * 8 + g * 4, dqt[c][r4 * 4], dqt[c][r4 * 4 + 1], dqt[c][r4 * 4 + 2],
              dqt[c][r4 * 4 + 3]);
      if (g == 0) a.part[(int64_t)a.ns * R * DH + (int64_t)sp * R + r] = rs;
    }
    return;
  }
  if (qi < L) {
    T* dQ = static_cast<T*>(a.dq) + (row0 + qi) * a.ldg + h * DH;
#pragma unroll
    for (int c = 0; c < DH / 32; ++c)
#pragma unroll
      for (int r4 = 0; r4 < 4; ++r4) {
        const int col = c * 32 + r4 * 8 + g * 4;
        st4(dQ + col, (dqt[c][r4 * 4] - kbar[col] * rs) * a.scale,
            (dqt[c][r4 * 4 + 1] - kbar[col + 1] * rs) * a.scale,
            (dqt[c][r4 * 4 + 2] - kbar[col + 2] * rs) * a.scale,
            (dqt[c][r4 * 4 + 3] - kbar[col + 3] * rs) * a.scale);
      }
  }
}

// ---------------------------------------------------------------------------
// merges of the split partials (fixed order over the splits); one thread per
// (row, 8 columns), rows in (sample, head, position) order
// ---------------------------------------------------------------------------

// O, o32 and lse: each split's unnormalised output is rescaled to the largest
// of the splits' reference maxima, and the sum is divided by the combined row
// sum
template <int DH>
__global__ void __launch_bounds__(256) attn_fwd_merge(FwdArgs a) {
  constexpr int C8 = DH / 8;
  const int64_t R = (int64_t)a.B * a.H * a.L;
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= R * C8) return;
  const int64_t r = idx / C8;
  const int c0 = (int)(idx % C8) * 8;
  const float* pm = a.part + (int64_t)a.ns * R * DH;
  float M = -INFINITY;
  for (int s = 0; s < a.ns; ++s) M = fmaxf(M, pm[(int64_t)s * R + r]);
  float den = 0.f, acc[8];
#pragma unroll
  for (int u = 0; u < 8; ++u) acc[u] = 0.f;
  for (int s = 0; s < a.ns; ++s) {
    const float w = __builtin_amdgcn_exp2f(pm[(int64_t)s * R + r] - M);
    den += w * pm[(int64_t)(a.ns + s) * R + r];
    const float* po = a.part + ((int64_t)s * R + r) * DH + c0;
    const f32x4 x0 = *reinterpret_cast<const f32x4*>(po), x1 = *reinterpret_cast<const f32x4*>(po + 4);
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      acc[u] += w * x0[u];
      acc[4 + u] += w * x1[u];
    }
  }
  const float inv = 1.f / den;
  const int64_t bh = r / a.L;
  const int qi = (int)(r - bh * a.L), h = (int)(bh % a.H);
  const int64_t orow = (bh / a.H) * a.L + qi;
  bf16* O = static_cast<bf16*>(a.o) + orow * a.ldo + h * DH + c0;
  st4(O, acc[0] * inv, acc[1] * inv, acc[2] * inv, acc[3] * inv);
  st4(O + 4, acc[4] * inv, acc[5] * inv, acc[6] * inv, acc[7] * inv);
  if (a.o32) {
    float* O32 = a.o32 + orow * a.ldo32 + h * DH + c0;
    st4(O32, acc[0] * inv, acc[1] * inv, acc[2] * inv, acc[3] * inv);
    st4(O32 + 4, acc[4] * inv, acc[5] * inv, acc[6] * inv, acc[7] * inv);
  }
  if (c0 == 0) a.lse[r] = (M + __log2f(den)) * kLn2;
}

// dK = (sum of the splits' dK^T + qbar (sum cs - sum csr)) / sqrt(dh), dV = sum of dV^T
template <int DH>
__global__ void __launch_bounds__(256) attn_dkdv_merge(BwdArgs a) {
  constexpr int C8 = DH / 8;
  const int64_t R = (int64_t)a.B * a.H * a.L;
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= R * C8) return;
  const int64_t r = idx / C8;
  const int c0 = (int)(idx % C8) * 8;
  const float* pc = a.part + (int64_t)2 * a.ns * R * DH;
  float cs = 0.f, csr = 0.f, k8[8], v8[8];
#pragma unroll
  for (int u = 0; u < 8; ++u) k8[u] = v8[u] = 0.f;
  for (int s = 0; s < a.ns; ++s) {
    cs += pc[(int64_t)s * R + r];
    csr += pc[(int64_t)(a.ns + s) * R + r];
    const float* pk = a.part + ((int64_t)s * R + r) * DH + c0;
    const float* pv = a.part + ((int64_t)(a.ns + s) * R + r) * DH + c0;
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      k8[u] += pk[u];
      v8[u] += pv[u];
    }
  }
  const float corr = cs - csr;
  const int64_t bh = r / a.L;
  const int kv = (int)(r - bh * a.L), h = (int)(bh % a.H);
  const int64_t orow = (bh / a.H) * a.L + kv;
  float dk[8];
#pragma unroll
  for (int u = 0; u < 8; ++u) dk[u] = (k8[u] + a.qsum[bh * DH + c0 + u] / (float)a.L * corr) * a.scale;
  bf16* dK = static_cast<bf16*>(a.dk) + orow * a.ldg + h * DH + c0;
  bf16* dV = static_cast<bf16*>(a.dv) + orow * a.ldg + h * DH + c0;
  st4(dK, dk[0], dk[1], dk[2], dk[3]);
  st4(dK + 4, dk[4], dk[5], dk[6], dk[7]);
  st4(dV, v8[0], v8[1], v8[2], v8[3]);
  st4(dV + 4, v8[4], v8[5], v8[6], v8[7]);
}

// dQ = (sum of the splits' dQ^T - kbar sum rs) / sqrt(dh)
template <int DH>
__global__ void __launch_bounds__(256) attn_dq_merge(BwdArgs a) {
  constexpr int C8 = DH / 8;
  const int64_t R = (int64_t)a.B * a.H * a.L;
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= R * C8) return;
  const int64_t r = idx / C8;
  const int c0 = (int)(idx % C8) * 8;
  float rs = 0.f, q8[8];
#pragma unroll
  for (int u = 0; u < 8; ++u) q8[u] = 0.f;
  for (int s = 0; s < a.ns; ++s) {
    rs += a.part[(int64_t)a.ns * R * DH + (int64_t)s * R + r];
    const float* pq = a.part + ((int64_t)s * R + r) * DH + c0;
#pragma unroll
    for (int u = 0; u < 8; ++u) q8[u] += pq[u];
  }
  const int64_t bh = r / a.L;
  const int qi = (int)(r - bh * a.L), h = (int)(bh % a.H);
  const int64_t orow = (bh / a.H) * a.L + qi;
  float dq[8];
#pragma unroll
  for (int u = 0; u < 8; ++u) dq[u] = (q8[u] - a.ksum[bh * DH + c0 + u] / (float)a.L * rs) * a.scale;
  bf16* dQ = static_cast<bf16*>(a.dq) + orow * a.ldg + h * DH + c0;
  st4(dQ, dq[0], dq[1], dq[2], dq[3]);
  st4(dQ + 4, dq[4], dq[5], dq[6], dq[7]);
}

// the bf16 kernels address one (sample, head) slice of q, k, v (and dO) with
// 32-bit byte offsets (tiles reach up to 256 rows past the last one, and an
// out-of-range marker of 2^31 is added to such offsets), and the backward
// preprocess indexes head rows in 32 bits
bool slices_fit(const AttnIO& io, int64_t ld_extra) {
  const int64_t ld = std::max(std::max(io.ldq, io.ldk), std::max(io.ldv, ld_extra));
  return ((int64_t)io.L + 256) * ld * 4 < ((int64_t)1 << 31) && (int64_t)io.B * io.L * io.H < ((int64_t)1 << 31);
}

// bf16 grids of fewer than 256 blocks of 128 positions (one sample-head pair
// per block row) leave CUs idle: the sweep (keys for the forward and dQ,
// queries for dK, dV) is then split over 2 blocks whose float32 partials a
// merge kernel combines
int attn_splits(int B, int H, int L) {
  return cdiv(L, 128) * (int64_t)H * B < 256 && L >= 512 ? 2 : 1;
}
// the partials of a split launch: ns x rows x (2 dh + 2) floats covers the
// backward's dK/dV partials (and, reused afterwards, its dQ partials) and the
// forward's output partials
size_t split_bytes(int B, int H, int L, int dh) {
  const int ns = attn_splits(B, H, L);
  return ns > 1 ? align_up((size_t)ns * B * H * L * (2 * dh + 2) * sizeof(float)) : 0;
}
size_t attn_bwd_base_bytes(int B, int H, int L, int dh) {
  return align_up((size_t)B * H * (L + 2 * dh) * sizeof(float)) + 2 * colsum_part_bytes(L, H * dh, false, B);
}

template <typename T, int DH>
orbit_status fwd_t(const AttnIO& io, void* o, int64_t ldo, float* lse, float* o32, int64_t ldo32, void* scratch,
                   size_t scratch_bytes, hipStream_t s) {
  if (!slices_fit(io, 0)) {
    set_error("attention: sequence length %d x row stride too large for 32-bit slice offsets", io.L);
    return ORBIT_E_UNSUPPORTED;
  }
  FwdArgs a{io.q, io.k, io.v, o, lse, o32, io.ldq, io.ldk, io.ldv, ldo, ldo32, io.H, io.L, kLog2e / sqrtf((float)DH)};
  const double bh = (double)io.B * io.H;
  KernelInfo ki{sizeof(T) == 2 ? "attn_fwd_kernel<bf16>" : "attn_fwd_kernel<f32>",
                4.0 * bh * io.L * (double)io.L * DH, 4.0 * bh * io.L * DH * sizeof(T)};
  if constexpr (sizeof(T) == 2) {
    const int ns = attn_splits(io.B, io.H, io.L);
    if (ns > 1 && scratch && scratch_bytes >= split_bytes(io.B, io.H, io.L, DH)) {
      a.B = io.B;
      a.ns = ns;
      a.part = static_cast<float*>(scratch);
      ORBIT_TRY(launch(ki, attn_fwd_tr<DH>, dim3((unsigned)(cdiv(io.L, 128) * ns), io.H, io.B), dim3(256), 0, s, a));
      const int64_t rows = (int64_t)io.B * io.H * io.L;
      KernelInfo km{"attn_fwd_merge<bf16>", 0.0,
                    (double)rows * (ns * (DH + 2) * 4.0 + DH * (sizeof(T) + (o32 ? 4.0 : 0.0)))};
      return launch(km, attn_fwd_merge<DH>, dim3((unsigned)cdiv(rows * (DH / 8), 256)), dim3(256), 0, s, a);
    }
    return launch(ki, attn_fwd_tr<DH>, dim3((unsigned)cdiv(io.L, 128), io.H, io.B), dim3(256), 0, s, a);
  }
  return launch(ki, attn_fwd_kernel<T, DH>, dim3((unsigned)cdiv(io.L, 128), io.H, io.B), dim3(256), 0, s, a);
}

template <typename T, int DH>
orbit_status bwd_t(const AttnIO& io, const void* o, int64_t ldo, int o_f32, const float* lse, const void* dO,
                   int64_t lddo, void* dq, void* dk, void* dv, int64_t ldg, float* D, hipStream_t s) {
  if (!slices_fit(io, lddo)) {
    set_error("attention: sequence length %d x row stride too large for 32-bit slice offsets", io.L);
    return ORBIT_E_UNSUPPORTED;
  }
  const double bh = (double)io.B * io.H;
  const int64_t rows = (int64_t)io.B * io.L * io.H;
  KernelInfo kp{sizeof(T) == 2 ? "attn_bwd_pre<bf16>" : "attn_bwd_pre<f32>", 2.0 * rows * DH,
                rows * DH * (sizeof(T) + (o_f32 ? 4.0 : sizeof(T)))};
  const dim3 gp((unsigned)cdiv(rows, 256 / pow2_ceil(DH / 8)));
  if (o_f32)
    ORBIT_TRY(launch(kp, attn_bwd_pre<T, float, DH>, gp, dim3(256), 0, s, (const float*)o, ldo, (const T*)dO, lddo,
                     D, io.B, io.H, io.L));
  else
    ORBIT_TRY(launch(kp, attn_bwd_pre<T, T, DH>, gp, dim3(256), 0, s, (const T*)o, ldo, (const T*)dO, lddo, D,
                     io.B, io.H, io.L));
  // per (sample, head) feature sums of q and k over the sequence
  float* qsum = D + (int64_t)io.B * io.H * io.L;
  float* ksum = qsum + (int64_t)io.B * io.H * DH;
  float* cws = ksum + (int64_t)io.B * io.H * DH;
  const int A = io.H * DH;
  {
    ColJob j[2];
    j[0].src = io.q; j[0].ld = io.ldq; j[0].sbatch = (int64_t)io.L * io.ldq; j[0].n = A; j[0].batch = io.B;
    j[0].part = cws; j[0].out_sum = qsum; j[0].sout = A;
    j[1].src = io.k; j[1].ld = io.ldk; j[1].sbatch = (int64_t)io.L * io.ldk; j[1].n = A; j[1].batch = io.B;
    j[1].part = cws + colsum_part_bytes(io.L, A, false, io.B) / sizeof(float); j[1].out_sum = ksum; j[1].sout = A;
    ORBIT_TRY(colsum_partials(sizeof(T) == 2 ? ORBIT_BF16 : ORBIT_F32, j, 2, io.L, s));
    ColFinal f;
    f.add_job(j[0], io.L);
    f.add_job(j[1], io.L);
    ORBIT_TRY(f.run(0, s));
  }
  BwdArgs a{io.q, io.k, io.v, dO, lse, D, qsum, ksum, dq, dk, dv, io.ldq, io.ldk, io.ldv, lddo, ldg, io.H, io.L,
            kLog2e / sqrtf((float)DH), 1.f / sqrtf((float)DH)};
  const int ns = sizeof(T) == 2 ? attn_splits(io.B, io.H, io.L) : 1;
  if (ns > 1) {
    a.B = io.B;
    a.ns = ns;
    a.part = reinterpret_cast<float*>(reinterpret_cast<char*>(D) + attn_bwd_base_bytes(io.B, io.H, io.L, DH));
  }
  // algorithmic backward = 2x forward; kernels split it 3:2 (dK,dV: 4 products, dQ: 3 incl. recompute)
  const double fl = 4.0 * bh * io.L * (double)io.L * DH;
  KernelInfo k1{sizeof(T) == 2 ? "attn_bwd_dkdv<bf16>" : "attn_bwd_dkdv<f32>", 2 * fl * 0.6,
                6.0 * bh * io.L * DH * sizeof(T)};
  const dim3 grid((unsigned)(cdiv(io.L, 128) * ns), io.H, io.B);
  if constexpr (sizeof(T) == 2) {
    // at most one block per CU (few sample x head pairs): two wave groups per
    // block split the queries, so each SIMD still runs two waves
    const bool few = (int64_t)grid.x * grid.y * grid.z <= 256;
    if constexpr (DH == 128) {
      if (few) ORBIT_TRY(launch(k1, attn_bwd_dkdv_tr<DH, 1, 2>, grid, dim3(512), 0, s, a));
      else ORBIT_TRY(launch(k1, attn_bwd_dkdv_tr<DH, 1>, grid, dim3(256), 0, s, a));
    } else {
      (void)few;
      ORBIT_TRY(launch(k1, attn_bwd_dkdv_tr<DH, DH == 64 ? 2 : 1>, grid, dim3(256), 0, s, a));
    }
  } else {
    ORBIT_TRY(launch(k1, attn_bwd_dkdv<T, DH>, grid, dim3(256), 0, s, a));
  }
  KernelInfo k2{sizeof(T) == 2 ? "attn_bwd_dq<bf16>" : "attn_bwd_dq<f32>", 2 * fl * 0.4,
                5.0 * bh * io.L * DH * sizeof(T)};
  if constexpr (sizeof(T) == 2) {
    const dim3 gm((unsigned)cdiv(rows * (DH / 8), 256));
    if (ns > 1) {
      KernelInfo km{"attn_dkdv_merge<bf16>", 0.0, (double)rows * (ns * (2 * DH + 2) * 4.0 + 2 * DH * sizeof(T))};
      ORBIT_TRY(launch(km, attn_dkdv_merge<DH>, gm, dim3(256), 0, s, a));
    }
    bool done = false;
    if constexpr (DH == 128) {
      if ((int64_t)grid.x * grid.y * grid.z <= 256) {
        ORBIT_TRY(launch(k2, attn_bwd_dq_tr<DH, 2>, grid, dim3(512), 0, s, a));
        done = true;
      }
    }
    if (!done) ORBIT_TRY(launch(k2, attn_bwd_dq_tr<DH>, grid, dim3(256), 0, s, a));
    if (ns == 1) return ORBIT_OK;
    KernelInfo km{"attn_dq_merge<bf16>", 0.0, (double)rows * (ns * (DH + 1) * 4.0 + DH * sizeof(T))};
    return launch(km, attn_dq_merge<DH>, gm, dim3(256), 0, s, a);
  }
  return launch(k2, attn_bwd_dq<T, DH>, grid, dim3(256), 0, s, a);
}

}  // namespace

size_t attn_bwd_workspace_bytes(int B, int H, int L, int dh) {
  return attn_bwd_base_bytes(B, H, L, dh) + split_bytes(B, H, L, dh);
}

orbit_status attn_fwd(orbit_dtype dt, const AttnIO& io, void* o, int64_t ldo, float* lse, float* o32,
                      int64_t ldo32, void* scratch, size_t scratch_bytes, hipStream_t s) {
#define AF(TT, D) return fwd_t<TT, D>(io, o, ldo, lse, o32, ldo32, scratch, scratch_bytes, s)
  if (dt == ORBIT_BF16) {
    if (io.dh == 32) AF(bf16, 32);
    if (io.dh == 64) AF(bf16, 64);
    if (io.dh == 128) AF(bf16, 128);
    if (io.dh == 192) AF(bf16, 192);
    if (io.dh == 256) AF(bf16, 256);
  } else {
    if (io.dh == 32) AF(float, 32);
    if (io.dh == 64) AF(float, 64);
    if (io.dh == 128) AF(float, 128);
  }
#undef AF
  set_error("attention: head_dim %d unsupported", io.dh);
  return ORBIT_E_UNSUPPORTED;
}

orbit_status attn_bwd(orbit_dtype dt, const AttnIO& io, const void* o, int64_t ldo, int o_f32, const float* lse,
                      const void* dO, int64_t lddo, void* dq, void* dk, void* dv, int64_t ldg, float* Dbuf,
                      hipStream_t s) {
#define AB(TT, D) return bwd_t<TT, D>(io, o, ldo, o_f32, lse, dO, lddo, dq, dk, dv, ldg, Dbuf, s)
  if (dt == ORBIT_BF16) {
    if (io.dh == 32) AB(bf16, 32);
    if (io.dh == 64) AB(bf16, 64);
    if (io.dh == 128) AB(bf16, 128);
    if (io.dh == 192) AB(bf16, 192);
    if (io.dh == 256) AB(bf16, 256);
  } else {
    if (io.dh == 32) AB(float, 32);
    if (io.dh == 64) AB(float, 64);
    if (io.dh == 128) AB(float, 128);
  }
#undef AB
  set_error("attention: head_dim %d unsupported", io.dh);
  return ORBIT_E_UNSUPPORTED;
}

}  // namespace orbit
