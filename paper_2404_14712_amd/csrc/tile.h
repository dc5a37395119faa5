// HBM -> LDS staging shared by the GEMM and the attention kernels: the
// buffer unit's direct 1 KB wave copies (dma16), and the register-staged
// copy of one operand tile (TileLoader).
//
// The LDS copy is always K-contiguous: S[row][k] with a row pitch of KD + 16
// bytes (the padding spreads the 16-byte fragment reads of 32 consecutive
// rows over distinct banks). Two source layouts:
//   KMAJ = true : element (row, k) at X[row*ld + k]  (rows are contiguous in k)
//   KMAJ = false: element (row, k) at X[k*ld + row]  (rows are contiguous in the
//                 row dimension; transposed on the way: each thread loads a
//                 4(k) x 16-byte tile and writes 4-element k-runs)
#pragma once
#include "common.h"

namespace orbit {

// one wave copies 64 x 16 bytes from rsrc + voff (per lane) to LDS byte address
// lds + 16 * lane. M0 carries the wave-uniform LDS address; the copy is
// written as inline assembly so that the compiler does not order LDS reads
// behind it (completion is awaited explicitly with s_waitcnt vmcnt).
ORBIT_DEV void dma16(__amdgpu_buffer_rsrc_t r, unsigned lds, unsigned voff) {
  asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds" ::"s"(lds), "v"(voff), "s"(r)
               : "memory", "m0");
}
template <int N> ORBIT_DEV void wait_vmcnt() { asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory"); }

template <typename T, int ROWS, int KD, int NT, bool KMAJ>
struct TileLoader {
  static constexpr int E = 16 / (int)sizeof(T);
  static constexpr int PITCH = KD + E;
  static_assert(KD % E == 0 && ROWS % E == 0 && KD % 4 == 0, "tile shape");
  static constexpr int NCH = KMAJ ? ROWS * (KD / E) : (KD / 4) * (ROWS / E);
  static constexpr int PER = (NCH + NT - 1) / NT;
  static constexpr int REGS = KMAJ ? PER : PER * 4;
  U128 r[REGS];

  // X: operand base. Tile rows row0 .. row0+ROWS-1 (valid while < rlim), k
  // range k0 .. k0+KD-1 (valid while < kend). For the transposed layout a
  // second source X2 supplies the k-rows at and after ksplit (concatenated K).
  ORBIT_DEV void load(const T* X, const T* X2, int ksplit, int64_t ld, int row0, int rlim,
                      int k0, int kend, int tid) {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int c = tid + i * NT;
      if (KMAJ) {
        const int row = c / (KD / E), kc = c % (KD / E);
        const int gr = row0 + row, gk = k0 + kc * E;
        r[i] = (c < NCH && gr < rlim && gk < kend) ? ld128(X + (int64_t)gr * ld + gk) : zero128();
      } else {
        const int kg = c / (ROWS / E), rc = c % (ROWS / E);
        const int gr = row0 + rc * E;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int gk = k0 + kg * 4 + j;
          const bool ok = c < NCH && gr < rlim && gk < kend;
          const T* base = (X2 && gk >= ksplit) ? X2 + (int64_t)(gk - ksplit) * ld : X + (int64_t)gk * ld;
          r[i * 4 + j] = ok ? ld128(base + gr) : zero128();
        }
      }
    }
  }

  ORBIT_DEV void store(T* S, int tid) const {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int c = tid + i * NT;
      if (c >= NCH) continue;
      if (KMAJ) {
        const int row = c / (KD / E), kc = c % (KD / E);
        st128(S + row * PITCH + kc * E, r[i]);
      } else {
        const int kg = c / (ROWS / E), rc = c % (ROWS / E);
        store_transposed(S + (rc * E) * PITCH + kg * 4, &r[i * 4]);
      }
    }
  }

  // transposed layout only: as store(), with mean[row] subtracted from every
  // element first (in float32, then rounded back to T)
  ORBIT_DEV void store_sub(T* S, int tid, const float* mean) const {
    static_assert(!KMAJ, "store_sub applies to the transposed layout");
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int c = tid + i * NT;
      if (c >= NCH) continue;
      const int kg = c / (ROWS / E), rc = c % (ROWS / E);
      store_transposed_sub(S + (rc * E) * PITCH + kg * 4, &r[i * 4], mean + rc * E);
    }
  }

  static ORBIT_DEV float elem(const U128& u, int e) {
    if constexpr (sizeof(T) == 2) {
      const uint32_t w = u.w[e >> 1];
      return __uint_as_float((e & 1) ? (w & 0xffff0000u) : (w << 16));
    } else {
      return __uint_as_float(u.w[e]);
    }
  }

  static ORBIT_DEV void store_transposed_sub(T* S, const U128* q, const float* mean) {
#pragma unroll
    for (int e = 0; e < E; ++e) {
      const float m = mean[e];
      const float v0 = elem(q[0], e) - m, v1 = elem(q[1], e) - m;
      const float v2 = elem(q[2], e) - m, v3 = elem(q[3], e) - m;
      if constexpr (sizeof(T) == 2) {
        bf16x4 o = {(bf16)v0, (bf16)v1, (bf16)v2, (bf16)v3};
        *reinterpret_cast<bf16x4*>(S + e * PITCH) = o;
      } else {
        f32x4 o = {v0, v1, v2, v3};
        *reinterpret_cast<f32x4*>(S + e * PITCH) = o;
      }
    }
  }

  // q[0..3]: four k-rows of E row-elements; writes E runs of 4 k-values
  static ORBIT_DEV void store_transposed(T* S, const U128* q) {
    if constexpr (sizeof(T) == 2) {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int w = e >> 1, sh = (e & 1) * 16;
        const uint32_t v0 = (q[0].w[w] >> sh) & 0xffffu;
        const uint32_t v1 = (q[1].w[w] >> sh) & 0xffffu;
        const uint32_t v2 = (q[2].w[w] >> sh) & 0xffffu;
        const uint32_t v3 = (q[3].w[w] >> sh) & 0xffffu;
        uint2 o;
        o.x = v0 | (v1 << 16);
        o.y = v2 | (v3 << 16);
        *reinterpret_cast<uint2*>(S + e * PITCH) = o;
      }
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        U128 o;
        o.w[0] = q[0].w[e];
        o.w[1] = q[1].w[e];
        o.w[2] = q[2].w[e];
        o.w[3] = q[3].w[e];
        st128(S + e * PITCH, o);
      }
    }
  }
};

}  // namespace orbit

namespace orbit {

// Staging of one GEMM operand tile (ROWS x KD) into a K-contiguous LDS copy
// S[row][k] (pitch KD + 16 bytes), read from HBM either K-major
// (X[row*ld + k]) or M/N-major (X[k*ld + row]).
//
// Thread mapping keeps both the HBM reads and the LDS writes conflict-free:
// consecutive lanes take consecutive 16-byte k-chunks of one LDS row, so 8
// lanes (bf16: 8 chunks of 8) write one full 128-byte row. For the M/N-major
// source each thread owns an E x E block (E k-rows of E row-elements), loads
// it as E 16-byte reads (a wave reads 8 rows x 128 contiguous bytes per
// instruction), transposes it in registers and writes E 16-byte k-runs.
// NTL: K-major tiles loaded non-temporally (operands the product reads once)
template <typename T, int ROWS, int KD, int NT, bool KMAJ, bool NTL = false>
struct GemmStage {
  static constexpr int E = 16 / (int)sizeof(T);
  static constexpr int KC = KD / E;                 // 16-byte chunks per row
  static constexpr int PITCH = KD + E;
  static constexpr int NCH = KMAJ ? ROWS * KC : (KD / E) * (ROWS / E);
  static constexpr int PER = (NCH + NT - 1) / NT;
  static constexpr int REGS = KMAJ ? PER : PER * E;
  static_assert(ROWS % E == 0 && KD % E == 0, "tile shape");
  static constexpr int SIZE = ROWS * PITCH;         // elements of LDS per stage
  U128 r[REGS];

  // MFMA fragment of rows row0 .. row0+31 for the 16-deep step kk
  static ORBIT_DEV void frag(Frag<T>& f, const T* S, int row0, int kk, int lane) {
    ld_frag(f, S + (row0 + (lane & 31)) * PITCH + kk * 16 + (lane >> 5) * 8);
  }

  ORBIT_DEV void load(const T* X, const T* X2, int ksplit, int64_t ld, int row0, int rlim, int k0, int kend,
                      int tid) {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int c = tid + i * NT;
      if (KMAJ) {
        const int row = c / KC, kc = c % KC;
        const int gr = row0 + row, gk = k0 + kc * E;
        const T* src = X + (int64_t)gr * ld + gk;
        r[i] = (c < NCH && gr < rlim && gk < kend) ? (NTL ? ld128nt(src) : ld128(src)) : zero128();
      } else {
        const int kc = c % KC, rc = c / KC;
        const int gr = row0 + rc * E;
#pragma unroll
        for (int j = 0; j < E; ++j) {
          const int gk = k0 + kc * E + j;
          const bool ok = c < NCH && gr < rlim && gk < kend;
          const T* base = (X2 && gk >= ksplit) ? X2 + (int64_t)(gk - ksplit) * ld : X + (int64_t)gk * ld;
          r[i * E + j] = ok ? ld128(base + gr) : zero128();
        }
      }
    }
  }

  ORBIT_DEV void store(T* S, int tid) const {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int c = tid + i * NT;
      if (c >= NCH) continue;
      if (KMAJ) {
        const int row = c / KC, kc = c % KC;
        st128(S + row * PITCH + kc * E, r[i]);
      } else {
        const int kc = c % KC, rc = c / KC;
        T* base = S + (rc * E) * PITCH + kc * E;
        if constexpr (sizeof(T) == 2) {
          // in[j] = k-row j holds row-elements e = 0..7 (2 per word);
          // out[e] = row e holds k-values j = 0..7
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const int w = e >> 1;
            U128 o;
#pragma unroll
            for (int q = 0; q < 4; ++q) {
              const uint32_t lo = r[i * 8 + 2 * q].w[w], hi = r[i * 8 + 2 * q + 1].w[w];
              o.w[q] = (e & 1) ? ((lo >> 16) | (hi & 0xffff0000u)) : ((lo & 0xffffu) | (hi << 16));
            }
            st128(base + e * PITCH, o);
          }
        } else {
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            U128 o;
#pragma unroll
            for (int q = 0; q < 4; ++q) o.w[q] = r[i * 4 + q].w[e];
            st128(base + e * PITCH, o);
          }
        }
      }
    }
  }

};

// bf16 M/N-major operand tile kept as it is in HBM: S[k][row], rows
// contiguous. The row pitch is chosen so that consecutive k-rows start 64 or
// 192 bytes apart modulo 256: the four k-rows one 16-lane group reads in a
// transposing LDS read (ds_read_b64_tr_b16) then fall in distinct banks.
// Staging is a plain 16-byte copy (coalesced along the rows in HBM); the MFMA
// fragments (8 consecutive k of one row per lane, as the K-major stage gives)
// come from two transposing reads.
template <int ROWS, int KD, int NT>
struct GemmStageMN {
  using T = bf16;
  static constexpr int E = 8;
  static constexpr int PAD = ((2 * ROWS) % 256 == 0 || (2 * ROWS) % 256 == 128) ? 32 : 0;
  static constexpr int PITCH = ROWS + PAD;
  static constexpr int RC = ROWS / E;               // 16-byte chunks per k-row
  static constexpr int NCH = KD * RC;
  static constexpr int PER = (NCH + NT - 1) / NT;
  static constexpr int SIZE = KD * PITCH;
  static_assert(ROWS % E == 0 && KD % 16 == 0, "tile shape");
  U128 r[PER];

  static ORBIT_DEV void frag(Frag<T>& f, const T* S, int row0, int kk, int lane) {
    typedef short s16x4 __attribute__((ext_vector_type(4)));
    typedef short s16x8 __attribute__((ext_vector_type(8)));
    const int G = lane >> 4, q = lane & 15;
    // group G: k-rows 8*(G/2) + q/4 (+4 for the second read), rows 16*(G%2) + 4*(q%4) .. +3;
    // lane 16G + i receives row 16*(G%2) + i at those four k
    T* p0 = const_cast<T*>(S) + (kk * 16 + 8 * (G >> 1) + (q >> 2)) * PITCH + row0 + 16 * (G & 1) + 4 * (q & 3);
    T* p1 = p0 + 4 * PITCH;
    const s16x4 x = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4*)p0);
    const s16x4 y = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4*)p1);
    const s16x8 xy = __builtin_shufflevector(x, y, 0, 1, 2, 3, 4, 5, 6, 7);
    f.v = __builtin_bit_cast(bf16x8, xy);
  }

  ORBIT_DEV void load(const T* X, const T* X2, int ksplit, int64_t ld, int row0, int rlim, int k0, int kend,
                      int tid) {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int c = tid + i * NT;
      const int kr = c / RC, rc = c % RC;
      const int gk = k0 + kr, gr = row0 + rc * E;
      const bool ok = c < NCH && gr < rlim && gk < kend;
      const T* base = (X2 && gk >= ksplit) ? X2 + (int64_t)(gk - ksplit) * ld : X + (int64_t)gk * ld;
      r[i] = ok ? ld128(base + gr) : zero128();
    }
  }

  ORBIT_DEV void store(T* S, int tid) const {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int c = tid + i * NT;
      if (c >= NCH) continue;
      st128(S + (c / RC) * PITCH + (c % RC) * E, r[i]);
    }
  }
};

}  // namespace orbit
