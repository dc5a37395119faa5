// Shared device types, MFMA fragment helpers, error handling and the launch
// wrapper used by every kernel of the library (gfx950 / CDNA4 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>
#include <math.h>

#include "orbit.h"

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

#define ORBIT_DEV __device__ __forceinline__

namespace orbit {

// ---------------------------------------------------------------------------
// scalar conversion
// ---------------------------------------------------------------------------
ORBIT_DEV float to_f(float x) { return x; }
ORBIT_DEV float to_f(bf16 x) { return (float)x; }
template <typename T> ORBIT_DEV T from_f(float x);
template <> ORBIT_DEV float from_f<float>(float x) { return x; }
template <> ORBIT_DEV bf16 from_f<bf16>(float x) { return (bf16)x; }  // RNE (v_cvt_pk_bf16_f32)

// ---------------------------------------------------------------------------
// 16-byte vector access. E16<T> elements fill 16 bytes.
// ---------------------------------------------------------------------------
template <typename T> struct E16c { static constexpr int v = 16 / (int)sizeof(T); };

struct alignas(16) U128 { uint32_t w[4]; };

ORBIT_DEV U128 ld128(const void* p) { return *reinterpret_cast<const U128*>(p); }
// non-temporal load (data read once: streamed past the caches' normal retention)
ORBIT_DEV U128 ld128nt(const void* p) {
  typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
  return __builtin_bit_cast(U128, __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p)));
}
ORBIT_DEV void st128(void* p, const U128& v) { *reinterpret_cast<U128*>(p) = v; }
ORBIT_DEV U128 zero128() { U128 z; z.w[0] = z.w[1] = z.w[2] = z.w[3] = 0u; return z; }

// unpack 16 bytes of T into floats (8 for bf16, 4 for float)
ORBIT_DEV void unpack(const U128& u, float* f, bf16*) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    f[2 * i] = __uint_as_float(u.w[i] << 16);
    f[2 * i + 1] = __uint_as_float(u.w[i] & 0xffff0000u);
  }
}
ORBIT_DEV void unpack(const U128& u, float* f, float*) {
#pragma unroll
  for (int i = 0; i < 4; ++i) f[i] = __uint_as_float(u.w[i]);
}
ORBIT_DEV U128 pack(const float* f, bf16*) {
  U128 u;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    bf16 lo = (bf16)f[2 * i], hi = (bf16)f[2 * i + 1];
    u.w[i] = (uint32_t)__builtin_bit_cast(uint16_t, lo) | ((uint32_t)__builtin_bit_cast(uint16_t, hi) << 16);
  }
  return u;
}
ORBIT_DEV U128 pack(const float* f, float*) {
  U128 u;
#pragma unroll
  for (int i = 0; i < 4; ++i) u.w[i] = __float_as_uint(f[i]);
  return u;
}

// ---------------------------------------------------------------------------
// MFMA 32x32 tiles on 16-deep K steps.
//
// A "fragment" is the 8 consecutive K-elements a lane supplies for one
// 32x32x16 step: lane l provides row (or column) l%32 and K-slots
// 8*(l/32) .. 8*(l/32)+7. Since the MFMA sums over K, the order in which K
// indices are assigned to slots only has to agree between the A and B
// fragments; kernels exploit this to read fragments as contiguous runs.
// bf16: one v_mfma_f32_32x32x16_bf16. float: eight v_mfma_f32_32x32x2_f32,
// slot j of each lane group feeding the j-th instruction.
// Accumulator layout (both): lane l holds C[row][col] with
// col = l%32, row = 8*(i/4) + 4*(l/32) + i%4 for register i = 0..15.
// ---------------------------------------------------------------------------
template <typename T> struct Frag;
template <> struct Frag<bf16> { bf16x8 v; };
template <> struct Frag<float> { f32x4 lo, hi; };

ORBIT_DEV void mma16(f32x16& acc, const Frag<bf16>& a, const Frag<bf16>& b) {
  acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a.v, b.v, acc, 0, 0, 0);
}
ORBIT_DEV void mma16(f32x16& acc, const Frag<float>& a, const Frag<float>& b) {
#pragma unroll
  for (int j = 0; j < 4; ++j) acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a.lo[j], b.lo[j], acc, 0, 0, 0);
#pragma unroll
  for (int j = 0; j < 4; ++j) acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a.hi[j], b.hi[j], acc, 0, 0, 0);
}

// read a fragment of 8 consecutive elements (16B-aligned for bf16, 32B for float)
ORBIT_DEV void ld_frag(Frag<bf16>& f, const bf16* p) { f.v = *reinterpret_cast<const bf16x8*>(p); }
ORBIT_DEV void ld_frag(Frag<float>& f, const float* p) {
  f.lo = *reinterpret_cast<const f32x4*>(p);
  f.hi = *reinterpret_cast<const f32x4*>(p + 4);
}
// fragment from two runs of 4 consecutive elements (p0[0..3], p1[0..3])
ORBIT_DEV void ld_frag2(Frag<bf16>& f, const bf16* p0, const bf16* p1) {
  bf16x4 a = *reinterpret_cast<const bf16x4*>(p0);
  bf16x4 b = *reinterpret_cast<const bf16x4*>(p1);
  f.v = __builtin_shufflevector(a, b, 0, 1, 2, 3, 4, 5, 6, 7);
}
ORBIT_DEV void ld_frag2(Frag<float>& f, const float* p0, const float* p1) {
  f.lo = *reinterpret_cast<const f32x4*>(p0);
  f.hi = *reinterpret_cast<const f32x4*>(p1);
}
// fragment from 8 floats (accumulator values) converted to T
ORBIT_DEV void frag_from(Frag<bf16>& f, const float* x) {
#pragma unroll
  for (int j = 0; j < 8; ++j) f.v[j] = (bf16)x[j];
}
ORBIT_DEV void frag_from(Frag<float>& f, const float* x) {
#pragma unroll
  for (int j = 0; j < 4; ++j) { f.lo[j] = x[j]; f.hi[j] = x[4 + j]; }
}

// erf(x) for x >= 0 from Abramowitz & Stegun, Handbook of Mathematical
// Functions, formula 7.1.26 (absolute error below 1.5e-7), given e = exp(-x^2):
// erf(x) = 1 - (a1 t + a2 t^2 + a3 t^3 + a4 t^4 + a5 t^5) e,  t = 1 / (1 + p x).
// The GELU epilogues run with the matrix cores idle, so one reciprocal and
// one exponential (shared with the derivative's normal density) matter.
ORBIT_DEV float erf_pos_as(float x, float e) {
  const float t = __builtin_amdgcn_rcpf(fmaf(0.3275911f, x, 1.0f));
  float y = fmaf(1.061405429f, t, -1.453152027f);
  y = fmaf(y, t, 1.421413741f);
  y = fmaf(y, t, -0.284496736f);
  y = fmaf(y, t, 0.254829592f);
  return 1.0f - y * t * e;
}
// GELU(u) = u Phi(u), Phi(u) = (1 + erf(u / sqrt 2)) / 2
ORBIT_DEV float gelu_f(float u) {
  const float x = fabsf(u) * 0.70710678118654752f;
  const float e = __expf(-x * x);
  const float er = copysignf(erf_pos_as(x, e), u);
  return 0.5f * u * (1.0f + er);
}
// GELU'(u) = Phi(u) + u phi(u), phi(u) = exp(-u^2 / 2) / sqrt(2 pi)
ORBIT_DEV float gelu_grad_f(float u) {
  const float x = fabsf(u) * 0.70710678118654752f;
  const float e = __expf(-x * x);
  const float er = copysignf(erf_pos_as(x, e), u);
  return 0.5f * (1.0f + er) + u * 0.39894228040143268f * e;
}

ORBIT_DEV float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
ORBIT_DEV float wave_max(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

// ---------------------------------------------------------------------------
// host side: errors, timing, launches
// ---------------------------------------------------------------------------
void set_error(const char* fmt, ...);
void clear_error();

struct KernelInfo {
  const char* name;   // kernel symbol family (static string)
  double flops;       // algorithmic flops of this launch
  double bytes;       // algorithmic HBM bytes of this launch
};
bool timing_on();
void timing_begin(hipStream_t s, const KernelInfo& k);
void timing_end(hipStream_t s);

// smallest power of two >= n (n >= 1)
constexpr int pow2_ceil(int n) { return n <= 1 ? 1 : 2 * pow2_ceil((n + 1) / 2); }

#define ORBIT_TRY(expr)                                   \
  do {                                                    \
    orbit_status st__ = (expr);                           \
    if (st__ != ORBIT_OK) return st__;                    \
  } while (0)

// Launch `kern` and convert a launch failure into ORBIT_E_DEVICE.
template <typename... KArgs, typename... Args>
orbit_status launch(const KernelInfo& info, void (*kern)(KArgs...), dim3 grid, dim3 block,
                    size_t lds, hipStream_t s, Args... args) {
  if (grid.x == 0 || grid.y == 0 || grid.z == 0) return ORBIT_OK;
  bool t = timing_on();
  if (t) timing_begin(s, info);
  hipLaunchKernelGGL(kern, grid, block, lds, s, args...);
  if (t) timing_end(s);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) {
    set_error("launch of %s failed: %s", info.name, hipGetErrorString(e));
    return ORBIT_E_DEVICE;
  }
  return ORBIT_OK;
}

inline int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }
inline size_t align_up(size_t x, size_t a = 256) { return (x + a - 1) / a * a; }

// Sequential carving of a caller-provided buffer into 256-byte aligned pieces.
struct Carver {
  char* base;
  size_t off = 0;
  explicit Carver(void* b) : base(static_cast<char*>(b)) {}
  template <typename T> T* take(size_t count) {
    off = align_up(off);
    T* p = base ? reinterpret_cast<T*>(base + off) : nullptr;
    off += count * sizeof(T);
    return p;
  }
  size_t used() const { return align_up(off); }
};

}  // namespace orbit
