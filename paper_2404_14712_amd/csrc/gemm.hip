// MFMA GEMMs for gfx950 with fused epilogues (bias, GELU with pre-activation
// store, GELU derivative, residual, accumulate). Three operand layouts cover
// all linear layers: forward (A K-major, B N-major), input gradient (both
// K-major) and weight gradient (both M/N-major: the reduction runs over
// tokens; the DMA kernel also forms the column sums of B there, the layer's
// bias gradient).
//
// Large bf16 products run on gemm_dma_kernel: 256x256 tiles, 8 waves (two per
// SIMD, each owning a 128x64 block of C), operands copied HBM -> LDS by the
// buffer unit (buffer_load ... lds, 16 bytes per lane, no register staging)
// into a four-stage ring of 32-deep K slices, XOR-swizzled so that both the
// copies and the MFMA fragment reads are free of bank conflicts. K-major
// slices are read with ds_read_b128, M/N-major slices (kept as stored) with
// transposing reads (ds_read_b64_tr_b16). With K-major A the eight waves run
// as two groups half a K slice apart, so that one group's MFMAs overlap the
// other group's fragment reads and copies.
//
// Every other product (float32, small or unaligned shapes, concatenated K)
// runs on gemm_kernel: register-prefetched, double-buffered LDS tiles with
// K-contiguous staging.
#include <stdio.h>
#include <string>

#include <algorithm>
#include <type_traits>

#include "gemm.h"
#include "tile.h"

namespace orbit {
namespace {

struct Epi {
  float alpha;
  int accumulate;
  const void* bias; int64_t sBias;
  void* gelu_out; int64_t ldgo;
  const void* gelu_in; int64_t ldgi;
  const void* res; int64_t ldr, sR; int res_row_mod;
};

struct GemmKArgs {
  const void* A; const void* B; const void* B2; void* C;
  int M, N, K, k_split;
  int64_t lda, ldb, ldc;
  int64_t sA, sB, sB2, sC;
  int batch, splits, k_per_split;
  int vec_ok;      // N, ldc, batch strides and epilogue operands allow 16-byte access
  float* partial;  // splits > 1: float32 partials [splits][batch][M][N]
  float* bsum;     // column sums of B: [splits][bs_groups][batch][N] (A M-major, B N-major)
  int bs_groups;   // tile rows that form them, each from a strided subset of the K slices
  Epi epi;
};

template <typename T, typename OutT>
ORBIT_DEV void epi_apply(const Epi& e, int64_t bz, int r, int c, float v, OutT* C, int64_t ldc) {
  v *= e.alpha;
  const int64_t off = (int64_t)r * ldc + c;
  if (e.accumulate) v += to_f(C[off]);
  if (e.bias) v += to_f(static_cast<const T*>(e.bias)[bz * e.sBias + c]);
  if (e.gelu_out) {
    static_cast<T*>(e.gelu_out)[(int64_t)r * e.ldgo + c] = from_f<T>(v);
    v = gelu_f(v);
  }
  if (e.gelu_in) v *= gelu_grad_f(to_f(static_cast<const T*>(e.gelu_in)[(int64_t)r * e.ldgi + c]));
  if (e.res) {
    const int rr = e.res_row_mod ? r % e.res_row_mod : r;
    v += to_f(static_cast<const T*>(e.res)[bz * e.sR + (int64_t)rr * e.ldr + c]);
  }
  C[off] = from_f<OutT>(v);
}

// 8 consecutive columns c0..c0+7 of row r (16-byte aligned rows)
template <typename T> ORBIT_DEV void ld8(const T* p, float* f) {
  unpack(ld128(p), f, (T*)nullptr);
  if constexpr (sizeof(T) == 4) unpack(ld128(p + 4), f + 4, (T*)nullptr);
}
template <typename T> ORBIT_DEV void st8(T* p, const float* f) {
  st128(p, pack(f, (T*)nullptr));
  if constexpr (sizeof(T) == 4) st128(p + 4, pack(f + 4, (T*)nullptr));
}

// b8: the bias of columns c0..c0+7 when the caller loaded it ahead (else NULL)
template <typename T, typename OutT>
ORBIT_DEV void epi_apply8(const Epi& e, int64_t bz, int r, int c0, float* v, OutT* C, int64_t ldc,
                          const float* b8 = nullptr) {
  const int64_t off = (int64_t)r * ldc + c0;
#pragma unroll
  for (int i = 0; i < 8; ++i) v[i] *= e.alpha;
  float t[8];
  if (e.accumulate) {
    ld8(C + off, t);
#pragma unroll
    for (int i = 0; i < 8; ++i) v[i] += t[i];
  }
  if (e.bias) {
    if (b8) {
#pragma unroll
      for (int i = 0; i < 8; ++i) t[i] = b8[i];
    } else {
      ld8(static_cast<const T*>(e.bias) + bz * e.sBias + c0, t);
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) v[i] += t[i];
  }
  if (e.gelu_out) {
    st8(static_cast<T*>(e.gelu_out) + (int64_t)r * e.ldgo + c0, v);
#pragma unroll
    for (int i = 0; i < 8; ++i) v[i] = gelu_f(v[i]);
  }
  if (e.gelu_in) {
    ld8(static_cast<const T*>(e.gelu_in) + (int64_t)r * e.ldgi + c0, t);
#pragma unroll
    for (int i = 0; i < 8; ++i) v[i] *= gelu_grad_f(t[i]);
  }
  if (e.res) {
    const int rr = e.res_row_mod ? r % e.res_row_mod : r;
    ld8(static_cast<const T*>(e.res) + bz * e.sR + (int64_t)rr * e.ldr + c0, t);
#pragma unroll
    for (int i = 0; i < 8; ++i) v[i] += t[i];
  }
  st8(C + off, v);
}

// operand staging: K-major tiles (and every float32 tile) as K-contiguous LDS
// rows; bf16 M/N-major tiles as they are, read through transposing LDS reads
template <typename T, bool KMAJ, int ROWS, int KD, int NT, bool NTL = false>
using StageOf = std::conditional_t<(!KMAJ && sizeof(T) == 2), GemmStageMN<ROWS, KD, NT>,
                                   GemmStage<T, ROWS, KD, NT, KMAJ, NTL>>;

// STREAM: the K-major operand tiles are loaded non-temporally (products whose
// operands are read once, e.g. the aggregation's score product over the
// token tensor)
template <typename T, typename OutT, int BM, int BN, int WM, int WN, bool AK, bool BKM, bool STREAM = false>
__global__ void __launch_bounds__(WM * WN * 64) gemm_kernel(GemmKArgs g) {
  constexpr int NT = WM * WN * 64;
  constexpr int BKE = 128 / (int)sizeof(T);
  constexpr int WTM = BM / WM, WTN = BN / WN, TM = WTM / 32, TN = WTN / 32;
  static_assert(TM >= 1 && TN >= 1, "wave tile must be at least 32x32");
  extern __shared__ __attribute__((aligned(16))) char smem[];
  T* lds = reinterpret_cast<T*>(smem);
  using SA = StageOf<T, AK, BM, BKE, NT, STREAM>;
  using SB = StageOf<T, BKM, BN, BKE, NT, STREAM>;
  constexpr int STAGE = SA::SIZE + SB::SIZE;
  static_assert((WM * WN) * 32 * (BN / WN + 8) * 4 <= 2 * STAGE * (int)sizeof(T), "epilogue fits the stages");

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave % WM, wn = wave / WM;
  const int z = blockIdx.z;
  const int split = z % g.splits;
  const int64_t bz = z / g.splits;

  // tile order: consecutive hardware ids go round-robin over the 8 XCDs, so
  // give each XCD a contiguous range of tiles, walked in groups of 8 tile
  // rows (the group's A panels and the B panels it sweeps stay in that L2)
  const int tiles_n = (g.N + BN - 1) / BN, tiles_m = (g.M + BM - 1) / BM;
  const int nt = tiles_m * tiles_n;
  int id = blockIdx.x;
  const int full = nt - nt % 8;
  if (id < full) id = (id % 8) * (full / 8) + id / 8;
  constexpr int GROUP = 8;
  const int per_group = GROUP * tiles_n;
  const int first_m = (id / per_group) * GROUP;
  const int gsize = min(tiles_m - first_m, GROUP);
  const int tile_m = first_m + (id % per_group) % gsize;
  const int tile_n = (id % per_group) / gsize;

  const T* A = static_cast<const T*>(g.A) + bz * g.sA;
  const T* B = static_cast<const T*>(g.B) + bz * g.sB;
  const T* B2 = g.B2 ? static_cast<const T*>(g.B2) + bz * g.sB2 : nullptr;
  const int m0 = tile_m * BM, n0 = tile_n * BN;
  const int kbeg = split * g.k_per_split;
  const int kend = min(g.K, kbeg + g.k_per_split);
  const int nk = (kend - kbeg + BKE - 1) / BKE;

  SA la;
  SB lb;

  f32x16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

  if (nk > 0) {
    la.load(A, nullptr, 0, g.lda, m0, g.M, kbeg, kend, tid);
    lb.load(B, B2, g.k_split, g.ldb, n0, g.N, kbeg, kend, tid);
    la.store(lds, tid);
    lb.store(lds + SA::SIZE, tid);
  }
  __syncthreads();

  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < nk) {
      const int k0 = kbeg + (kt + 1) * BKE;
      la.load(A, nullptr, 0, g.lda, m0, g.M, k0, kend, tid);
      lb.load(B, B2, g.k_split, g.ldb, n0, g.N, k0, kend, tid);
    }
    const T* As = lds + cur * STAGE;
    const T* Bs = As + SA::SIZE;
#pragma unroll
    for (int kk = 0; kk < BKE / 16; ++kk) {
      Frag<T> af[TM], bfr[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i) SA::frag(af[i], As, wm * WTM + i * 32, kk, lane);
#pragma unroll
      for (int j = 0; j < TN; ++j) SB::frag(bfr[j], Bs, wn * WTN + j * 32, kk, lane);
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) mma16(acc[i][j], af[i], bfr[j]);
    }
    if (kt + 1 < nk) {
      T* nxt = lds + (cur ^ 1) * STAGE;
      la.store(nxt, tid);
      lb.store(nxt + SA::SIZE, tid);
    }
    __syncthreads();
  }

  // Epilogue through LDS (the stages are free after the final barrier): each
  // wave parks 32 rows of its accumulators at a time in a private region, then
  // reads them back as 8 consecutive columns per lane for 16-byte stores.
  constexpr int EP = WTN + 8;                        // row pitch (floats)
  constexpr int LPR = WTN / 8;                       // lanes per row
  constexpr int RPI = 64 / LPR;                      // rows per iteration
  float* ew = reinterpret_cast<float*>(smem) + wave * 32 * EP;
  OutT* C = static_cast<OutT*>(g.C) + bz * g.sC;
  const bool raw = g.splits > 1;
#pragma unroll
  for (int i = 0; i < TM; ++i) {
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v)
        ew[((v >> 2) * 8 + (lane >> 5) * 4 + (v & 3)) * EP + j * 32 + (lane & 31)] = acc[i][j][v];
    __syncthreads();
    // kept rolled, so that the unrolled loops above index the accumulators statically
#pragma unroll 1
    for (int it = 0; it < 32 / RPI; ++it) {
      const int rl = it * RPI + lane / LPR;
      const int cl = (lane % LPR) * 8;
      const int r = m0 + wm * WTM + i * 32 + rl;
      const int c0 = n0 + wn * WTN + cl;
      float v8[8];
      const f32x4 lo = *reinterpret_cast<const f32x4*>(ew + rl * EP + cl);
      const f32x4 hi = *reinterpret_cast<const f32x4*>(ew + rl * EP + cl + 4);
#pragma unroll
      for (int q = 0; q < 4; ++q) { v8[q] = lo[q]; v8[4 + q] = hi[q]; }
      if (r < g.M && c0 < g.N) {
        if (raw) {
          float* P = g.partial + (((int64_t)split * g.batch + bz) * g.M + r) * g.N;
          if (g.vec_ok) {
            st8(P + c0, v8);
          } else {
            for (int q = 0; q < 8 && c0 + q < g.N; ++q) P[c0 + q] = v8[q];
          }
        } else if (g.vec_ok) {
          epi_apply8<T, OutT>(g.epi, bz, r, c0, v8, C, g.ldc);
        } else {
          for (int q = 0; q < 8 && c0 + q < g.N; ++q) epi_apply<T, OutT>(g.epi, bz, r, c0 + q, v8[q], C, g.ldc);
        }
      }
    }
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------
// gemm_dma_kernel: bf16, 32-deep K stages in an NS-deep LDS ring
// ---------------------------------------------------------------------------
constexpr int DBK = 32;
constexpr unsigned kOobOffset = 0x80000000u;    // beyond num_records: the copy reads zeros

#define ORBIT_LDS __attribute__((address_space(3)))

ORBIT_DEV __amdgpu_buffer_rsrc_t buffer_rsrc(const void* base) {
  // raw buffer over [base, base + 2 GiB); offsets at or past kOobOffset read zeros
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, 0x7fffffff, 0x00020000);
}


// Copy plan of one operand slice (ROWS rows x 32 k) over NW waves, per lane.
//  K-major source X[row*ld + k]: LDS row r holds 64 bytes (4 chunks of 8 k);
//    logical chunk c sits at physical chunk c ^ ((r >> 2) & 3). A 1 KB copy
//    covers 16 rows.
//  M/N-major source X[k*ld + row]: LDS k-row kr holds 2 ROWS bytes (ROWS / 8
//    chunks of 8 rows); logical chunk c sits at physical chunk c ^ (4 (kr & 3)).
//    A 1 KB copy covers 512 / ROWS k-rows.
template <bool KMAJ, int ROWS, int NW>
struct DmaPlan {
  static constexpr int BYTES = ROWS * DBK * 2;
  static constexpr int NL = BYTES / 1024 / NW;  // 1 KB copies per wave
  static_assert(NL >= 1 && BYTES % (1024 * NW) == 0, "copy split");
  unsigned voff[NL];
  ORBIT_DEV void init(int64_t ld, int row0, int rlim, int wave, int lane) {
#pragma unroll
    for (int j = 0; j < NL; ++j) {
      const int blk = wave * NL + j;
      if (KMAJ) {
        const int r = blk * 16 + (lane >> 2);
        const int c = (lane & 3) ^ ((lane >> 4) & 3);
        voff[j] = (row0 + r < rlim) ? (unsigned)(r * ld * 2 + c * 16) : kOobOffset;
      } else {
        constexpr int CPR = ROWS / 8, KPB = 64 / CPR;
        const int kr = blk * KPB + lane / CPR;
        const int c = (lane % CPR) ^ (4 * (kr & 3));
        voff[j] = (row0 + c * 8 < rlim) ? (unsigned)(kr * ld * 2 + c * 16) : kOobOffset;
      }
    }
  }
  ORBIT_DEV void issue(const bf16* base, unsigned lds, int wave) const {
    const __amdgpu_buffer_rsrc_t r = buffer_rsrc(base);
#pragma unroll
    for (int j = 0; j < NL; ++j) dma16(r, lds + (wave * NL + j) * 1024, voff[j]);
  }
};

// MFMA fragment reads from one operand slice: rows row0 + 32 i + (lane & 31),
// k-slots 8 (lane >> 5) .. +7 of the 16-deep step kk.
template <bool KMAJ, int NF, int ROWS>
struct DmaFrag {
  unsigned off[NF];
  unsigned x[2];
  ORBIT_DEV void init(int row0, int lane) {
    if (KMAJ) {
      const int f = (lane >> 2) & 3, h = lane >> 5;
#pragma unroll
      for (int kk = 0; kk < 2; ++kk) x[kk] = (unsigned)(((2 * kk + h) ^ f) << 4);
      off[0] = (unsigned)((row0 + (lane & 31)) * 64);
    } else {
      // transposing read: 16-lane group G reads k-rows 8 (G >> 1) + (q >> 2) (and
      // +4) at rows 16 (G & 1) + 4 (q & 3) .. +3; lane 16 G + i receives row
      // 16 (G & 1) + i at those k
      const int G = lane >> 4, q = lane & 15;
      const int xs = 4 * ((q >> 2) & 3);
      const int cb = 2 * (G & 1) + ((q & 3) >> 1);
#pragma unroll
      for (int i = 0; i < NF; ++i) {
        const int c = ((row0 >> 3) + i * 4 + cb) ^ xs;
        off[i] = (unsigned)((8 * (G >> 1) + (q >> 2)) * (2 * ROWS) + c * 16 + (q & 1) * 8);
      }
    }
  }
  ORBIT_DEV void read(bf16x8& f, const char* S, int i, int kk) const {
    if (KMAJ) {
      f = *reinterpret_cast<const bf16x8*>(S + off[0] + i * 2048 + x[kk]);
    } else {
      typedef short s16x4 __attribute__((ext_vector_type(4)));
      const char* p0 = S + off[i] + kk * 16 * (2 * ROWS);
      const s16x4 a = __builtin_amdgcn_ds_read_tr16_b64_v4i16((ORBIT_LDS s16x4*)p0);
      const s16x4 b = __builtin_amdgcn_ds_read_tr16_b64_v4i16((ORBIT_LDS s16x4*)(p0 + 4 * (2 * ROWS)));
      f = __builtin_bit_cast(bf16x8, __builtin_shufflevector(a, b, 0, 1, 2, 3, 4, 5, 6, 7));
    }
  }
};

// Tile configurations of the direct-to-LDS kernel. BIG: 256x256 on 8 waves
// (two per SIMD, 128x64 each), four stages, one block per CU. HALF: 256x128
// on 4 waves (128x64 each), three stages (72 KB), two independent blocks per
// CU, which fills the GPU on products with few 256x256 tiles.
template <int BM_, int BN_, int WM_, int WN_, int NS_, int OCC_, bool PP_ = false>
struct DmaCfg {
  static constexpr int BM = BM_, BN = BN_, WM = WM_, WN = WN_, NS = NS_, OCC = OCC_;
  static constexpr bool PP = PP_;
  static constexpr int NW = WM * WN, NT = NW * 64;
  static constexpr int TM = BM / WM / 32, TN = BN / WN / 32;
  static constexpr int OPA = BM * DBK * 2, OPB = BN * DBK * 2, STB = OPA + OPB;
  static constexpr int EPB = NW * 32 * (TN * 32 + 8) * 4;   // epilogue staging
  static constexpr int LDS = NS * STB > EPB ? NS * STB : EPB;
};
using DmaBig = DmaCfg<256, 256, 2, 4, 4, 1>;
using DmaHalf = DmaCfg<256, 128, 2, 2, 3, 2>;
using DmaPP = DmaCfg<256, 256, 2, 4, 4, 1, true>;   // BIG in two wave groups

// wait until stage s has landed when copies of the next `ahead` stages
// (each NLS copies per wave) may still be in flight
template <int NLS, int NS>
ORBIT_DEV void wait_stage(int ahead) {
  static_assert(NS == 3 || NS == 4, "ring depth");
  if (NS == 4 && ahead >= 2) wait_vmcnt<2 * NLS>();
  else if (ahead >= 1) wait_vmcnt<NLS>();
  else wait_vmcnt<0>();
}

template <bool AK, bool BKM, typename OutT, typename CF>
__global__ void __launch_bounds__(CF::NT, CF::OCC) gemm_dma_kernel(GemmKArgs g) {
  constexpr int BM = CF::BM, BN = CF::BN, WM = CF::WM, NS = CF::NS;
  constexpr int TM = CF::TM, TN = CF::TN, OPA = CF::OPA, STB = CF::STB;
  using PA = DmaPlan<AK, BM, CF::NW>;
  using PB = DmaPlan<BKM, BN, CF::NW>;
  constexpr int NLS = PA::NL + PB::NL;  // copies per stage per wave
  extern __shared__ __attribute__((aligned(1024))) char smem[];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave % WM, wn = wave / WM;
  int split = blockIdx.z % g.splits;
  const int64_t bz = blockIdx.z / g.splits;

  // tile order: XCD-contiguous ranges of tile ids, walked in groups of 8 tile rows
  const int tiles_n = (g.N + BN - 1) / BN, tiles_m = (g.M + BM - 1) / BM;
  const int nt = tiles_m * tiles_n;
  int id = blockIdx.x;
  const int full = nt - nt % 8;
  if (g.splits > 1 && g.batch == 1 && 8 % g.splits == 0 && (nt * g.splits) % 8 == 0) {
    // split K: each XCD takes one K range over a contiguous 8 / splits share of
    // the tiles, so its L2 holds one K range of the A and B panels its tiles
    // share (every XCD running every range fetched each panel slice from HBM
    // once per XCD)
    const int lin = blockIdx.x + nt * (int)blockIdx.z, xcd = lin % 8;
    split = xcd % g.splits;
    id = (xcd / g.splits) * (nt * g.splits / 8) + lin / 8;
  } else if (id < full) {
    id = (id % 8) * (full / 8) + id / 8;
  }
  // groups of tile rows sized so that an XCD's share of C is about as tall
  // as wide in elements (A and B panel bytes per tile in proportion)
  constexpr int GR = BN == 128 ? 4 : 8;
  const int per_group = GR * tiles_n;
  const int first_m = (id / per_group) * GR;
  const int gsize = min(tiles_m - first_m, GR);
  const int tile_m = first_m + (id % per_group) % gsize;
  const int tile_n = (id % per_group) / gsize;
  const int m0 = tile_m * BM, n0 = tile_n * BN;
  const int kbeg = split * g.k_per_split;
  const int kend = min(g.K, kbeg + g.k_per_split);
  const int nk = max(kend - kbeg, 0) / DBK;

  const bf16* A = static_cast<const bf16*>(g.A) + bz * g.sA;
  const bf16* B = static_cast<const bf16*>(g.B) + bz * g.sB;
  const bf16* Ab = AK ? A + (int64_t)m0 * g.lda + kbeg : A + (int64_t)kbeg * g.lda + m0;
  const bf16* Bb = BKM ? B + (int64_t)n0 * g.ldb + kbeg : B + (int64_t)kbeg * g.ldb + n0;
  const int64_t a_step = AK ? DBK : (int64_t)DBK * g.lda;
  const int64_t b_step = BKM ? DBK : (int64_t)DBK * g.ldb;

  PA pa;
  PB pb;
  pa.init(g.lda, m0, g.M, wave, lane);
  pb.init(g.ldb, n0, g.N, wave, lane);
  DmaFrag<AK, TM, BM> ra;
  DmaFrag<BKM, TN, BN> rb;
  ra.init(wm * TM * 32, lane);
  rb.init(wn * TN * 32, lane);

  f32x16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

  const unsigned lds0 = (unsigned)(uintptr_t)(ORBIT_LDS void*)smem;
  auto issue = [&](int st) {
    const unsigned b = lds0 + (st % NS) * STB;
    pa.issue(Ab + st * a_step, b, wave);
    pb.issue(Bb + st * b_step, b + OPA, wave);
  };
  // prologue: stages 0 .. NS-2 in flight (each wave's copies complete in issue
  // order), then wait for stage 0
#pragma unroll
  for (int st = 0; st < NS - 1; ++st)
    if (st < nk) issue(st);
  wait_stage<NLS, NS>(min(nk - 1, NS - 2));
  __syncthreads();

  bf16x8 fa[2][TM], fb[2][TN];
  if constexpr (CF::PP) {
    // Two wave groups (waves 0-3 and 4-7, one of each per SIMD) run half a
    // slice apart: while one group issues its MFMAs the other reads its next
    // fragments and copies, so the matrix pipe of every SIMD is fed by one wave
    // at a time. Group 1 starts one barrier late; every phase ends with a
    // barrier of all eight waves.
    const int grp = wave >> 2;
    if (grp) __builtin_amdgcn_s_barrier();
    for (int kt = 0; kt < nk; ++kt) {
      const char* cur = smem + (kt % NS) * STB;
      // memory phase: this slice's fragments; the slot of slice kt + NS - 1
      // held slice kt - 1, whose reads every wave completed before the barrier
      // that ended its previous memory phase
#pragma unroll
      for (int kk = 0; kk < 2; ++kk) {
#pragma unroll
        for (int i = 0; i < TM; ++i) ra.read(fa[kk][i], cur, i, kk);
#pragma unroll
        for (int j = 0; j < TN; ++j) rb.read(fb[kk][j], cur + OPA, j, kk);
      }
      if (kt + NS - 1 < nk) issue(kt + NS - 1);
      wait_stage<NLS, NS>(min(nk - kt - 2, NS - 2));
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
      __builtin_amdgcn_sched_barrier(0);
      __builtin_amdgcn_s_barrier();
      __builtin_amdgcn_sched_barrier(0);
      // compute phase, at raised wave priority: the other group's fragment
      // reads and copy issues then do not delay this group's MFMA issue
      __builtin_amdgcn_s_setprio(1);
#pragma unroll
      for (int kk = 0; kk < 2; ++kk)
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int j = 0; j < TN; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[kk][i], fb[kk][j], acc[i][j], 0, 0, 0);
      __builtin_amdgcn_s_setprio(0);
      __builtin_amdgcn_sched_barrier(0);
      __builtin_amdgcn_s_barrier();
      __builtin_amdgcn_sched_barrier(0);
    }
    if (!grp) __builtin_amdgcn_s_barrier();
  } else {
  // weight gradients: the column sums of B (a bias gradient) are formed by the
  // first bs_groups tile rows, tile row i from the K slices kt = i (mod
  // bs_groups), so that no block carries much of the extra work; the waves of
  // a block's first wave row hold every column of B in their fragments, each
  // lane 8 k of one column per fragment
  constexpr bool kCanBs = !AK && !BKM;
  const bool bs_on = kCanBs && g.bsum != nullptr && tile_m < g.bs_groups && wm == 0;
  int bs_next = tile_m;
  bool bs_now = false;
  float bs[TN];
#pragma unroll
  for (int j = 0; j < TN; ++j) bs[j] = 0.f;
  auto bsum_add = [&](const bf16x8* f) {
    if constexpr (kCanBs) {
      if (bs_now) {
        const bf16x2 one = {(bf16)1.f, (bf16)1.f};
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const bf16x2 pr = {f[j][2 * q], f[j][2 * q + 1]};
            bs[j] = __builtin_amdgcn_fdot2_f32_bf16(pr, one, bs[j], false);
          }
      }
    }
  };
#pragma unroll
  for (int i = 0; i < TM; ++i) ra.read(fa[0][i], smem, i, 0);
#pragma unroll
  for (int j = 0; j < TN; ++j) rb.read(fb[0][j], smem + OPA, j, 0);

  for (int kt = 0; kt < nk; ++kt) {
    const char* cur = smem + (kt % NS) * STB;
    const char* nxt = smem + ((kt + 1) % NS) * STB;
    // the slot of stage kt + NS - 1 held stage kt - 1, which every wave finished
    // reading before the barrier that ended the previous iteration
    if (kt + NS - 1 < nk) issue(kt + NS - 1);
    if constexpr (kCanBs) {
      bs_now = bs_on && kt == bs_next;
      if (bs_now) bs_next += g.bs_groups;
    }
#pragma unroll
    for (int i = 0; i < TM; ++i) ra.read(fa[1][i], cur, i, 1);
#pragma unroll
    for (int j = 0; j < TN; ++j) rb.read(fb[1][j], cur + OPA, j, 1);
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[0][i], fb[0][j], acc[i][j], 0, 0, 0);
    bsum_add(fb[0]);
    // stage kt + 1 landed (copies of the stages after it may still be in flight)
    wait_stage<NLS, NS>(min(nk - kt - 2, NS - 2));
    __syncthreads();
    // next stage's first fragments (unconditionally: past the last stage this
    // reads a stale but in-bounds slot, and keeping the loop branch-free lets
    // the reads overlap the MFMAs below)
#pragma unroll
    for (int i = 0; i < TM; ++i) ra.read(fa[0][i], nxt, i, 0);
#pragma unroll
    for (int j = 0; j < TN; ++j) rb.read(fb[0][j], nxt + OPA, j, 0);
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[1][i], fb[1][j], acc[i][j], 0, 0, 0);
    bsum_add(fb[1]);
  }
  if (bs_on) {
    // lanes l and l + 32 hold the two k halves of column l & 31
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const float t = bs[j] + __shfl_xor(bs[j], 32, 64);
      const int c = n0 + wn * TN * 32 + j * 32 + lane;
      const int64_t part = (int64_t)split * g.bs_groups + tile_m;
      if (lane < 32 && c < g.N) g.bsum[(part * g.batch + bz) * g.N + c] = t;
    }
  }
  }
  wait_vmcnt<0>();
  __syncthreads();

  // epilogue through LDS: each wave parks 32 rows of its accumulators in a
  // private region and reads them back as 8 consecutive columns per lane
  constexpr int WTN = TN * 32, EP = WTN + 8, LPR = WTN / 8, RPI = 64 / LPR;
  float* ew = reinterpret_cast<float*>(smem) + wave * 32 * EP;
  OutT* C = static_cast<OutT*>(g.C) + bz * g.sC;
  const bool raw = g.splits > 1;
  // a lane's 8 output columns are the same for all its rows: its bias is
  // loaded once, not once per row pass
  float b8[8];
  {
    const int pcol = n0 + wn * WTN + (lane % LPR) * 8;
#pragma unroll
    for (int q = 0; q < 8; ++q) b8[q] = 0.f;
    if (!raw && g.vec_ok && g.epi.bias && pcol < g.N)
      ld8(static_cast<const bf16*>(g.epi.bias) + bz * g.epi.sBias + pcol, b8);
  }
#pragma unroll
  for (int i = 0; i < TM; ++i) {
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v)
        ew[((v >> 2) * 8 + (lane >> 5) * 4 + (v & 3)) * EP + j * 32 + (lane & 31)] = acc[i][j][v];
    __builtin_amdgcn_wave_barrier();
#pragma unroll 1
    for (int it = 0; it < 32 / RPI; ++it) {
      const int rl = it * RPI + lane / LPR;
      const int cl = (lane % LPR) * 8;
      const int r = m0 + wm * TM * 32 + i * 32 + rl;
      const int c0 = n0 + wn * WTN + cl;
      float v8[8];
      const f32x4 lo = *reinterpret_cast<const f32x4*>(ew + rl * EP + cl);
      const f32x4 hi = *reinterpret_cast<const f32x4*>(ew + rl * EP + cl + 4);
#pragma unroll
      for (int q = 0; q < 4; ++q) { v8[q] = lo[q]; v8[4 + q] = hi[q]; }
      if (r < g.M && c0 < g.N) {
        if (raw) {
          float* P = g.partial + (((int64_t)split * g.batch + bz) * g.M + r) * g.N;
          if (g.vec_ok) {
            st8(P + c0, v8);
          } else {
            for (int q = 0; q < 8 && c0 + q < g.N; ++q) P[c0 + q] = v8[q];
          }
        } else if (g.vec_ok) {
          epi_apply8<bf16, OutT>(g.epi, bz, r, c0, v8, C, g.ldc, b8);
        } else {
          for (int q = 0; q < 8 && c0 + q < g.N; ++q) epi_apply<bf16, OutT>(g.epi, bz, r, c0 + q, v8[q], C, g.ldc);
        }
      }
    }
    __builtin_amdgcn_wave_barrier();
  }
}

// C = epilogue(sum over splits of the float32 partials): 8 consecutive columns
// per thread, rows on grid.y (strided), batch on grid.z; 32-bit index math
template <typename T, typename OutT>
__global__ void __launch_bounds__(64) splitk_reduce(GemmKArgs g) {
  const int c0 = (blockIdx.x * 64 + threadIdx.x) * 8;
  if (c0 >= g.N) return;
  const int64_t bz = blockIdx.z;
  const int64_t MN = (int64_t)g.M * g.N;
  OutT* C = static_cast<OutT*>(g.C) + bz * g.sC;
  for (int r = blockIdx.y; r < g.M; r += gridDim.y) {
    const float* p = g.partial + bz * MN + (int64_t)r * g.N + c0;
    const int64_t stride = (int64_t)g.batch * MN;
    if (g.vec_ok) {
      float v[8], t[8];
      ld8(p, v);
      for (int s = 1; s < g.splits; ++s) {
        ld8(p + s * stride, t);
#pragma unroll
        for (int i = 0; i < 8; ++i) v[i] += t[i];
      }
      epi_apply8<T, OutT>(g.epi, bz, r, c0, v, C, g.ldc);
    } else {
      for (int q = 0; q < 8 && c0 + q < g.N; ++q) {
        float v = 0.f;
        for (int s = 0; s < g.splits; ++s) v += p[s * stride + q];
        epi_apply<T, OutT>(g.epi, bz, r, c0 + q, v, C, g.ldc);
      }
    }
  }
}

// ---------------------------------------------------------------------------
// host dispatch
// ---------------------------------------------------------------------------
struct TileCfg {
  int BM, BN, WM, WN;
  bool dma = false;  // gemm_dma_kernel (bf16 only)
  bool operator==(const TileCfg& o) const {
    return BM == o.BM && BN == o.BN && WM == o.WM && WN == o.WN && dma == o.dma;
  }
};
constexpr TileCfg kDma{DmaBig::BM, DmaBig::BN, DmaBig::WM, DmaBig::WN, true};
constexpr TileCfg kDmaHalf{DmaHalf::BM, DmaHalf::BN, DmaHalf::WM, DmaHalf::WN, true};
constexpr TileCfg kT256{256, 256, 2, 4};
constexpr TileCfg kBig{128, 128, 2, 2};
constexpr TileCfg kNarrowN{128, 32, 4, 1};
constexpr TileCfg kNarrowM{32, 128, 1, 4};
constexpr TileCfg kSmall{64, 64, 2, 2};

int64_t tiles_of(const Gemm& g, const TileCfg& t) { return cdiv(g.M, t.BM) * cdiv(g.N, t.BN) * (int64_t)g.batch; }

int bke_of(orbit_dtype dt) { return dt == ORBIT_BF16 ? 64 : 32; }

// gemm_dma_kernel's requirements: whole 32-deep K slices, 16-byte aligned
// operand rows, and per-lane byte offsets within a tile below 2^31
bool dma_ok(const Gemm& g) {
  auto al16 = [](const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; };
  const int64_t lim = (int64_t)1 << 24;
  return g.dtype == ORBIT_BF16 && g.B2 == nullptr && g.K % DBK == 0 && (g.a_kmajor || !g.b_kmajor) &&
         g.lda % 8 == 0 && g.ldb % 8 == 0 && g.sA % 8 == 0 && g.sB % 8 == 0 && g.lda < lim && g.ldb < lim &&
         al16(g.A) && al16(g.B);
}

// bf16 products: the (tile, split) pair with the least modelled time. The
// model was fitted (least squares on log time) to every tile and split on the
// block products of five model sizes, measured on MI355X. A launch runs in
// rounds of `slots` concurrent work items (tile x K range; one 256x256 DMA
// block per CU, two of the smaller tiles); a round of ks 64-deep K steps takes
// c + r * ks microseconds with every CU busy, r depending on the operand
// layout (forward: A K-major, B N-major; input gradient: both K-major; weight
// gradient: A M-major, B N-major). The last round, with a fraction f of the
// slots filled, runs faster by 1 + beta (1 - f), up to `cap`: the chip is
// power-limited, and with fewer CUs busy they clock higher and share the
// memory system among fewer (a 144-tile launch on 256 CUs reaches 85% of the
// full-chip rate). A split adds its float32 partials, written and read back,
// at 0.29 us per MB.
struct Choice { TileCfg t; int splits; };

Choice pick_bf16(const Gemm& g) {
  struct Cand { TileCfg t; int slots; double c, fwd, dx, dw, beta, cap; };
  const Cand cands[] = {{kDma, 256, 11.38, 1.540, 1.610, 1.683, 0.85, 1.562},
                        {kDmaHalf, 512, 8.41, 1.951, 1.906, 1.995, 1.343, 2.093},
                        {kT256, 256, 9.97, 2.083, 1.986, 2.166, 0.239, 1.114},
                        {kBig, 512, 5.47, 1.367, 1.197, 1.394, 0.60, 1.425}};
  constexpr double kSplitUsPerMB = 0.2922;
  const bool dma = dma_ok(g);
  Choice best{kBig, 1};
  double best_us = 1e300;
  for (const Cand& c : cands) {
    if (g.M < c.t.BM || g.N < c.t.BN) continue;
    if (c.t.dma && !dma) continue;
    const double rate = g.a_kmajor ? (g.b_kmajor ? c.dx : c.fwd) : c.dw;
    const int64_t tiles = tiles_of(g, c.t);
    const int64_t ksteps = cdiv(g.K, 64);
    for (int sp = 1; sp <= 16; sp *= 2) {
      if (sp > 1 && (ksteps / sp < 8 || tiles * sp > 2048)) break;
      const int64_t items = tiles * sp;
      const int64_t ks = cdiv(cdiv(g.K, sp), 64);
      const int64_t n = cdiv(items, c.slots);
      const double f = (double)(items - (n - 1) * c.slots) / c.slots;
      const double boost = std::min(c.cap, 1.0 + c.beta * (1.0 - f));
      double us = ((double)(n - 1) + 1.0 / boost) * (c.c + rate * (double)ks);
      if (sp > 1) us += kSplitUsPerMB * sp * (double)g.M * g.N * g.batch * 4.0 / 1e6;
      if (us < best_us) {
        best_us = us;
        best = {c.t, sp};
      }
    }
  }
  return best;
}

TileCfg pick_tile(const Gemm& g) {
  // a long reduction against a few columns (the aggregation's score product,
  // K = d = 16384 on the 113B shard): 64x64 tiles stream A ~4% faster
  if (g.N <= 32) return g.dtype == ORBIT_BF16 && g.a_kmajor && g.b_kmajor && g.K >= 8192 ? kSmall : kNarrowN;
  if (g.M <= 32) return kNarrowM;
  if (g.M <= 64 || g.N <= 64) return kSmall;
  if (g.dtype == ORBIT_BF16 && g.K >= 256 && g.M >= 128 && g.N >= 128) return pick_bf16(g).t;
  // short reductions with a large output (a per-head product over head_dim):
  // the output write dominates, and the two-blocks-per-CU DMA tile overlaps
  // one block's stores with the other's loads (25% faster than 128x128 tiles)
  if (g.dtype == ORBIT_BF16 && g.K >= DBK && g.M >= 256 && g.N >= 128 && dma_ok(g)) return kDmaHalf;
  return kBig;
}

// K ranges actually launched for a requested split count: whole 64-deep steps
// per range, so fewer ranges than requested can cover K
int used_splits(const Gemm& g, int splits) {
  if (splits <= 1 || g.K <= 0) return 1;
  const int bke = bke_of(g.dtype);
  const int per = (int)cdiv(cdiv(g.K, bke), splits) * bke;
  return (int)cdiv(g.K, per);
}

int pick_splits(const Gemm& g, const TileCfg& t) {
  if (g.dtype == ORBIT_BF16 && g.K >= 256 && g.M >= 128 && g.N >= 128 && t == pick_bf16(g).t)
    return pick_bf16(g).splits;
  const int64_t tiles = tiles_of(g, t);
  const int bke = bke_of(g.dtype);
  const int64_t ksteps = cdiv(g.K, bke);
  // fewer than two blocks per CU: split K (with one 4-wave block per CU a
  // long K loop leaves HBM latency exposed; the per-head weight gradient of
  // the aggregation at 256 tiles is 25% faster split in two)
  if (tiles >= 512 || ksteps < 8) return 1;
  int64_t s = cdiv(512, tiles);
  s = std::min<int64_t>(s, ksteps / 4);
  s = std::min<int64_t>(s, 64);
  return (int)std::max<int64_t>(s, 1);
}

template <typename OutT>
orbit_status splitk_finish(const Gemm& g, GemmKArgs& a, hipStream_t s);

template <bool AK, bool BKM, typename OutT, typename CF>
orbit_status run_dma(const Gemm& g, GemmKArgs& a, hipStream_t s) {
  static const std::string name = std::string(CF::PP ? "gemm_dma_pp<" : "gemm_dma<") + std::to_string(CF::BM) + "x" + std::to_string(CF::BN) +
                                  "," + (AK ? "AK" : "AM") + "," + (BKM ? "BK" : "BN") + "," +
                                  (sizeof(OutT) == 2 ? "bf16" : "f32") + ">";
  const double flops = 2.0 * g.M * g.N * (double)g.K * g.batch;
  const double bytes = ((double)g.M * g.K + (double)g.K * g.N) * 2.0 * g.batch +
                       (double)g.M * g.N * sizeof(OutT) * g.batch;
  KernelInfo ki{name.c_str(), flops, bytes};
  static const bool attr = [] {
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(gemm_dma_kernel<AK, BKM, OutT, CF>),
                              hipFuncAttributeMaxDynamicSharedMemorySize, CF::LDS);
    (void)hipGetLastError();
    return true;
  }();
  (void)attr;
  dim3 grid((unsigned)(cdiv(g.N, CF::BN) * cdiv(g.M, CF::BM)), 1, (unsigned)(g.batch * a.splits));
  ORBIT_TRY(launch(ki, gemm_dma_kernel<AK, BKM, OutT, CF>, grid, dim3(CF::NT), (size_t)CF::LDS, s, a));
  return a.splits > 1 ? splitk_finish<OutT>(g, a, s) : ORBIT_OK;
}

template <typename T, typename OutT, int BM, int BN, int WM, int WN, bool AK, bool BKM, bool STREAM>
const char* kname() {
  static std::string s = [] {
    char b[160];
    snprintf(b, sizeof b, "gemm_kernel<%s,%s,%d,%d,%d,%d,%s,%s%s>", sizeof(T) == 2 ? "bf16" : "f32",
             sizeof(OutT) == 2 ? "bf16" : "f32", BM, BN, WM, WN, AK ? "AK" : "AM", BKM ? "BK" : "BN",
             STREAM ? ",stream" : "");
    return std::string(b);
  }();
  return s.c_str();
}

template <typename T, typename OutT, int BM, int BN, int WM, int WN, bool AK, bool BKM, bool STREAM = false>
orbit_status run_cfg(const Gemm& g, GemmKArgs& a, hipStream_t s) {
  const double flops = 2.0 * g.M * g.N * (double)g.K * g.batch;
  const double bytes = ((double)g.M * g.K + (double)g.K * g.N) * sizeof(T) * g.batch +
                       (double)g.M * g.N * sizeof(OutT) * g.batch;
  KernelInfo ki{kname<T, OutT, BM, BN, WM, WN, AK, BKM, STREAM>(), flops, bytes};
  dim3 grid((unsigned)(cdiv(g.N, BN) * cdiv(g.M, BM)), 1, (unsigned)(g.batch * a.splits));
  constexpr int NT = WM * WN * 64, BKE = 128 / (int)sizeof(T);
  constexpr size_t lds = 2 * (size_t)(StageOf<T, AK, BM, BKE, NT>::SIZE + StageOf<T, BKM, BN, BKE, NT>::SIZE) * sizeof(T);
  static const bool attr = [] {
    // lift the default dynamic-LDS cap for this instantiation (a failure here
    // surfaces as a launch error below)
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(gemm_kernel<T, OutT, BM, BN, WM, WN, AK, BKM, STREAM>),
                              hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    (void)hipGetLastError();
    return true;
  }();
  (void)attr;
  ORBIT_TRY(launch(ki, gemm_kernel<T, OutT, BM, BN, WM, WN, AK, BKM, STREAM>, grid, dim3(WM * WN * 64), lds, s, a));
  return a.splits > 1 ? splitk_finish<OutT>(g, a, s) : ORBIT_OK;
}

template <typename OutT>
orbit_status splitk_finish(const Gemm& g, GemmKArgs& a, hipStream_t s) {
  const int64_t total = (int64_t)g.M * g.N * g.batch;
  KernelInfo kr{sizeof(OutT) == 2 ? "splitk_reduce<bf16>" : "splitk_reduce<f32>", 0.0,
                (double)total * 4 * (a.splits + 1)};
  const dim3 grid((unsigned)cdiv(g.N, 512), (unsigned)std::min(g.M, 16384), (unsigned)g.batch);
  if (g.dtype == ORBIT_BF16) return launch(kr, splitk_reduce<bf16, OutT>, grid, dim3(64), 0, s, a);
  return launch(kr, splitk_reduce<float, OutT>, grid, dim3(64), 0, s, a);
}

template <typename T, typename OutT, bool AK, bool BKM>
orbit_status run_layout(const Gemm& g, GemmKArgs& a, const TileCfg& t, hipStream_t s) {
  if constexpr (sizeof(T) == 2) {
    if (t.dma && t.BN == DmaHalf::BN) return run_dma<AK, BKM, OutT, DmaHalf>(g, a, s);
    // K-major A (forward and input-gradient products): the two-group loop,
    // 1-4% faster there; with M-major A (weight gradients) it is 2-3% slower
    if (t.dma) {
      if constexpr (AK) return run_dma<AK, BKM, OutT, DmaPP>(g, a, s);
      else return run_dma<AK, BKM, OutT, DmaBig>(g, a, s);
    }
    if (t.BM == 256 && t.BN == 256 && t.WM == 2) return run_cfg<T, OutT, 256, 256, 2, 4, AK, BKM>(g, a, s);
    if (t.BM == 256 && t.BN == 256 && t.WM == 4) return run_cfg<T, OutT, 256, 256, 4, 2, AK, BKM>(g, a, s);
  }
  if (t.BM == 128 && t.BN == 128) return run_cfg<T, OutT, 128, 128, 2, 2, AK, BKM>(g, a, s);
  if constexpr (sizeof(T) == 2 && AK && BKM) {
    if (g.stream && t.BM == 64 && t.BN == 64) return run_cfg<T, OutT, 64, 64, 2, 2, AK, BKM, true>(g, a, s);
  }
  if (t.BM == 128 && t.BN == 32) return run_cfg<T, OutT, 128, 32, 4, 1, AK, BKM>(g, a, s);
  if (t.BM == 32 && t.BN == 128) return run_cfg<T, OutT, 32, 128, 1, 4, AK, BKM>(g, a, s);
  return run_cfg<T, OutT, 64, 64, 2, 2, AK, BKM>(g, a, s);
}

template <typename T, typename OutT>
orbit_status run_typed(const Gemm& g, GemmKArgs& a, const TileCfg& t, hipStream_t s) {
  if (g.a_kmajor && !g.b_kmajor) return run_layout<T, OutT, true, false>(g, a, t, s);
  if (g.a_kmajor && g.b_kmajor) return run_layout<T, OutT, true, true>(g, a, t, s);
  if (!g.a_kmajor && !g.b_kmajor) return run_layout<T, OutT, false, false>(g, a, t, s);
  set_error("gemm: layout (A M-major, B K-major) is not supported");
  return ORBIT_E_UNSUPPORTED;
}

}  // namespace

// tile rows that form the column sums of B: as many as the partial budget
// allows per K range, at most every tile row
static int bsum_groups(const Gemm& g, const TileCfg& t, int splits) {
  return (int)std::max<int64_t>(1, std::min<int64_t>(cdiv(g.M, t.BM), g.bsum_max_parts / splits));
}

int gemm_bsum_parts(const Gemm& g) {
  if (g.dtype != ORBIT_BF16 || g.a_kmajor || g.b_kmajor || g.M <= 0 || g.N <= 0 || g.K < DBK) return 0;
  const TileCfg t = pick_tile(g);
  if (!t.dma || !dma_ok(g)) return 0;
  const int sp = used_splits(g, pick_splits(g, t));
  if (sp > g.bsum_max_parts) return 0;
  return sp * bsum_groups(g, t, sp);
}

size_t gemm_workspace_bytes(const Gemm& g) {
  const TileCfg t = pick_tile(g);
  const int s = pick_splits(g, t);
  return s > 1 ? align_up((size_t)s * g.batch * (size_t)g.M * g.N * sizeof(float)) : 0;
}

namespace {

// one product on tile configuration t with the K range cut into `splits`
// slices (when the workspace holds their float32 partials; else one slice)
orbit_status gemm_run(const Gemm& g, const TileCfg& t, int splits, void* ws, size_t ws_bytes, hipStream_t s) {
  GemmKArgs a{};
  a.A = g.A; a.B = g.B; a.B2 = g.B2; a.C = g.C;
  a.M = g.M; a.N = g.N; a.K = g.K; a.k_split = g.B2 ? g.k_split : g.K;
  a.lda = g.lda; a.ldb = g.ldb; a.ldc = g.ldc;
  a.sA = g.sA; a.sB = g.sB; a.sB2 = g.sB2; a.sC = g.sC;
  a.batch = g.batch;
  a.splits = 1;
  a.k_per_split = g.K;
  a.partial = nullptr;
  a.bsum = g.bsum;
  a.bs_groups = 1;
  if (splits > 1 && ws && ws_bytes >= (size_t)splits * g.batch * (size_t)g.M * g.N * sizeof(float)) {
    const int bke = bke_of(g.dtype);
    const int64_t ksteps = cdiv(g.K, bke);
    const int per = (int)cdiv(ksteps, splits) * bke;
    a.splits = (int)cdiv(g.K, per);
    a.k_per_split = per;
    a.partial = static_cast<float*>(ws);
  }
  if (g.K <= 0) a.k_per_split = 0;
  if (g.bsum) a.bs_groups = bsum_groups(g, t, a.splits);
  {
    auto al = [](int64_t x) { return x % 8 == 0; };
    auto ap = [](const void* p) { return p == nullptr || (reinterpret_cast<uintptr_t>(p) & 15u) == 0; };
    a.vec_ok = al(g.N) && al(g.ldc) && al(g.sC) && al(g.sBias) && al(g.ldgo) && al(g.ldgi) && al(g.ldr) &&
               al(g.sR) && ap(g.C) && ap(g.bias) && ap(g.gelu_out) && ap(g.gelu_in) && ap(g.res);
  }
  a.epi.alpha = g.alpha;
  a.epi.accumulate = g.accumulate ? 1 : 0;
  a.epi.bias = g.bias;
  a.epi.sBias = g.sBias;
  a.epi.gelu_out = g.gelu_out; a.epi.ldgo = g.ldgo;
  a.epi.gelu_in = g.gelu_in; a.epi.ldgi = g.ldgi;
  a.epi.res = g.res; a.epi.ldr = g.ldr; a.epi.sR = g.sR; a.epi.res_row_mod = g.res_row_mod;
  if (g.dtype == ORBIT_BF16) {
    return g.out_f32 ? run_typed<bf16, float>(g, a, t, s) : run_typed<bf16, bf16>(g, a, t, s);
  }
  // float operands always produce float
  return run_typed<float, float>(g, a, t, s);
}

}  // namespace

orbit_status gemm(const Gemm& g, void* ws, size_t ws_bytes, hipStream_t s) {
  if (g.M <= 0 || g.N <= 0 || g.batch <= 0) return ORBIT_OK;
  // K-major operands are read in 16-byte chunks along K: with K % 8 != 0 the
  // last chunk runs past K, which is only sound when the other operand's rows
  // are masked (M/N-major) and the K-major rows are zero-padded (internal use).
  if (g.K % 8 != 0 && g.a_kmajor && g.b_kmajor) {
    set_error("gemm: K=%d must be a multiple of 8 when both operands are K-major", g.K);
    return ORBIT_E_ARG;
  }
  if (g.accumulate && !g.out_f32) {
    set_error("gemm: accumulate needs a float32 output");
    return ORBIT_E_ARG;
  }
  const TileCfg t = pick_tile(g);
  const int splits = pick_splits(g, t);
  if (g.bsum) {
    // the column sums come from gemm_dma_kernel's M-major-A, N-major-B form,
    // one partial per K split
    if (gemm_bsum_parts(g) == 0) {
      set_error("gemm: column sums of B are formed only by bf16 weight-gradient products on the DMA kernel");
      return ORBIT_E_UNSUPPORTED;
    }
    if (splits > 1 && ws_bytes < gemm_workspace_bytes(g)) {
      set_error("gemm: a product with column sums needs its split-K workspace (%zu bytes)", gemm_workspace_bytes(g));
      return ORBIT_E_ARG;
    }
  }
  return gemm_run(g, t, splits > 1 && ws_bytes >= gemm_workspace_bytes(g) ? splits : 1, ws, ws_bytes, s);
}

}  // namespace orbit
