// Dense products C = alpha * A B (+ fused epilogue) on MFMA, used by every
// linear layer of the model: the forward x W (A K-major, B N-major), the input
// gradient dY W^T (both K-major) and the weight gradient X^T dY (both
// M/N-major, reduction over tokens).
#pragma once
#include "common.h"

namespace orbit {

struct Gemm {
  // C[M, N] (+)= alpha * sum_k A[m, k] B[k, n], batched over `batch`
  const void* A = nullptr;  int64_t lda = 0;  bool a_kmajor = true;   // A[m,k] at m*lda+k, else k*lda+m
  const void* B = nullptr;  int64_t ldb = 0;  bool b_kmajor = false;  // B[k,n] at n*ldb+k, else k*ldb+n
  // concatenated K: rows k >= k_split of an N-major B are read from B2 (row k - k_split)
  const void* B2 = nullptr; int k_split = 0;
  void* C = nullptr;        int64_t ldc = 0;
  int M = 0, N = 0, K = 0;
  int batch = 1;
  int64_t sA = 0, sB = 0, sB2 = 0, sC = 0;      // batch strides (elements)
  // epilogue, applied in this order to the float32 accumulator v:
  float alpha = 1.f;                             // v *= alpha
  bool accumulate = false;                       // v += C[m,n]     (float32 C only)
  const void* bias = nullptr; int64_t sBias = 0; // v += bias[n]    (dtype; batch stride sBias)
  void* gelu_out = nullptr;  int64_t ldgo = 0;   // store v (dtype), then v = GELU(v)
  const void* gelu_in = nullptr; int64_t ldgi = 0; // v *= GELU'(gelu_in[m,n])
  const void* res = nullptr; int64_t ldr = 0; int64_t sR = 0;
  int res_row_mod = 0;                           // v += res[(m % mod or m), n]
  bool out_f32 = false;                          // C is float32 (else dtype)
  // weight-gradient products only (A M-major, B N-major): also the column sums
  // of B over the K range (a bias gradient) as float32 partials, partial p of
  // column n of batch b at bsum[(p * batch + b) * N + n] for p < gemm_bsum_parts(g)
  // (at most bsum_max_parts partials)
  float* bsum = nullptr;
  int bsum_max_parts = 1;
  orbit_dtype dtype = ORBIT_BF16;                // operand type of A and B
  // operands read once by this product (bf16, both K-major, 64x64 tiles): their
  // tiles are loaded non-temporally
  bool stream = false;
  const char* tag = "gemm";                      // name prefix for timing
};

// bytes of float32 split-K partials the product may use (0 if none)
size_t gemm_workspace_bytes(const Gemm& g);
// number of column-sum partials gemm() writes for g.bsum (0: the product's
// kernel does not form them, and g.bsum must be NULL)
int gemm_bsum_parts(const Gemm& g);
orbit_status gemm(const Gemm& g, void* ws, size_t ws_bytes, hipStream_t s);

}  // namespace orbit
