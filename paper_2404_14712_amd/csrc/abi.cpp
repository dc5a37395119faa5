// C ABI entry points: argument validation, carving of the caller's saved /
// workspace buffers, and the kernel sequence of each call on one stream.
#include <string.h>

#include <algorithm>

#include "agg.h"
#include "gemm.h"
#include "kernels.h"

using namespace orbit;

namespace {

size_t esz(int dt) { return dt == ORBIT_BF16 ? 2 : 4; }
hipStream_t S(void* st) { return static_cast<hipStream_t>(st); }

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

#define REQ(cond, code, ...)        \
  do {                              \
    if (!(cond)) {                  \
      set_error(__VA_ARGS__);       \
      return code;                  \
    }                               \
  } while (0)

#define PTR(p, name)                                                        \
  do {                                                                      \
    REQ((p) != nullptr, ORBIT_E_ARG, "%s: %s is NULL", fn, name);           \
    REQ(aligned16(p), ORBIT_E_ARG, "%s: %s is not 16-byte aligned", fn, name); \
  } while (0)

#define OPT_PTR(p, name)                                                    \
  do {                                                                      \
    if (p) REQ(aligned16(p), ORBIT_E_ARG, "%s: %s is not 16-byte aligned", fn, name); \
  } while (0)

orbit_status check_dtype(const char* fn, int dt) {
  REQ(dt == ORBIT_F32 || dt == ORBIT_BF16, ORBIT_E_ARG, "%s: dtype %d is not ORBIT_F32 or ORBIT_BF16", fn, dt);
  return ORBIT_OK;
}

// attention head widths with kernels: 32, 64 and 128 in both dtypes; 192 and
// 256 (the paper's 1B/113B and 10B head widths) in bf16
orbit_status head_dim_check(const char* fn, int dt, int dh) {
  REQ(dh == 32 || dh == 64 || dh == 128 || (dt == ORBIT_BF16 && (dh == 192 || dh == 256)), ORBIT_E_UNSUPPORTED,
      "%s: head_dim %d unsupported (32, 64, 128; 192 and 256 in bf16)", fn, dh);
  return ORBIT_OK;
}

// ---------------------------------------------------------------------------
// block
// ---------------------------------------------------------------------------
struct BlockDims {
  int B, L, d, H, dh, A, F;
  int64_t T;
  int qk;
  float eps;
  orbit_dtype dt;
};

orbit_status block_dims(const char* fn, const orbit_block_desc* desc, BlockDims* o) {
  REQ(desc != nullptr, ORBIT_E_ARG, "%s: desc is NULL", fn);
  ORBIT_TRY(check_dtype(fn, desc->dtype));
  const orbit_block_desc& d = *desc;
  REQ(d.B > 0 && d.L > 0 && d.d > 0 && d.heads > 0 && d.head_dim > 0 && d.mlp > 0, ORBIT_E_ARG,
      "%s: sizes must be positive (B=%d L=%d d=%d heads=%d head_dim=%d mlp=%d)", fn, d.B, d.L, d.d, d.heads,
      d.head_dim, d.mlp);
  ORBIT_TRY(head_dim_check(fn, d.dtype, d.head_dim));
  REQ(d.d % 8 == 0 && d.mlp % 8 == 0, ORBIT_E_ARG, "%s: d=%d and mlp=%d must be multiples of 8", fn, d.d, d.mlp);
  REQ(d.d <= 16384, ORBIT_E_UNSUPPORTED, "%s: d=%d exceeds 16384", fn, d.d);
  REQ(d.qk_norm == 0 || d.qk_norm == 1, ORBIT_E_ARG, "%s: qk_norm must be 0 or 1", fn);
  REQ(d.eps > 0.f, ORBIT_E_ARG, "%s: eps must be positive", fn);
  REQ((int64_t)d.B * d.L < (1ll << 31) && (int64_t)d.heads * d.head_dim * 3 < (1ll << 31), ORBIT_E_UNSUPPORTED,
      "%s: sizes too large", fn);
  // attention addresses a (sample, head) slice of the [L, 3A] projections with
  // 32-bit byte offsets; QK-LayerNorm and the attention preprocess index
  // (token, head) rows in 32 bits
  REQ((int64_t)d.L * d.heads * d.head_dim * 3 * 4 < (1ll << 31) && (int64_t)d.B * d.L * d.heads * 2 < (1ll << 31),
      ORBIT_E_UNSUPPORTED, "%s: L=%d with %d heads of %d exceeds the 32-bit attention slice offsets", fn, d.L,
      d.heads, d.head_dim);
  o->B = d.B; o->L = d.L; o->d = d.d; o->H = d.heads; o->dh = d.head_dim; o->A = d.heads * d.head_dim;
  o->F = d.mlp; o->T = (int64_t)d.B * d.L; o->qk = d.qk_norm; o->eps = d.eps; o->dt = (orbit_dtype)d.dtype;
  return ORBIT_OK;
}

struct BlockSaved {
  float *mu1, *r1;
  void* h1;
  void* qkv;
  void* qkn;
  float *qmu, *qr;
  void* o;
  float* o32;
  float* lse;
  void* x1;
  float *mu2, *r2;
  void* h2;
  void* u;
  void* g;
};

BlockSaved carve_block_saved(const BlockDims& z, void* base, size_t* used) {
  Carver c(base);
  const size_t e = esz(z.dt);
  BlockSaved s{};
  s.mu1 = c.take<float>(z.T);
  s.r1 = c.take<float>(z.T);
  s.h1 = c.take<char>(z.T * z.d * e);
  s.qkv = c.take<char>(z.T * 3 * z.A * e);
  if (z.qk) {
    s.qkn = c.take<char>(z.T * 2 * z.A * e);
    s.qmu = c.take<float>(z.T * 2 * z.H);
    s.qr = c.take<float>(z.T * 2 * z.H);
  }
  s.o = c.take<char>(z.T * z.A * e);
  s.o32 = z.dt == ORBIT_BF16 ? c.take<float>(z.T * z.A) : nullptr;
  s.lse = c.take<float>(z.T * z.H);
  s.x1 = c.take<char>(z.T * z.d * e);
  s.mu2 = c.take<float>(z.T);
  s.r2 = c.take<float>(z.T);
  s.h2 = c.take<char>(z.T * z.d * e);
  s.u = c.take<char>(z.T * z.F * e);
  s.g = c.take<char>(z.T * z.F * e);
  if (used) *used = c.used();
  return s;
}

size_t block_saved_bytes(const BlockDims& z) {
  size_t u = 0;
  carve_block_saved(z, nullptr, &u);
  return u;
}

struct BlockWs {
  void* du;    // [T, F]
  void* dx1;   // [T, d]
  void* dh;    // [T, d]
  void* dO;    // [T, A]
  void* dqkv;  // [T, 3A]
  float* D;    // attention backward workspace
  float *p_fc1, *p_fc2, *p_ln2, *p_qkv, *p_ln1;  // column-sum partials
  void* qws;
  void* gws;
  size_t gws_bytes;
};

size_t block_gemm_ws(const BlockDims& z) {
  // every product of the block (forward and backward) with its shapes
  Gemm g;
  g.dtype = z.dt;
  size_t m = 0;
  const int T = (int)z.T;
  const int shapes[][5] = {
      // M, N, K, a_kmajor, b_kmajor
      {T, 3 * z.A, z.d, 1, 0}, {T, z.d, z.A, 1, 0}, {T, z.F, z.d, 1, 0}, {T, z.d, z.F, 1, 0},
      {z.F, z.d, T, 0, 0},     {T, z.F, z.d, 1, 1}, {z.d, z.F, T, 0, 0}, {T, z.d, z.F, 1, 1},
      {z.A, z.d, T, 0, 0},     {T, z.A, z.d, 1, 1}, {z.d, 3 * z.A, T, 0, 0}, {T, z.d, 3 * z.A, 1, 1}};
  for (auto& sh : shapes) {
    g.M = sh[0]; g.N = sh[1]; g.K = sh[2]; g.a_kmajor = sh[3]; g.b_kmajor = sh[4];
    m = std::max(m, gemm_workspace_bytes(g));
  }
  return m;
}

size_t block_ws_layout(const BlockDims& z, void* base, size_t bytes, BlockWs* w, bool inference_saved) {
  Carver c(base);
  const size_t e = esz(z.dt);
  if (inference_saved) c.take<char>(block_saved_bytes(z));
  BlockWs t{};
  t.du = c.take<char>(z.T * z.F * e);
  t.dx1 = c.take<char>(z.T * z.d * e);
  t.dh = c.take<char>(z.T * z.d * e);
  t.dO = c.take<char>(z.T * z.A * e);
  t.dqkv = c.take<char>(z.T * 3 * z.A * e);
  t.D = static_cast<float*>(static_cast<void*>(c.take<char>(attn_bwd_workspace_bytes(z.B, z.H, z.L, z.dh))));
  // partials of the block's column reductions (all finished by one launch)
  const int T = (int)z.T;
  t.p_fc1 = c.take<float>(colsum_part_bytes(T, z.F, false) / sizeof(float));
  t.p_fc2 = c.take<float>(colsum_part_bytes(T, z.d, false) / sizeof(float));
  t.p_ln2 = c.take<float>(ln_bwd_cols_part_bytes(T, z.d, true) / sizeof(float));
  t.p_qkv = c.take<float>(colsum_part_bytes(T, 3 * z.A, false) / sizeof(float));
  t.p_ln1 = c.take<float>(ln_bwd_cols_part_bytes(T, z.d, false) / sizeof(float));
  t.qws = c.take<char>(qk_norm_bwd_workspace_bytes(z.dh));
  const size_t g = block_gemm_ws(z);
  t.gws = c.take<char>(g);
  const size_t used = c.used();
  t.gws_bytes = base ? (bytes > used - g ? bytes - (used - g) : 0) : g;
  if (w) *w = t;
  return used;
}

size_t block_ws_bytes(const BlockDims& z) {
  // the backward layout; the forward needs only the GEMM part (plus the
  // saved-tensor region when called without `saved`)
  return block_ws_layout(z, nullptr, 0, nullptr, true);
}

// The forward's kernel sequence, writing the tensors the backward reads into
// `sv`. With y == NULL the last product (fc2, whose output the backward does
// not read) is skipped: the recompute of the activation-checkpoint backward.
orbit_status block_forward_steps(const BlockDims& z, const orbit_block_params* p, const void* x, void* y,
                                 const BlockSaved& sv, const BlockWs& w, hipStream_t s) {
  const int T = (int)z.T;
  const orbit_dtype dt = z.dt;
  ORBIT_TRY(layernorm_fwd(dt, x, z.d, p->ln1_g, p->ln1_b, sv.h1, z.d, sv.mu1, sv.r1, T, z.d, z.eps, s));
  {
    Gemm g; g.dtype = dt; g.tag = "qkv";
    g.A = sv.h1; g.lda = z.d; g.B = p->w_qkv; g.ldb = 3 * z.A; g.C = sv.qkv; g.ldc = 3 * z.A;
    g.M = T; g.N = 3 * z.A; g.K = z.d; g.bias = p->b_qkv;
    ORBIT_TRY(gemm(g, w.gws, w.gws_bytes, s));
  }
  const size_t e = esz(dt);
  AttnIO io{};
  io.B = z.B; io.H = z.H; io.L = z.L; io.dh = z.dh;
  io.v = static_cast<char*>(sv.qkv) + 2 * z.A * e; io.ldv = 3 * z.A;
  if (z.qk) {
    ORBIT_TRY(qk_norm_fwd(dt, sv.qkv, 3 * z.A, sv.qkn, 2 * z.A, p->qn_g, p->qn_b, p->kn_g, p->kn_b, sv.qmu, sv.qr,
                          T, z.H, z.dh, z.eps, s));
    io.q = sv.qkn; io.ldq = 2 * z.A;
    io.k = static_cast<char*>(sv.qkn) + z.A * e; io.ldk = 2 * z.A;
  } else {
    io.q = sv.qkv; io.ldq = 3 * z.A;
    io.k = static_cast<char*>(sv.qkv) + z.A * e; io.ldk = 3 * z.A;
  }
  // the attention backward's workspace is idle during the forward and holds
  // the forward's split partials
  ORBIT_TRY(attn_fwd(dt, io, sv.o, z.A, sv.lse, sv.o32, z.A, w.D, attn_bwd_workspace_bytes(z.B, z.H, z.L, z.dh), s));
  {
    Gemm g; g.dtype = dt; g.tag = "proj";
    g.A = sv.o; g.lda = z.A; g.B = p->w_proj; g.ldb = z.d; g.C = sv.x1; g.ldc = z.d;
    g.M = T; g.N = z.d; g.K = z.A; g.bias = p->b_proj; g.res = x; g.ldr = z.d;
    ORBIT_TRY(gemm(g, w.gws, w.gws_bytes, s));
  }
  ORBIT_TRY(layernorm_fwd(dt, sv.x1, z.d, p->ln2_g, p->ln2_b, sv.h2, z.d, sv.mu2, sv.r2, T, z.d, z.eps, s));
  {
    Gemm g; g.dtype = dt; g.tag = "fc1";
    g.A = sv.h2; g.lda = z.d; g.B = p->w_fc1; g.ldb = z.F; g.C = sv.g; g.ldc = z.F;
    g.M = T; g.N = z.F; g.K = z.d; g.bias = p->b_fc1; g.gelu_out = sv.u; g.ldgo = z.F;
    ORBIT_TRY(gemm(g, w.gws, w.gws_bytes, s));
  }
  if (y) {
    Gemm g; g.dtype = dt; g.tag = "fc2";
    g.A = sv.g; g.lda = z.F; g.B = p->w_fc2; g.ldb = z.d; g.C = y; g.ldc = z.d;
    g.M = T; g.N = z.d; g.K = z.F; g.bias = p->b_fc2; g.res = sv.x1; g.ldr = z.d;
    ORBIT_TRY(gemm(g, w.gws, w.gws_bytes, s));
  }
  return ORBIT_OK;
}

}  // namespace

extern "C" {

size_t orbit_vit_block_saved_bytes(const orbit_block_desc* desc) {
  BlockDims z;
  if (block_dims("orbit_vit_block_saved_bytes", desc, &z) != ORBIT_OK) return 0;
  return block_saved_bytes(z);
}

size_t orbit_vit_block_workspace_bytes(const orbit_block_desc* desc) {
  BlockDims z;
  if (block_dims("orbit_vit_block_workspace_bytes", desc, &z) != ORBIT_OK) return 0;
  return block_ws_bytes(z);
}

orbit_status orbit_vit_block_fwd(const orbit_block_desc* desc, const orbit_block_params* p, const void* x, void* y,
                                 void* saved, void* ws, size_t ws_bytes, void* stream) {
  const char* fn = "orbit_vit_block_fwd";
  clear_error();
  BlockDims z;
  ORBIT_TRY(block_dims(fn, desc, &z));
  REQ(p != nullptr, ORBIT_E_ARG, "%s: params is NULL", fn);
  PTR(x, "x");
  PTR(y, "y");
  REQ(x != y, ORBIT_E_ARG, "%s: y must not alias x", fn);
  PTR(p->ln1_g, "ln1_g"); PTR(p->ln1_b, "ln1_b"); PTR(p->w_qkv, "w_qkv"); PTR(p->b_qkv, "b_qkv");
  PTR(p->w_proj, "w_proj"); PTR(p->b_proj, "b_proj"); PTR(p->ln2_g, "ln2_g"); PTR(p->ln2_b, "ln2_b");
  PTR(p->w_fc1, "w_fc1"); PTR(p->b_fc1, "b_fc1"); PTR(p->w_fc2, "w_fc2"); PTR(p->b_fc2, "b_fc2");
  if (z.qk) { PTR(p->qn_g, "qn_g"); PTR(p->qn_b, "qn_b"); PTR(p->kn_g, "kn_g"); PTR(p->kn_b, "kn_b"); }
  OPT_PTR(saved, "saved");
  PTR(ws, "ws");
  const size_t need = block_ws_bytes(z);
  REQ(ws_bytes >= need, ORBIT_E_ARG, "%s: workspace of %zu bytes is smaller than the %zu required", fn, ws_bytes,
      need);
  hipStream_t s = S(stream);
  const bool inference = saved == nullptr;
  BlockWs w;
  block_ws_layout(z, ws, ws_bytes, &w, true);
  const BlockSaved sv = carve_block_saved(z, inference ? ws : saved, nullptr);
  return block_forward_steps(z, p, x, y, sv, w, s);
}

orbit_status orbit_vit_block_bwd(const orbit_block_desc* desc, const orbit_block_params* p, const void* x,
                                 const void* saved, const void* dy, void* dx, const orbit_block_grads* gr,
                                 int accumulate, void* ws, size_t ws_bytes, void* stream) {
  const char* fn = "orbit_vit_block_bwd";
  clear_error();
  BlockDims z;
  ORBIT_TRY(block_dims(fn, desc, &z));
  REQ(p != nullptr && gr != nullptr, ORBIT_E_ARG, "%s: params or grads is NULL", fn);
  PTR(x, "x"); OPT_PTR(saved, "saved"); PTR(dy, "dy"); PTR(dx, "dx"); PTR(ws, "ws");
  PTR(p->ln1_g, "ln1_g"); PTR(p->w_qkv, "w_qkv"); PTR(p->w_proj, "w_proj"); PTR(p->ln2_g, "ln2_g");
  PTR(p->w_fc1, "w_fc1"); PTR(p->w_fc2, "w_fc2");
  if (z.qk) { PTR(p->qn_g, "qn_g"); PTR(p->kn_g, "kn_g"); }
  REQ(dx != x, ORBIT_E_ARG, "%s: dx must not alias x", fn);
  const bool recompute = saved == nullptr;
  if (recompute) {
    // the forward's other parameters are read again by the recompute
    PTR(p->ln1_b, "ln1_b"); PTR(p->b_qkv, "b_qkv"); PTR(p->b_proj, "b_proj"); PTR(p->ln2_b, "ln2_b");
    PTR(p->b_fc1, "b_fc1");
    if (z.qk) { PTR(p->qn_b, "qn_b"); PTR(p->kn_b, "kn_b"); }
  }
  PTR(gr->ln1_g, "grads.ln1_g"); PTR(gr->ln1_b, "grads.ln1_b"); PTR(gr->w_qkv, "grads.w_qkv");
  PTR(gr->b_qkv, "grads.b_qkv"); PTR(gr->qn_g, "grads.qn_g"); PTR(gr->qn_b, "grads.qn_b");
  PTR(gr->kn_g, "grads.kn_g"); PTR(gr->kn_b, "grads.kn_b"); PTR(gr->w_proj, "grads.w_proj");
  PTR(gr->b_proj, "grads.b_proj"); PTR(gr->ln2_g, "grads.ln2_g"); PTR(gr->ln2_b, "grads.ln2_b");
  PTR(gr->w_fc1, "grads.w_fc1"); PTR(gr->b_fc1, "grads.b_fc1"); PTR(gr->w_fc2, "grads.w_fc2");
  PTR(gr->b_fc2, "grads.b_fc2");
  REQ(accumulate == 0 || accumulate == 1, ORBIT_E_ARG, "%s: accumulate must be 0 or 1", fn);
  const size_t need = block_ws_bytes(z);
  REQ(ws_bytes >= need, ORBIT_E_ARG, "%s: workspace of %zu bytes is smaller than the %zu required", fn, ws_bytes,
      need);
  hipStream_t s = S(stream);
  BlockWs w;
  block_ws_layout(z, ws, ws_bytes, &w, true);
  // activation checkpointing: the saved tensors are recomputed from x into the
  // workspace's saved-tensor region (the region the inference forward uses)
  const BlockSaved sv = carve_block_saved(z, recompute ? ws : const_cast<void*>(saved), nullptr);
  if (recompute) ORBIT_TRY(block_forward_steps(z, p, x, nullptr, sv, w, s));
  const int T = (int)z.T;
  const orbit_dtype dt = z.dt;
  const size_t e = esz(dt);
  const bool acc = accumulate != 0;

  ColFinal fin;  // parameter-gradient column sums, finished together at the end
  // a bias gradient is the column sum of its weight-gradient product's B
  // operand: taken from that product where its kernel forms it, else from a
  // column-sum job
  auto dw_bias = [&](Gemm& g, float* part, float* out) -> bool {
    g.bsum_max_parts = colsum_chunks(T);
    const int parts = gemm_bsum_parts(g);
    if (parts <= 0 || parts > colsum_chunks(T)) return false;
    g.bsum = part;
    fin.add(part, g.N, parts, g.N, out);
    return true;
  };
  auto bias_job = [](ColJob& j, const void* src, int64_t n, float* part, float* out) {
    j.src = src; j.ld = n; j.n = (int)n; j.part = part; j.out_sum = out;
  };
  // feed-forward sub-layer
  bool fused_fc2, fused_fc1;
  {
    Gemm g; g.dtype = dt; g.tag = "fc2_dw";
    g.A = sv.g; g.lda = z.F; g.a_kmajor = false; g.B = dy; g.ldb = z.d; g.b_kmajor = false;
    g.C = gr->w_fc2; g.ldc = z.d; g.out_f32 = true; g.accumulate = acc;
    g.M = z.F; g.N = z.d; g.K = T;
    fused_fc2 = dw_bias(g, w.p_fc2, gr->b_fc2);
    ORBIT_TRY(gemm(g, w.gws, w.gws_bytes, s));
  }
  {
    Gemm g; g.dtype = dt; g.tag = "fc2_dx";
    g.A = dy; g.lda = z.d; g.B = p->w_fc2; g.ldb = z.d; g.b_kmajor = true;
    g.C = w.du; g.ldc = z.F; g.M = T; g.N = z.F; g.K = z.d; g.gelu_in = sv.u; g.ldgi = z.F;
    ORBIT_TRY(gemm(g, w.gws, w.gws_bytes, s));
  }
  {
    Gemm g; g.dtype = dt; g.tag = "fc1_dw";
    g.A = sv.h2; g.lda = z.d; g.a_kmajor = false; g.B = w.du; g.ldb = z.F; g.b_kmajor = false;
    g.C = gr->w_fc1; g.ldc = z.F; g.out_f32 = true; g.accumulate = acc;
    g.M = z.d; g.N = z.F; g.K = T;
    fused_fc1 = dw_bias(g, w.p_fc1, gr->b_fc1);
    ORBIT_TRY(gemm(g, w.gws, w.gws_bytes, s));
  }
  {
    ColJob j[2];
    int nj = 0;
    if (!fused_fc1) bias_job(j[nj++], w.du, z.F, w.p_fc1, gr->b_fc1);
    if (!fused_fc2) bias_job(j[nj++], dy, z.d, w.p_fc2, gr->b_fc2);
    if (nj) ORBIT_TRY(colsum_partials(dt, j, nj, T, s));
    for (int i = 0; i < nj; ++i) fin.add_job(j[i], T);
  }
  {
    Gemm g; g.dtype = dt; g.tag = "fc1_dx";
    g.A = w.du; g.lda = z.F; g.B = p->w_fc1; g.ldb = z.F; g.b_kmajor = true;
    g.C = w.dh; g.ldc = z.d; g.M = T; g.N = z.d; g.K = z.F;
    ORBIT_TRY(gemm(g, w.gws, w.gws_bytes, s));
  }
  // LN2 backward; the chunk sums of its rows give the LN2 parameter gradients
  // and, summed over its output dx1, the projection's bias gradient
  ORBIT_TRY(layernorm_bwd_cols(dt, w.dh, z.d, sv.x1, z.d, sv.mu2, sv.r2, p->ln2_g, dy, w.dx1, z.d, T, z.d, w.p_ln2,
                               gr->ln2_b, gr->ln2_g, gr->b_proj, fin, s));
  {
    Gemm g; g.dtype = dt; g.tag = "proj_dw";
    g.A = sv.o; g.lda = z.A; g.a_kmajor = false; g.B = w.dx1; g.ldb = z.d; g.b_kmajor = false;
    g.C = gr->w_proj; g.ldc = z.d; g.out_f32 = true; g.accumulate = acc;
    g.M = z.A; g.N = z.d; g.K = T;
    ORBIT_TRY(gemm(g, w.gws, w.gws_bytes, s));
  }
  // attention sub-layer
  {
    Gemm g; g.dtype = dt; g.tag = "proj_dx";
    g.A = w.dx1; g.lda = z.d; g.B = p->w_proj; g.ldb = z.d; g.b_kmajor = true;
    g.C = w.dO; g.ldc = z.A; g.M = T; g.N = z.A; g.K = z.d;
    ORBIT_TRY(gemm(g, w.gws, w.gws_bytes, s));
  }
  AttnIO io{};
  io.B = z.B; io.H = z.H; io.L = z.L; io.dh = z.dh;
  io.v = static_cast<char*>(sv.qkv) + 2 * z.A * e; io.ldv = 3 * z.A;
  if (z.qk) {
    io.q = sv.qkn; io.ldq = 2 * z.A; io.k = static_cast<char*>(sv.qkn) + z.A * e; io.ldk = 2 * z.A;
  } else {
    io.q = sv.qkv; io.ldq = 3 * z.A; io.k = static_cast<char*>(sv.qkv) + z.A * e; io.ldk = 3 * z.A;
  }
  char* dq = static_cast<char*>(w.dqkv);
  if (sv.o32)
    ORBIT_TRY(attn_bwd(dt, io, sv.o32, z.A, 1, sv.lse, w.dO, z.A, dq, dq + z.A * e, dq + 2 * z.A * e, 3 * z.A, w.D, s));
  else
    ORBIT_TRY(attn_bwd(dt, io, sv.o, z.A, 0, sv.lse, w.dO, z.A, dq, dq + z.A * e, dq + 2 * z.A * e, 3 * z.A, w.D, s));
  if (z.qk) {
    ORBIT_TRY(qk_norm_bwd(dt, w.dqkv, 3 * z.A, sv.qkv, 3 * z.A, sv.qmu, sv.qr, p->qn_g, p->kn_g, gr->qn_g, gr->qn_b,
                          gr->kn_g, gr->kn_b, accumulate, T, z.H, z.dh, w.qws, &fin, s));
  } else if (!acc) {
    ORBIT_TRY(fill_f32(gr->qn_g, z.dh, 0.f, s));
    ORBIT_TRY(fill_f32(gr->qn_b, z.dh, 0.f, s));
    ORBIT_TRY(fill_f32(gr->kn_g, z.dh, 0.f, s));
    ORBIT_TRY(fill_f32(gr->kn_b, z.dh, 0.f, s));
  }
  bool fused_qkv;
  {
    Gemm g; g.dtype = dt; g.tag = "qkv_dw";
    g.A = sv.h1; g.lda = z.d; g.a_kmajor = false; g.B = w.dqkv; g.ldb = 3 * z.A; g.b_kmajor = false;
    g.C = gr->w_qkv; g.ldc = 3 * z.A; g.out_f32 = true; g.accumulate = acc;
    g.M = z.d; g.N = 3 * z.A; g.K = T;
    fused_qkv = dw_bias(g, w.p_qkv, gr->b_qkv);
    ORBIT_TRY(gemm(g, w.gws, w.gws_bytes, s));
  }
  {
    Gemm g; g.dtype = dt; g.tag = "qkv_dx";
    g.A = w.dqkv; g.lda = 3 * z.A; g.B = p->w_qkv; g.ldb = 3 * z.A; g.b_kmajor = true;
    g.C = w.dh; g.ldc = z.d; g.M = T; g.N = z.d; g.K = 3 * z.A;
    ORBIT_TRY(gemm(g, w.gws, w.gws_bytes, s));
  }
  ORBIT_TRY(layernorm_bwd_cols(dt, w.dh, z.d, x, z.d, sv.mu1, sv.r1, p->ln1_g, w.dx1, dx, z.d, T, z.d, w.p_ln1,
                               gr->ln1_b, gr->ln1_g, nullptr, fin, s));
  if (!fused_qkv) {
    ColJob j[1];
    bias_job(j[0], w.dqkv, 3 * z.A, w.p_qkv, gr->b_qkv);
    ORBIT_TRY(colsum_partials(dt, j, 1, T, s));
    fin.add_job(j[0], T);
  }
  return fin.run(accumulate, s);
}

// ---------------------------------------------------------------------------
// patch embedding
// ---------------------------------------------------------------------------
static orbit_status embed_check(const char* fn, const orbit_embed_desc* d) {
  REQ(d != nullptr, ORBIT_E_ARG, "%s: desc is NULL", fn);
  ORBIT_TRY(check_dtype(fn, d->dtype));
  REQ(d->B > 0 && d->V > 0 && d->H > 0 && d->W > 0 && d->d > 0, ORBIT_E_ARG, "%s: sizes must be positive", fn);
  REQ(d->patch == 4, ORBIT_E_UNSUPPORTED, "%s: patch size %d unsupported (4)", fn, d->patch);
  REQ(d->H % 4 == 0 && d->W % 4 == 0, ORBIT_E_ARG, "%s: H=%d and W=%d must be multiples of the patch", fn, d->H,
      d->W);
  REQ(d->d % 8 == 0, ORBIT_E_ARG, "%s: d=%d must be a multiple of 8", fn, d->d);
  REQ((int64_t)d->B * (d->H / 4) * (d->W / 4) * d->V < (1ll << 31), ORBIT_E_UNSUPPORTED, "%s: too many tokens", fn);
  return ORBIT_OK;
}

orbit_status orbit_patch_embed(const orbit_embed_desc* desc, const float* img, const void* w_pe, const void* b_pe,
                               const void* ve, void* tok, void* stream) {
  const char* fn = "orbit_patch_embed";
  clear_error();
  ORBIT_TRY(embed_check(fn, desc));
  PTR(img, "img"); PTR(w_pe, "w_pe"); PTR(b_pe, "b_pe"); OPT_PTR(ve, "ve"); PTR(tok, "tok");
  return patch_embed_fwd((orbit_dtype)desc->dtype, img, w_pe, b_pe, ve, tok, desc->B, desc->V, desc->H, desc->W, 4,
                         desc->d, S(stream));
}

size_t orbit_patch_embed_workspace_bytes(const orbit_embed_desc* desc) {
  if (embed_check("orbit_patch_embed_workspace_bytes", desc) != ORBIT_OK) return 0;
  return patch_embed_bwd_workspace_bytes(desc->B, desc->V, desc->H, desc->W, 4, desc->d);
}

orbit_status orbit_patch_embed_bwd(const orbit_embed_desc* desc, const float* img, const void* dtok, float* dw_pe,
                                   float* db_pe, float* dve, int accumulate, void* ws, size_t ws_bytes,
                                   void* stream) {
  const char* fn = "orbit_patch_embed_bwd";
  clear_error();
  ORBIT_TRY(embed_check(fn, desc));
  PTR(img, "img"); PTR(dtok, "dtok"); PTR(dw_pe, "dw_pe"); PTR(db_pe, "db_pe"); OPT_PTR(dve, "dve"); PTR(ws, "ws");
  REQ(accumulate == 0 || accumulate == 1, ORBIT_E_ARG, "%s: accumulate must be 0 or 1", fn);
  const size_t need = patch_embed_bwd_workspace_bytes(desc->B, desc->V, desc->H, desc->W, 4, desc->d);
  REQ(ws_bytes >= need, ORBIT_E_ARG, "%s: workspace of %zu bytes is smaller than the %zu required", fn, ws_bytes,
      need);
  return patch_embed_bwd((orbit_dtype)desc->dtype, img, dtok, dw_pe, db_pe, dve, accumulate, desc->B, desc->V,
                         desc->H, desc->W, 4, desc->d, ws, S(stream));
}

// ---------------------------------------------------------------------------
// variable aggregation
// ---------------------------------------------------------------------------
static orbit_status agg_check(const char* fn, const orbit_agg_desc* d) {
  REQ(d != nullptr, ORBIT_E_ARG, "%s: desc is NULL", fn);
  ORBIT_TRY(check_dtype(fn, d->dtype));
  REQ(d->B > 0 && d->L > 0 && d->V > 0 && d->d > 0 && d->heads > 0 && d->head_dim > 0, ORBIT_E_ARG,
      "%s: sizes must be positive", fn);
  REQ(d->d % 8 == 0 && d->head_dim % 8 == 0, ORBIT_E_ARG, "%s: d and head_dim must be multiples of 8", fn);
  REQ(d->head_dim <= 8192, ORBIT_E_UNSUPPORTED, "%s: head_dim=%d above 8192", fn, d->head_dim);
  // per-token rows of `heads` values are read as 16-byte vectors
  REQ((d->heads * (int)esz(d->dtype)) % 16 == 0, ORBIT_E_UNSUPPORTED,
      "%s: heads=%d must be a multiple of %d for this dtype", fn, d->heads, 16 / (int)esz(d->dtype));
  // the softmax over variables runs one wave per token with 64 / heads lanes per head
  REQ(64 % d->heads == 0, ORBIT_E_UNSUPPORTED, "%s: heads=%d must divide 64", fn, d->heads);
  REQ((int64_t)d->B * d->L * d->V < (1ll << 31), ORBIT_E_UNSUPPORTED, "%s: too many tokens", fn);
  return ORBIT_OK;
}

size_t orbit_var_aggregate_saved_bytes(const orbit_agg_desc* desc) {
  if (agg_check("orbit_var_aggregate_saved_bytes", desc) != ORBIT_OK) return 0;
  return agg_saved_bytes(*desc);
}

size_t orbit_var_aggregate_workspace_bytes(const orbit_agg_desc* desc) {
  if (agg_check("orbit_var_aggregate_workspace_bytes", desc) != ORBIT_OK) return 0;
  return agg_workspace_bytes(*desc);
}

orbit_status orbit_var_aggregate(const orbit_agg_desc* desc, const void* tok, const orbit_agg_params* p, void* z,
                                 void* saved, void* ws, size_t ws_bytes, void* stream) {
  const char* fn = "orbit_var_aggregate";
  clear_error();
  ORBIT_TRY(agg_check(fn, desc));
  REQ(p != nullptr, ORBIT_E_ARG, "%s: params is NULL", fn);
  PTR(tok, "tok"); PTR(z, "z"); PTR(saved, "saved"); PTR(ws, "ws");
  PTR(p->q0, "q0"); PTR(p->w_q, "w_q"); PTR(p->b_q, "b_q"); PTR(p->w_k, "w_k"); PTR(p->b_k, "b_k");
  PTR(p->w_v, "w_v"); PTR(p->b_v, "b_v"); PTR(p->w_o, "w_o"); PTR(p->b_o, "b_o"); OPT_PTR(p->pos, "pos");
  const size_t need = agg_workspace_bytes(*desc);
  REQ(ws_bytes >= need, ORBIT_E_ARG, "%s: workspace of %zu bytes is smaller than the %zu required", fn, ws_bytes,
      need);
  return agg_forward(*desc, tok, *p, z, saved, ws, ws_bytes, S(stream));
}

orbit_status orbit_var_aggregate_bwd(const orbit_agg_desc* desc, const void* tok, const orbit_agg_params* p,
                                     const void* saved, const void* dz, void* dtok, const orbit_agg_grads* g,
                                     int accumulate, void* ws, size_t ws_bytes, void* stream) {
  const char* fn = "orbit_var_aggregate_bwd";
  clear_error();
  ORBIT_TRY(agg_check(fn, desc));
  REQ(p != nullptr && g != nullptr, ORBIT_E_ARG, "%s: params or grads is NULL", fn);
  PTR(tok, "tok"); PTR(saved, "saved"); PTR(dz, "dz"); PTR(dtok, "dtok"); PTR(ws, "ws");
  PTR(p->q0, "q0"); PTR(p->w_q, "w_q"); PTR(p->w_k, "w_k"); PTR(p->w_v, "w_v"); PTR(p->w_o, "w_o");
  PTR(g->q0, "grads.q0"); PTR(g->w_q, "grads.w_q"); PTR(g->b_q, "grads.b_q"); PTR(g->w_k, "grads.w_k");
  PTR(g->b_k, "grads.b_k"); PTR(g->w_v, "grads.w_v"); PTR(g->b_v, "grads.b_v"); PTR(g->w_o, "grads.w_o");
  PTR(g->b_o, "grads.b_o"); OPT_PTR(g->pos, "grads.pos");
  REQ(accumulate == 0 || accumulate == 1, ORBIT_E_ARG, "%s: accumulate must be 0 or 1", fn);
  const size_t need = agg_workspace_bytes(*desc);
  REQ(ws_bytes >= need, ORBIT_E_ARG, "%s: workspace of %zu bytes is smaller than the %zu required", fn, ws_bytes,
      need);
  return agg_backward(*desc, tok, *p, saved, dz, dtok, *g, accumulate, ws, ws_bytes, S(stream));
}

// ---------------------------------------------------------------------------
// head
// ---------------------------------------------------------------------------
static orbit_status head_check(const char* fn, const orbit_head_desc* d) {
  REQ(d != nullptr, ORBIT_E_ARG, "%s: desc is NULL", fn);
  ORBIT_TRY(check_dtype(fn, d->dtype));
  REQ(d->B > 0 && d->L > 0 && d->d > 0 && d->out > 0, ORBIT_E_ARG, "%s: sizes must be positive", fn);
  REQ(d->d % 8 == 0 && d->out % 8 == 0, ORBIT_E_ARG, "%s: d and out must be multiples of 8", fn);
  REQ(d->d <= 16384, ORBIT_E_UNSUPPORTED, "%s: d=%d exceeds 16384", fn, d->d);
  REQ(d->final_ln == 0 || d->final_ln == 1, ORBIT_E_ARG, "%s: final_ln must be 0 or 1", fn);
  REQ(d->eps > 0.f, ORBIT_E_ARG, "%s: eps must be positive", fn);
  REQ(d->hidden >= 0 && d->hidden <= 8, ORBIT_E_ARG, "%s: hidden=%d must be 0..8", fn, d->hidden);
  REQ((int64_t)d->B * d->L < (1ll << 31), ORBIT_E_UNSUPPORTED, "%s: too many tokens", fn);
  return ORBIT_OK;
}

// saved: LN_f statistics and output, then per hidden layer its
// pre-activation u_k and output g_k = GELU(u_k) ([T, d] each)
struct HeadSaved { float *mu, *r; void* hf; void* u[8]; void* g[8]; };
static HeadSaved carve_head_saved(const orbit_head_desc& d, void* base, size_t* used) {
  Carver c(base);
  const int64_t T = (int64_t)d.B * d.L;
  const size_t e = esz(d.dtype);
  HeadSaved s{};
  s.mu = c.take<float>(T);
  s.r = c.take<float>(T);
  s.hf = c.take<char>(T * d.d * e);
  for (int k = 0; k < d.hidden; ++k) {
    s.u[k] = c.take<char>(T * d.d * e);
    s.g[k] = c.take<char>(T * d.d * e);
  }
  if (used) *used = c.used();
  return s;
}

static size_t head_gemm_ws(const orbit_head_desc& d) {
  Gemm g;
  g.dtype = (orbit_dtype)d.dtype;
  const int T = d.B * d.L;
  size_t m = 0;
  for (int n : {d.out, d.d}) {
    if (n == d.d && d.hidden == 0) continue;
    g.a_kmajor = true; g.b_kmajor = false;
    g.M = T; g.N = n; g.K = d.d; m = std::max(m, gemm_workspace_bytes(g));
    g.M = d.d; g.N = n; g.K = T; g.a_kmajor = false; m = std::max(m, gemm_workspace_bytes(g));
    g.M = T; g.N = d.d; g.K = n; g.a_kmajor = true; g.b_kmajor = true; m = std::max(m, gemm_workspace_bytes(g));
  }
  return m;
}

// workspace: dpred in the compute dtype, the gradient of the current
// activation and of the next (ping-pong over the hidden layers), column-sum
// scratch and the GEMM split-K partials
struct HeadWs { void* dpb; void* dh[2]; void* cws; void* gws; size_t gws_bytes; };
static size_t head_ws_layout(const orbit_head_desc& d, void* base, size_t bytes, HeadWs* w) {
  Carver c(base);
  const int64_t T = (int64_t)d.B * d.L;
  HeadWs t{};
  t.dpb = c.take<char>(T * d.out * esz(d.dtype));
  t.dh[0] = c.take<char>(T * d.d * esz(d.dtype));
  t.dh[1] = d.hidden > 0 ? c.take<char>(T * d.d * esz(d.dtype)) : nullptr;
  t.cws = c.take<char>(std::max({colsum_workspace_bytes((int)T, d.out), colsum_workspace_bytes((int)T, d.d),
                                  ln_bwd_cols_part_bytes((int)T, d.d, false)}));
  const size_t g = head_gemm_ws(d);
  t.gws = c.take<char>(g);
  const size_t used = c.used();
  t.gws_bytes = base ? bytes - (used - g) : g;
  if (w) *w = t;
  return used;
}

size_t orbit_head_saved_bytes(const orbit_head_desc* desc) {
  if (head_check("orbit_head_saved_bytes", desc) != ORBIT_OK) return 0;
  size_t u = 0;
  carve_head_saved(*desc, nullptr, &u);
  return u;
}

size_t orbit_head_workspace_bytes(const orbit_head_desc* desc) {
  if (head_check("orbit_head_workspace_bytes", desc) != ORBIT_OK) return 0;
  size_t u = 0;
  carve_head_saved(*desc, nullptr, &u);
  return u + head_ws_layout(*desc, nullptr, 0, nullptr);
}

orbit_status orbit_head_fwd(const orbit_head_desc* desc, const void* x, const orbit_head_params* p, float* pred,
                            void* saved, void* ws, size_t ws_bytes, void* stream) {
  const char* fn = "orbit_head_fwd";
  clear_error();
  ORBIT_TRY(head_check(fn, desc));
  REQ(p != nullptr, ORBIT_E_ARG, "%s: params is NULL", fn);
  PTR(x, "x"); PTR(pred, "pred"); PTR(p->w_h, "w_h"); PTR(p->b_h, "b_h"); OPT_PTR(saved, "saved"); PTR(ws, "ws");
  if (desc->final_ln) { PTR(p->lnf_g, "lnf_g"); PTR(p->lnf_b, "lnf_b"); }
  if (desc->hidden) { PTR(p->w_hid, "w_hid"); PTR(p->b_hid, "b_hid"); }
  const size_t need = orbit_head_workspace_bytes(desc);
  REQ(ws_bytes >= need, ORBIT_E_ARG, "%s: workspace of %zu bytes is smaller than the %zu required", fn, ws_bytes,
      need);
  const orbit_head_desc& d = *desc;
  const orbit_dtype dt = (orbit_dtype)d.dtype;
  const size_t e = esz(dt);
  hipStream_t s = S(stream);
  size_t sv_bytes = 0;
  carve_head_saved(d, nullptr, &sv_bytes);
  const HeadSaved sv = carve_head_saved(d, saved ? saved : ws, nullptr);
  HeadWs w;
  head_ws_layout(d, static_cast<char*>(ws) + sv_bytes, ws_bytes - sv_bytes, &w);
  const int T = d.B * d.L;
  const void* hin = x;
  if (d.final_ln) {
    ORBIT_TRY(layernorm_fwd(dt, x, d.d, p->lnf_g, p->lnf_b, sv.hf, d.d, sv.mu, sv.r, T, d.d, d.eps, s));
    hin = sv.hf;
  }
  for (int k = 0; k < d.hidden; ++k) {
    // g_k = GELU(h W_k + b_k), pre-activation u_k stored by the epilogue
    Gemm g; g.dtype = dt; g.tag = "head_hidden";
    g.A = hin; g.lda = d.d; g.B = static_cast<const char*>(p->w_hid) + (size_t)k * d.d * d.d * e; g.ldb = d.d;
    g.C = sv.g[k]; g.ldc = d.d; g.M = T; g.N = d.d; g.K = d.d;
    g.bias = static_cast<const char*>(p->b_hid) + (size_t)k * d.d * e;
    g.gelu_out = sv.u[k]; g.ldgo = d.d;
    ORBIT_TRY(gemm(g, w.gws, w.gws_bytes, s));
    hin = sv.g[k];
  }
  Gemm g; g.dtype = dt; g.tag = "head";
  g.A = hin; g.lda = d.d; g.B = p->w_h; g.ldb = d.out; g.C = pred; g.ldc = d.out; g.out_f32 = true;
  g.M = T; g.N = d.out; g.K = d.d; g.bias = p->b_h;
  return gemm(g, w.gws, w.gws_bytes, s);
}

orbit_status orbit_head_bwd(const orbit_head_desc* desc, const void* x, const orbit_head_params* p,
                            const void* saved, const float* dpred, void* dx, const orbit_head_grads* gr,
                            int accumulate, void* ws, size_t ws_bytes, void* stream) {
  const char* fn = "orbit_head_bwd";
  clear_error();
  ORBIT_TRY(head_check(fn, desc));
  REQ(p != nullptr && gr != nullptr, ORBIT_E_ARG, "%s: params or grads is NULL", fn);
  PTR(x, "x"); PTR(saved, "saved"); PTR(dpred, "dpred"); PTR(dx, "dx"); PTR(p->w_h, "w_h"); PTR(ws, "ws");
  PTR(gr->w_h, "grads.w_h"); PTR(gr->b_h, "grads.b_h");
  if (desc->final_ln) {
    PTR(p->lnf_g, "lnf_g"); PTR(gr->lnf_g, "grads.lnf_g"); PTR(gr->lnf_b, "grads.lnf_b");
  }
  if (desc->hidden) {
    PTR(p->w_hid, "w_hid"); PTR(gr->w_hid, "grads.w_hid"); PTR(gr->b_hid, "grads.b_hid");
  }
  REQ(accumulate == 0 || accumulate == 1, ORBIT_E_ARG, "%s: accumulate must be 0 or 1", fn);
  const size_t need = orbit_head_workspace_bytes(desc);
  REQ(ws_bytes >= need, ORBIT_E_ARG, "%s: workspace of %zu bytes is smaller than the %zu required", fn, ws_bytes,
      need);
  const orbit_head_desc& d = *desc;
  const orbit_dtype dt = (orbit_dtype)d.dtype;
  const size_t e = esz(dt);
  hipStream_t s = S(stream);
  size_t sv_bytes = 0;
  carve_head_saved(d, nullptr, &sv_bytes);
  const HeadSaved sv = carve_head_saved(d, const_cast<void*>(saved), nullptr);
  HeadWs w;
  head_ws_layout(d, static_cast<char*>(ws) + sv_bytes, ws_bytes - sv_bytes, &w);
  const int T = d.B * d.L;
  const void* hf = d.final_ln ? sv.hf : x;
  const int nh = d.hidden;
  ORBIT_TRY(colsum_f32(dpred, d.out, T, d.out, gr->b_h, accumulate, w.cws, s));
  const void* dpb = dpred;
  if (dt == ORBIT_BF16) {
    ORBIT_TRY(cast_from_f32(dt, dpred, w.dpb, (int64_t)T * d.out, s));
    dpb = w.dpb;
  }
  {
    Gemm g; g.dtype = dt; g.tag = "head_dw";
    g.A = nh ? sv.g[nh - 1] : hf; g.lda = d.d; g.a_kmajor = false; g.B = dpb; g.ldb = d.out; g.b_kmajor = false;
    g.C = gr->w_h; g.ldc = d.out; g.out_f32 = true; g.accumulate = accumulate != 0;
    g.M = d.d; g.N = d.out; g.K = T;
    ORBIT_TRY(gemm(g, w.gws, w.gws_bytes, s));
  }
  // gradient entering the last activation; with hidden layers the GELU
  // derivative of its pre-activation is fused into the product
  void* dcur = (nh == 0 && !d.final_ln) ? dx : w.dh[0];
  {
    Gemm g; g.dtype = dt; g.tag = "head_dx";
    g.A = dpb; g.lda = d.out; g.B = p->w_h; g.ldb = d.out; g.b_kmajor = true;
    g.C = dcur; g.ldc = d.d; g.M = T; g.N = d.d; g.K = d.out;
    if (nh) { g.gelu_in = sv.u[nh - 1]; g.ldgi = d.d; }
    ORBIT_TRY(gemm(g, w.gws, w.gws_bytes, s));
  }
  for (int k = nh - 1; k >= 0; --k) {
    // dcur holds du_k, the gradient of the k-th pre-activation
    const void* hk = k ? sv.g[k - 1] : hf;
    {
      Gemm g; g.dtype = dt; g.tag = "head_hidden_dw";
      g.A = hk; g.lda = d.d; g.a_kmajor = false; g.B = dcur; g.ldb = d.d; g.b_kmajor = false;
      g.C = gr->w_hid + (size_t)k * d.d * d.d; g.ldc = d.d; g.out_f32 = true; g.accumulate = accumulate != 0;
      g.M = d.d; g.N = d.d; g.K = T;
      ORBIT_TRY(gemm(g, w.gws, w.gws_bytes, s));
    }
    ORBIT_TRY(colsum(dt, dcur, d.d, T, d.d, nullptr, 0, nullptr, nullptr, gr->b_hid + (size_t)k * d.d, nullptr,
                     accumulate, w.cws, s));
    void* dnext = (k == 0 && !d.final_ln) ? dx : (dcur == w.dh[0] ? w.dh[1] : w.dh[0]);
    Gemm g; g.dtype = dt; g.tag = "head_hidden_dx";
    g.A = dcur; g.lda = d.d; g.B = static_cast<const char*>(p->w_hid) + (size_t)k * d.d * d.d * e; g.ldb = d.d;
    g.b_kmajor = true; g.C = dnext; g.ldc = d.d; g.M = T; g.N = d.d; g.K = d.d;
    if (k) { g.gelu_in = sv.u[k - 1]; g.ldgi = d.d; }
    ORBIT_TRY(gemm(g, w.gws, w.gws_bytes, s));
    dcur = dnext;
  }
  if (d.final_ln) {
    ColFinal f;
    ORBIT_TRY(layernorm_bwd_cols(dt, dcur, d.d, x, d.d, sv.mu, sv.r, p->lnf_g, nullptr, dx, d.d, T, d.d,
                                 reinterpret_cast<float*>(w.cws), gr->lnf_b, gr->lnf_g, nullptr, f, s));
    ORBIT_TRY(f.run(accumulate, s));
  } else if (!accumulate) {
    if (gr->lnf_g) ORBIT_TRY(fill_f32(gr->lnf_g, d.d, 0.f, s));
    if (gr->lnf_b) ORBIT_TRY(fill_f32(gr->lnf_b, d.d, 0.f, s));
  }
  return ORBIT_OK;
}

// ---------------------------------------------------------------------------
// loss
// ---------------------------------------------------------------------------
size_t orbit_mse_workspace_bytes(int64_t n) { return n > 0 ? mse_workspace_bytes(n) : 0; }

orbit_status orbit_mse_loss(const float* pred, const float* tgt, int64_t n, float scale, float* loss, float* dpred,
                            void* ws, size_t ws_bytes, void* stream) {
  const char* fn = "orbit_mse_loss";
  clear_error();
  REQ(n > 0, ORBIT_E_ARG, "%s: n must be positive", fn);
  PTR(pred, "pred"); PTR(tgt, "tgt"); PTR(loss, "loss"); OPT_PTR(dpred, "dpred"); PTR(ws, "ws");
  REQ(ws_bytes >= mse_workspace_bytes(n), ORBIT_E_ARG, "%s: workspace too small", fn);
  return mse(pred, tgt, n, scale, loss, dpred, ws, S(stream));
}

orbit_status orbit_mfma_probe(int32_t blocks, int32_t iters, uint32_t seed, float x, float* out, void* stream) {
  const char* fn = "orbit_mfma_probe";
  clear_error();
  REQ(blocks >= 1 && blocks <= (1 << 20), ORBIT_E_ARG, "%s: blocks=%d outside [1, 2^20]", fn, blocks);
  REQ(iters >= 1 && iters <= (1 << 20), ORBIT_E_ARG, "%s: iters=%d outside [1, 2^20]", fn, iters);
  PTR(out, "out");
  return mfma_probe(blocks, iters, seed, x, out, S(stream));
}

static orbit_status wmse_check(const char* fn, const orbit_wmse_desc* d) {
  REQ(d != nullptr, ORBIT_E_ARG, "%s: desc is NULL", fn);
  REQ(d->B > 0 && d->H > 0 && d->W > 0 && d->V > 0, ORBIT_E_ARG, "%s: sizes must be positive", fn);
  REQ(d->patch == 4, ORBIT_E_UNSUPPORTED, "%s: patch size %d unsupported (4)", fn, d->patch);
  REQ(d->H % 4 == 0 && d->W % 4 == 0, ORBIT_E_ARG, "%s: H=%d and W=%d must be multiples of the patch", fn, d->H,
      d->W);
  REQ((int64_t)d->B * (d->H / 4) * (d->W / 4) < (1ll << 31) && (int64_t)d->V * 16 < (1ll << 31),
      ORBIT_E_UNSUPPORTED, "%s: too many tokens", fn);
  return ORBIT_OK;
}

size_t orbit_wmse_workspace_bytes(const orbit_wmse_desc* desc) {
  if (wmse_check("orbit_wmse_workspace_bytes", desc) != ORBIT_OK) return 0;
  return wmse_workspace_bytes((int64_t)desc->B * (desc->H / 4) * (desc->W / 4));
}

orbit_status orbit_wmse_loss(const orbit_wmse_desc* desc, const float* pred, const float* tgt, float scale,
                             float* loss, float* dpred, void* ws, size_t ws_bytes, void* stream) {
  const char* fn = "orbit_wmse_loss";
  clear_error();
  ORBIT_TRY(wmse_check(fn, desc));
  PTR(pred, "pred"); PTR(tgt, "tgt"); PTR(loss, "loss"); OPT_PTR(dpred, "dpred"); PTR(ws, "ws");
  const orbit_wmse_desc& d = *desc;
  const int L = (d.H / 4) * (d.W / 4);
  REQ(ws_bytes >= wmse_workspace_bytes((int64_t)d.B * L), ORBIT_E_ARG, "%s: workspace too small", fn);
  return wmse(pred, tgt, d.B, L, d.W / 4, d.H, d.V * 16, scale, loss, dpred, ws, S(stream));
}

// ---------------------------------------------------------------------------
// building blocks
// ---------------------------------------------------------------------------
static Gemm make_gemm(int32_t dtype, int32_t M, int32_t N, int32_t K, int32_t a_kmajor, int32_t b_kmajor) {
  Gemm g;
  g.dtype = (orbit_dtype)dtype;
  g.M = M; g.N = N; g.K = K; g.a_kmajor = a_kmajor != 0; g.b_kmajor = b_kmajor != 0;
  return g;
}

size_t orbit_gemm_workspace_bytes(int32_t dtype, int32_t M, int32_t N, int32_t K, int32_t a_kmajor,
                                  int32_t b_kmajor) {
  if ((dtype != ORBIT_F32 && dtype != ORBIT_BF16) || M <= 0 || N <= 0 || K < 0) return 0;
  return std::max<size_t>(256, gemm_workspace_bytes(make_gemm(dtype, M, N, K, a_kmajor, b_kmajor)));
}

orbit_status orbit_gemm(int32_t dtype, int32_t M, int32_t N, int32_t K, const void* A, int64_t lda,
                        int32_t a_kmajor, const void* B, int64_t ldb, int32_t b_kmajor, void* C, int64_t ldc,
                        int32_t c_f32, float alpha, const void* bias, int32_t accumulate, void* ws, size_t ws_bytes,
                        void* stream) {
  const char* fn = "orbit_gemm";
  clear_error();
  ORBIT_TRY(check_dtype(fn, dtype));
  REQ(M > 0 && N > 0 && K >= 0, ORBIT_E_ARG, "%s: bad sizes M=%d N=%d K=%d", fn, M, N, K);
  REQ(a_kmajor || !b_kmajor, ORBIT_E_UNSUPPORTED, "%s: A M-major with B K-major is not supported", fn);
  PTR(A, "A"); PTR(B, "B"); PTR(C, "C"); OPT_PTR(bias, "bias"); OPT_PTR(ws, "ws");
  const int64_t ca = a_kmajor ? K : M, cb = b_kmajor ? K : N;
  REQ(ca % 8 == 0 || (a_kmajor && !b_kmajor), ORBIT_E_ARG, "%s: contiguous dimension of A must be a multiple of 8", fn);
  REQ(cb % 8 == 0, ORBIT_E_ARG, "%s: contiguous dimension of B must be a multiple of 8", fn);
  REQ(lda >= ca && ldb >= cb && ldc >= N && lda % 8 == 0 && ldb % 8 == 0, ORBIT_E_ARG,
      "%s: leading dimensions too small or not multiples of 8", fn);
  REQ(!accumulate || c_f32, ORBIT_E_ARG, "%s: accumulate needs a float32 C", fn);
  Gemm g = make_gemm(dtype, M, N, K, a_kmajor, b_kmajor);
  g.A = A; g.lda = lda; g.B = B; g.ldb = ldb; g.C = C; g.ldc = ldc; g.out_f32 = c_f32 != 0 || dtype == ORBIT_F32;
  g.alpha = alpha; g.bias = bias; g.accumulate = accumulate != 0;
  return gemm(g, ws, ws ? ws_bytes : 0, S(stream));
}

static orbit_status attn_check(const char* fn, int32_t dtype, int32_t B, int32_t H, int32_t L, int32_t dh) {
  ORBIT_TRY(check_dtype(fn, dtype));
  REQ(B > 0 && H > 0 && L > 0, ORBIT_E_ARG, "%s: sizes must be positive", fn);
  ORBIT_TRY(head_dim_check(fn, dtype, dh));
  return ORBIT_OK;
}

}  // extern "C"

namespace orbit {
// arguments of the attention backward other than its workspace
orbit_status attention_bwd_check(const char* fn, int32_t dtype, int32_t B, int32_t H, int32_t L, int32_t head_dim,
                                 const void* q, int64_t ldq, const void* k, int64_t ldk, const void* v, int64_t ldv,
                                 const void* o, int64_t ldo, const float* lse, const void* dO, int64_t lddo,
                                 const void* dq, const void* dk, const void* dv, int64_t ldg) {
  ORBIT_TRY(attn_check(fn, dtype, B, H, L, head_dim));
  PTR(q, "q"); PTR(k, "k"); PTR(v, "v"); PTR(o, "o"); PTR(lse, "lse"); PTR(dO, "dO");
  PTR(dq, "dq"); PTR(dk, "dk"); PTR(dv, "dv");
  const int64_t A = (int64_t)H * head_dim;
  REQ(ldq >= A && ldk >= A && ldv >= A && ldo >= A && lddo >= A && ldg >= A, ORBIT_E_ARG,
      "%s: leading dimensions must be >= heads*head_dim", fn);
  REQ(ldq % 8 == 0 && ldk % 8 == 0 && ldv % 8 == 0 && ldo % 8 == 0 && lddo % 8 == 0 && ldg % 8 == 0, ORBIT_E_ARG,
      "%s: leading dimensions must be multiples of 8", fn);
  return ORBIT_OK;
}
}  // namespace orbit

extern "C" {

orbit_status orbit_attention_fwd(int32_t dtype, int32_t B, int32_t H, int32_t L, int32_t head_dim, const void* q,
                                 int64_t ldq, const void* k, int64_t ldk, const void* v, int64_t ldv, void* o,
                                 int64_t ldo, float* lse, float* o32, int64_t ldo32, void* stream) {
  const char* fn = "orbit_attention_fwd";
  clear_error();
  ORBIT_TRY(attn_check(fn, dtype, B, H, L, head_dim));
  PTR(q, "q"); PTR(k, "k"); PTR(v, "v"); PTR(o, "o"); PTR(lse, "lse"); OPT_PTR(o32, "o32");
  const int64_t A = (int64_t)H * head_dim;
  REQ(ldq >= A && ldk >= A && ldv >= A && ldo >= A && ldq % 8 == 0 && ldk % 8 == 0 && ldv % 8 == 0 && ldo % 8 == 0,
      ORBIT_E_ARG, "%s: leading dimensions must be >= heads*head_dim and multiples of 8", fn);
  REQ(!o32 || (ldo32 >= A && ldo32 % 8 == 0), ORBIT_E_ARG, "%s: bad ldo32", fn);
  AttnIO io{q, k, v, ldq, ldk, ldv, B, H, L, head_dim};
  return attn_fwd((orbit_dtype)dtype, io, o, ldo, lse, o32, ldo32, nullptr, 0, S(stream));
}

orbit_status orbit_attention_bwd(int32_t dtype, int32_t B, int32_t H, int32_t L, int32_t head_dim, const void* q,
                                 int64_t ldq, const void* k, int64_t ldk, const void* v, int64_t ldv, const void* o,
                                 int64_t ldo, int32_t o_f32, const float* lse, const void* dO, int64_t lddo, void* dq,
                                 void* dk, void* dv, int64_t ldg, void* ws, size_t ws_bytes, void* stream) {
  const char* fn = "orbit_attention_bwd";
  clear_error();
  ORBIT_TRY(attention_bwd_check(fn, dtype, B, H, L, head_dim, q, ldq, k, ldk, v, ldv, o, ldo, lse, dO, lddo, dq, dk,
                                dv, ldg));
  PTR(ws, "ws");
  REQ(ws_bytes >= attn_bwd_workspace_bytes(B, H, L, head_dim), ORBIT_E_ARG, "%s: workspace too small", fn);
  AttnIO io{q, k, v, ldq, ldk, ldv, B, H, L, head_dim};
  return attn_bwd((orbit_dtype)dtype, io, o, ldo, o_f32 ? 1 : 0, lse, dO, lddo, dq, dk, dv, ldg,
                  static_cast<float*>(ws), S(stream));
}

size_t orbit_attention_bwd_workspace_bytes(int32_t B, int32_t H, int32_t L, int32_t head_dim) {
  if (B <= 0 || H <= 0 || L <= 0 || head_dim <= 0) return 0;
  return attn_bwd_workspace_bytes(B, H, L, head_dim);
}

orbit_status orbit_layernorm_fwd(int32_t dtype, int32_t rows, int32_t n, const void* x, const void* g,
                                 const void* b, float eps, void* y, float* mean, float* rstd, void* stream) {
  const char* fn = "orbit_layernorm_fwd";
  clear_error();
  ORBIT_TRY(check_dtype(fn, dtype));
  REQ(rows > 0 && n > 0 && n % 8 == 0 && n <= 16384, ORBIT_E_ARG, "%s: bad sizes rows=%d n=%d", fn, rows, n);
  REQ(eps > 0.f, ORBIT_E_ARG, "%s: eps must be positive", fn);
  PTR(x, "x"); PTR(g, "g"); PTR(b, "b"); PTR(y, "y"); OPT_PTR(mean, "mean"); OPT_PTR(rstd, "rstd");
  return layernorm_fwd((orbit_dtype)dtype, x, n, g, b, y, n, mean, rstd, rows, n, eps, S(stream));
}

}  // extern "C"
