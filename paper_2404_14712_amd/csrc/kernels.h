// Host launchers of the non-GEMM kernels. Each enqueues on `s` and returns a
// status; shapes are validated by the callers in abi.cpp.
#pragma once
#include <vector>

#include "common.h"

namespace orbit {

// ---- LayerNorm over rows of length n (pre-LN and final LN) ----------------
// y = g * (x - mean) * rstd + b; mean/rstd [rows] float32 (may be null).
orbit_status layernorm_fwd(orbit_dtype dt, const void* x, int64_t ldx, const void* g, const void* b,
                           void* y, int64_t ldy, float* mean, float* rstd, int rows, int n,
                           float eps, hipStream_t s);

// ---- deterministic column reductions over rows ----------------------------
// Phase 1 (colsum_partials, one launch for up to kColMaxJobs jobs over the
// same number of rows): per-chunk partial sums of src[r, c] and, for LN jobs
// (x != null), of src[r, c] * xhat[r, c] with xhat = (x - mean[r]) * rstd[r],
// into the job's `part` buffer (colsum_part_bytes). A job may cover `batch`
// independent row blocks (src + b * sbatch, outputs at out + b * sout).
// Phase 2 (ColFinal): fixed-order sums of the partials into float32 outputs
// (overwrite or accumulate), any number of outputs per launch.
constexpr int kColMaxJobs = 8;
constexpr int kColMaxFinal = 16;
struct ColJob {
  const void* src = nullptr; int64_t ld = 0; int64_t sbatch = 0;
  const void* x = nullptr; int64_t ldx = 0; int64_t sxbatch = 0;
  const float* mean = nullptr; const float* rstd = nullptr;
  int n = 0, batch = 1;
  float* part = nullptr;
  float* out_sum = nullptr; float* out_xsum = nullptr; int64_t sout = 0;
};
int colsum_chunks(int rows);
size_t colsum_part_bytes(int rows, int n, bool ln, int batch = 1);
orbit_status colsum_partials(orbit_dtype dt, ColJob* jobs, int njobs, int rows, hipStream_t s);
class ColFinal {
 public:
  void add(const float* part, int64_t ldp, int chunks, int n, float* out);
  void add_job(const ColJob& J, int rows);
  orbit_status run(int accumulate, hipStream_t s);
 private:
  struct Item { const float* part; int64_t ldp; float* out; int chunks, n; };
  std::vector<Item> items;
};
// LayerNorm backward, dx = rstd * (dy*g - mean(dy*g) - xhat * mean(dy*g*xhat))
// [+ dres] (n a multiple of 8 up to 16384; dx may alias dres), that also forms,
// per chunk of 8 or 16 rows, the column sums of dy (-> out_b), dy * xhat
// (-> out_g) and, when out_o is given, of the output dx (-> out_o); their
// fixed-order final sums are queued on `fin`. part: ln_bwd_cols_part_bytes.
size_t ln_bwd_cols_part_bytes(int rows, int n, bool osum);
orbit_status layernorm_bwd_cols(orbit_dtype dt, const void* dy, int64_t lddy, const void* x, int64_t ldx,
                                const float* mean, const float* rstd, const void* g, const void* dres, void* dx,
                                int64_t lddx, int rows, int n, float* part, float* out_b, float* out_g,
                                float* out_o, ColFinal& fin, hipStream_t s);
// both phases for one (optionally LN) job; workspace: colsum_workspace_bytes
size_t colsum_workspace_bytes(int rows, int n);
orbit_status colsum(orbit_dtype dt, const void* dy, int64_t lddy, int rows, int n,
                    const void* x, int64_t ldx, const float* mean, const float* rstd,
                    float* out_sum, float* out_xsum, int accumulate, void* ws, hipStream_t s);
// float32 input variant (dpred of the head)
orbit_status colsum_f32(const float* dy, int64_t lddy, int rows, int n, float* out_sum,
                        int accumulate, void* ws, hipStream_t s);

// ---- QK-LayerNorm: per-head LN over head_dim on q and k --------------------
// src row t: q at src[t*lds + h*dh], k at src[t*lds + A + h*dh]; dst the same
// with ldd. stats: mean/rstd [T, 2H] (q heads then k heads).
orbit_status qk_norm_fwd(orbit_dtype dt, const void* src, int64_t lds, void* dst, int64_t ldd,
                         const void* qg, const void* qb, const void* kg, const void* kb,
                         float* mean, float* rstd, int T, int H, int dh, float eps, hipStream_t s);
// in place on dq/dk (rows of `d`, ld ldd): dxhat -> dx; gain/shift grads
// (their final sums are queued on `fin` when given, else run here).
size_t qk_norm_bwd_workspace_bytes(int dh);
orbit_status qk_norm_bwd(orbit_dtype dt, void* d, int64_t ldd, const void* src, int64_t lds,
                         const float* mean, const float* rstd, const void* qg, const void* kg,
                         float* dqg, float* dqb, float* dkg, float* dkb, int accumulate,
                         int T, int H, int dh, void* ws, ColFinal* fin, hipStream_t s);

// ---- attention: O = softmax(q k^T / sqrt(dh)) v per (sample, head) --------
struct AttnIO {
  const void *q, *k, *v;
  int64_t ldq, ldk, ldv;
  int B, H, L, dh;
};
// o32 (optional): float32 copy of O, used by the backward for rowsum(dO * O).
// scratch (optional; attn_bwd_workspace_bytes always suffices): with it, bf16
// grids of few blocks split the keys over two blocks and merge their partials
orbit_status attn_fwd(orbit_dtype dt, const AttnIO& io, void* o, int64_t ldo, float* lse, float* o32, int64_t ldo32,
                      void* scratch, size_t scratch_bytes, hipStream_t s);
// workspace of attn_bwd: D[b,h,l] = rowsum(dO * O), sums of q and k over the
// sequence, the column-reduction scratch and the partials of a split launch
size_t attn_bwd_workspace_bytes(int B, int H, int L, int dh);
// validation of the attention backward's arguments other than its workspace
// (shared by the entry points that take a workspace and the one that does not)
orbit_status attention_bwd_check(const char* fn, int32_t dtype, int32_t B, int32_t H, int32_t L, int32_t head_dim,
                                 const void* q, int64_t ldq, const void* k, int64_t ldk, const void* v, int64_t ldv,
                                 const void* o, int64_t ldo, const float* lse, const void* dO, int64_t lddo,
                                 const void* dq, const void* dk, const void* dv, int64_t ldg);
// O is float32 when o_f32, else dtype
orbit_status attn_bwd(orbit_dtype dt, const AttnIO& io, const void* o, int64_t ldo, int o_f32, const float* lse,
                      const void* dO, int64_t lddo, void* dq, void* dk, void* dv, int64_t ldg,
                      float* ws, hipStream_t s);

// ---- patch embedding --------------------------------------------------------
orbit_status patch_embed_fwd(orbit_dtype dt, const float* img, const void* w, const void* b,
                             const void* ve, void* tok, int B, int V, int Hg, int Wg, int p, int d,
                             hipStream_t s);
size_t patch_embed_bwd_workspace_bytes(int B, int V, int Hg, int Wg, int p, int d);
orbit_status patch_embed_bwd(orbit_dtype dt, const float* img, const void* dtok, float* dw, float* db,
                             float* dve, int accumulate, int B, int V, int Hg, int Wg, int p, int d,
                             void* ws, hipStream_t s);

// ---- loss ---------------------------------------------------------------------
size_t mse_workspace_bytes(int64_t n);
orbit_status mse(const float* pred, const float* tgt, int64_t n, float scale, float* loss,
                 float* dpred, void* ws, hipStream_t s);
// latitude-weighted MSE of token-layout predictions [B*L, out] on an H-row
// grid of 4x4 patches, Wp patches per row; workspace: one float per token
size_t wmse_workspace_bytes(int64_t tokens);
orbit_status wmse(const float* pred, const float* tgt, int B, int L, int Wp, int H, int out, float scale,
                  float* loss, float* dpred, void* ws, hipStream_t s);

// ---- measurement aid -------------------------------------------------------------
// blocks of 4 waves, each keeping 8 independent bf16 32x32x16 matrix products
// in flight for `iters` rounds; out[blocks * 4] receives one value per wave
double mfma_probe_flops(int blocks, int iters);
orbit_status mfma_probe(int blocks, int iters, unsigned seed, float x, float* out, hipStream_t s);

// ---- small helpers ------------------------------------------------------------
// dst[i] = (dtype) src[i] (float32 -> dtype); used for dpred before the head GEMMs
orbit_status cast_from_f32(orbit_dtype dt, const float* src, void* dst, int64_t n, hipStream_t s);
// out[i] = accumulate ? out[i] + v : v, for a float32 vector v given on device
orbit_status axpy_f32(const float* src, float* dst, int64_t n, int accumulate, hipStream_t s);
orbit_status fill_f32(float* dst, int64_t n, float v, hipStream_t s);

}  // namespace orbit
