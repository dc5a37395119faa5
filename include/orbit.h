/*
 * orbit.h — C ABI of the MI355X (gfx950) implementation of ORBIT's ViT hot path
 * (arXiv 2404.14712): per-variable patch tokenisation, cross-attention variable
 * aggregation, pre-LN transformer blocks with QK-LayerNorm, prediction head and
 * MSE loss, forward and backward, on one GPU's share of the model.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * Pointers.   Every tensor pointer is a DEVICE pointer owned by the caller and
 *             must be 16-byte aligned. The library never allocates, frees or
 *             keeps a pointer after a call returns. Scratch memory is passed in
 *             as `ws` / `ws_bytes` (size from the matching *_workspace_bytes
 *             query); tensors saved for the backward go to `saved` (size from
 *             *_saved_bytes). Their contents are opaque.
 * Layouts.    Row-major. Activations are [B, L, d] (token t = b*L + l).
 *             Weights are [in, out] and used as y = x W. Tokens of the patch
 *             embedding are [B, L, V, d] (the V x d slab of a patch contiguous).
 * Dtypes.     `dtype` (ORBIT_F32 or ORBIT_BF16) is the type of activations,
 *             tokens, weights, biases and LayerNorm parameters. Images, targets,
 *             predictions and the loss are always float32. Every parameter
 *             gradient is float32. In bf16 mode all products accumulate in
 *             float32; LayerNorm statistics, softmax and GELU run in float32.
 * Sizes.      Feature sizes (d, heads*head_dim, mlp, V*patch^2) must be
 *             multiples of 8; head_dim must be 32, 64 or 128, or in bf16 mode
 *             also 192 or 256 (the paper's 1B/113B and 10B widths); token counts
 *             (B, L, V) are arbitrary positive integers.
 * Streams.    `stream` is a hipStream_t passed as void* (NULL = the null
 *             stream). Every call only enqueues work on it and returns; results
 *             are valid once the stream reaches that point. No call
 *             synchronises the device.
 * Gradients.  accumulate = 0 overwrites the gradient buffers, 1 adds to them.
 * Errors.     Arguments are validated before anything is enqueued; on failure
 *             the call returns ORBIT_E_ARG or ORBIT_E_UNSUPPORTED, touches no
 *             output, and orbit_last_error() (thread-local) describes why. A
 *             failed launch returns ORBIT_E_DEVICE. Nothing aborts, prints or
 *             throws across the ABI.
 * Calls on different streams may run concurrently only if they share no
 * writable buffer (outputs, saved tensors, workspace, gradients).
 */
#ifndef ORBIT_H
#define ORBIT_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define ORBIT_ABI_VERSION 2

typedef enum {
  ORBIT_OK = 0,
  ORBIT_E_ARG = 1,          /* invalid argument (null, misaligned, bad size)   */
  ORBIT_E_UNSUPPORTED = 2,  /* valid but not implemented (e.g. head_dim 96)    */
  ORBIT_E_DEVICE = 3        /* a HIP launch or runtime call failed             */
} orbit_status;

typedef enum { ORBIT_F32 = 0, ORBIT_BF16 = 1 } orbit_dtype;

/* ------------------------------------------------------------------------ */
/* Transformer block (paper Sec. II; Sec. III-A sub-layers softmax(QK^T)V   */
/* and GeLU(xA)B; Sec. III-B QK-LayerNorm; Eq. (2) shard shapes)             */
/* ------------------------------------------------------------------------ */

/* One pre-LN block on x[B, L, d]:
 *   h1 = LN1(x); [q|k|v] = h1 W_qkv + b_qkv   (W_qkv [d, 3A], A = heads*head_dim,
 *        columns q then k then v, head h at columns h*head_dim .. +head_dim);
 *   if qk_norm: q, k <- per-head LayerNorm over head_dim (gain/shift [head_dim]
 *        shared by the heads);
 *   o = softmax(q k^T / sqrt(head_dim)) v per (sample, head), no mask;
 *   x1 = x + o W_proj + b_proj             (W_proj [A, d]);
 *   u  = LN2(x1) W_fc1 + b_fc1             (W_fc1 [d, mlp]);
 *   y  = x1 + GELU(u) W_fc2 + b_fc2        (W_fc2 [mlp, d]; exact erf GELU).
 * When A != d or mlp is a local width this is one GPU's share under Eq. (2):
 * W_qkv / W_fc1 are column shards, W_proj / W_fc2 row shards, and the
 * row-shard partial outputs are added to the residual without any reduction.
 * LayerNorms use the biased variance and eps. */
typedef struct {
  int32_t B, L, d, heads, head_dim, mlp, qk_norm;
  float eps;
  int32_t dtype; /* orbit_dtype */
} orbit_block_desc;

typedef struct {
  const void *ln1_g, *ln1_b;     /* [d]                                  */
  const void *w_qkv, *b_qkv;     /* [d, 3A], [3A]                        */
  const void *qn_g, *qn_b;       /* [head_dim] (ignored if !qk_norm)     */
  const void *kn_g, *kn_b;       /* [head_dim] (ignored if !qk_norm)     */
  const void *w_proj, *b_proj;   /* [A, d], [d]                          */
  const void *ln2_g, *ln2_b;     /* [d]                                  */
  const void *w_fc1, *b_fc1;     /* [d, mlp], [mlp]                      */
  const void *w_fc2, *b_fc2;     /* [mlp, d], [d]                        */
} orbit_block_params;

typedef struct { /* float32, same shapes as orbit_block_params */
  float *ln1_g, *ln1_b, *w_qkv, *b_qkv, *qn_g, *qn_b, *kn_g, *kn_b,
        *w_proj, *b_proj, *ln2_g, *ln2_b, *w_fc1, *b_fc1, *w_fc2, *b_fc2;
} orbit_block_grads;

/* Bytes of `saved` written by orbit_vit_block_fwd and read by _bwd; 0 on a bad descriptor. */
size_t orbit_vit_block_saved_bytes(const orbit_block_desc* desc);
/* Bytes of workspace needed by orbit_vit_block_fwd and _bwd; 0 on a bad descriptor. */
size_t orbit_vit_block_workspace_bytes(const orbit_block_desc* desc);

/* x, y: [B, L, d] (dtype), y must not alias x. saved: NULL for inference
 * (intermediates then live in ws), else orbit_vit_block_saved_bytes bytes. */
orbit_status orbit_vit_block_fwd(const orbit_block_desc* desc, const orbit_block_params* p,
                                 const void* x, void* y, void* saved,
                                 void* ws, size_t ws_bytes, void* stream);

/* Backward of orbit_vit_block_fwd given the same x and params and the `saved`
 * tensors of that call. dy, dx: [B, L, d] (dtype); dx may alias dy, not x.
 * saved == NULL selects activation checkpointing (Sec. III-B; Table I): the
 * call first recomputes the tensors the backward reads from x (the forward
 * without its last product, whose output the backward does not need) into
 * the workspace, then runs the backward; results are bitwise identical to
 * those from a stored `saved`. The caller then keeps only each block's input
 * between the passes (the forward can run with saved == NULL too). */
orbit_status orbit_vit_block_bwd(const orbit_block_desc* desc, const orbit_block_params* p,
                                 const void* x, const void* saved, const void* dy, void* dx,
                                 const orbit_block_grads* g, int accumulate,
                                 void* ws, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------ */
/* Per-variable patch tokenisation (Sec. II: every variable is tokenised     */
/* independently)                                                            */
/* ------------------------------------------------------------------------ */

/* img[B, V, H, W] float32 -> tok[B, L, V, d] (dtype), L = (H/patch)*(W/patch):
 *   tok[b, l, v, :] = P[b, v, l, :] W_pe[v] + b_pe[v] + ve[v]
 * with patch l = ph*(W/patch) + pw and pixel index i*patch + j inside it.
 * w_pe [V, patch*patch, d], b_pe [V, d], ve [V, d] (ve may be NULL).
 * H and W must be multiples of patch; patch must be 4. */
typedef struct {
  int32_t B, V, H, W, patch, d;
  int32_t dtype;
} orbit_embed_desc;

orbit_status orbit_patch_embed(const orbit_embed_desc* desc, const float* img,
                               const void* w_pe, const void* b_pe, const void* ve,
                               void* tok, void* stream);

size_t orbit_patch_embed_workspace_bytes(const orbit_embed_desc* desc);
/* Parameter gradients from dtok[B, L, V, d] (dtype). dve may be NULL. */
orbit_status orbit_patch_embed_bwd(const orbit_embed_desc* desc, const float* img,
                                   const void* dtok, float* dw_pe, float* db_pe, float* dve,
                                   int accumulate, void* ws, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------ */
/* Cross-attention variable aggregation (Sec. II)                            */
/* ------------------------------------------------------------------------ */

/* tok[B, L, V, d] -> z[B, L, d]: one learned query q0 attends over the V
 * tokens of each patch with multi-head attention semantics:
 *   q = q0 W_q + b_q;  K = X W_k + b_k;  Vv = X W_v + b_v   (X = tok[b, l]);
 *   a_h = softmax_v(q_h . K_{v,h} / sqrt(head_dim));  zh_h = sum_v a_{h,v} Vv_{v,h};
 *   z = concat_h(zh) W_o + b_o + pos[l].
 * W_q, W_k, W_v [d, A], biases [A], W_o [A, d], b_o [d], pos [L, d] (may be
 * NULL), A = heads*head_dim (a column shard of the projections when A != d,
 * with the W_o row-shard output left unreduced). The library evaluates the
 * exact algebraic refolding (query through W_k, weights applied before W_v),
 * which has the same value. heads must divide 64 and be a multiple of 8
 * (bf16) or 4 (float32), and head_dim at most 8192; otherwise
 * ORBIT_E_UNSUPPORTED. d and head_dim must be multiples of 8 (ORBIT_E_ARG). */
typedef struct {
  int32_t B, L, V, d, heads, head_dim;
  int32_t dtype;
} orbit_agg_desc;

typedef struct {
  const void *q0, *w_q, *b_q, *w_k, *b_k, *w_v, *b_v, *w_o, *b_o, *pos;
} orbit_agg_params;

typedef struct { /* float32 */
  float *q0, *w_q, *b_q, *w_k, *b_k, *w_v, *b_v, *w_o, *b_o, *pos;
} orbit_agg_grads;

size_t orbit_var_aggregate_saved_bytes(const orbit_agg_desc* desc);
size_t orbit_var_aggregate_workspace_bytes(const orbit_agg_desc* desc);

orbit_status orbit_var_aggregate(const orbit_agg_desc* desc, const void* tok,
                                 const orbit_agg_params* p, void* z, void* saved,
                                 void* ws, size_t ws_bytes, void* stream);

/* dz [B, L, d] -> dtok [B, L, V, d] and parameter gradients (pos grad may be
 * NULL when pos was NULL). `saved` is the forward's. */
orbit_status orbit_var_aggregate_bwd(const orbit_agg_desc* desc, const void* tok,
                                     const orbit_agg_params* p, const void* saved,
                                     const void* dz, void* dtok, const orbit_agg_grads* g,
                                     int accumulate, void* ws, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------ */
/* Prediction head (Sec. II: projection from feature space to image space)   */
/* ------------------------------------------------------------------------ */

/* x[B, L, d] -> pred[B, L, out] float32: h = LN_f(x) (skipped when
 * final_ln == 0); then `hidden` layers h <- GELU(h W_hid[k] + b_hid[k]) of
 * width d (the multi-layer decoder of the ClimaX architecture the paper
 * builds on; 0 = none); then pred = h W_h + b_h.
 * W_hid [hidden, d, d], b_hid [hidden, d] (NULL when hidden == 0), W_h
 * [d, out], b_h [out]; a token's output row holds its V patches, pixel index
 * v*patch^2 + i*patch + j. hidden is at most 8. */
typedef struct {
  int32_t B, L, d, out, final_ln;
  float eps;
  int32_t dtype;
  int32_t hidden;
} orbit_head_desc;

typedef struct { const void *lnf_g, *lnf_b, *w_h, *b_h, *w_hid, *b_hid; } orbit_head_params;
typedef struct { float *lnf_g, *lnf_b, *w_h, *b_h, *w_hid, *b_hid; } orbit_head_grads;

size_t orbit_head_saved_bytes(const orbit_head_desc* desc);
size_t orbit_head_workspace_bytes(const orbit_head_desc* desc);

orbit_status orbit_head_fwd(const orbit_head_desc* desc, const void* x,
                            const orbit_head_params* p, float* pred, void* saved,
                            void* ws, size_t ws_bytes, void* stream);

/* dpred [B, L, out] float32 -> dx [B, L, d] (dtype) and parameter gradients. */
orbit_status orbit_head_bwd(const orbit_head_desc* desc, const void* x,
                            const orbit_head_params* p, const void* saved,
                            const float* dpred, void* dx, const orbit_head_grads* g,
                            int accumulate, void* ws, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------ */
/* Training loss: mean squared error                                         */
/* ------------------------------------------------------------------------ */

/* loss[0] = sum((pred - tgt)^2) / n;  dpred = 2 (pred - tgt) / n * scale.
 * pred, tgt, dpred: n float32 values (dpred may be NULL); loss: 1 float32 on
 * the device. The sum is reduced in a fixed order (bitwise reproducible). */
size_t orbit_mse_workspace_bytes(int64_t n);
orbit_status orbit_mse_loss(const float* pred, const float* tgt, int64_t n, float scale,
                            float* loss, float* dpred, void* ws, size_t ws_bytes, void* stream);

/* Latitude-weighted mean squared error (Sec. IV: the training loss) of
 * predictions and targets in token layout pred, tgt [B, L, V*patch^2] float32
 * on an H x W grid (L = (H/patch)(W/patch), patch 4):
 *   loss[0] = mean over (b, v, y, x) of w_y (pred - tgt)^2,
 *   dpred = 2 w_y (pred - tgt) / n * scale   (n = B*L*V*patch^2),
 * w_y = cos(lat_y) / mean_y cos(lat_y) with rows at equally spaced latitudes,
 * cell centres lat_y = -90 + (y + 1/2) 180 / H degrees. dpred may be NULL.
 * Reduced in a fixed order (bitwise reproducible). */
typedef struct {
  int32_t B, H, W, V, patch;
} orbit_wmse_desc;
size_t orbit_wmse_workspace_bytes(const orbit_wmse_desc* desc);
orbit_status orbit_wmse_loss(const orbit_wmse_desc* desc, const float* pred, const float* tgt, float scale,
                             float* loss, float* dpred, void* ws, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------ */
/* Building blocks of the calls above, exposed for kernel-level testing      */
/* ------------------------------------------------------------------------ */

/* C[M, N] = alpha * A B (+ bias[n]) (+ C if accumulate), dtype operands,
 * float32 accumulation; the dense product behind every linear layer
 * (Sec. III-A: the sub-layers are chains of two such products).
 * A[m, k] is at A[m*lda + k] if a_kmajor else A[k*lda + m]; B[k, n] is at
 * B[n*ldb + k] if b_kmajor else B[k*ldb + n]; the pair (A M-major, B K-major)
 * is not supported. C is float32 if c_f32 else dtype (accumulate needs
 * float32). bias is dtype [N] or NULL. K must be a multiple of 8 when both
 * operands are K-major; contiguous dimensions must be multiples of 8. */
size_t orbit_gemm_workspace_bytes(int32_t dtype, int32_t M, int32_t N, int32_t K, int32_t a_kmajor,
                                  int32_t b_kmajor);
orbit_status orbit_gemm(int32_t dtype, int32_t M, int32_t N, int32_t K, const void* A, int64_t lda,
                        int32_t a_kmajor, const void* B, int64_t ldb, int32_t b_kmajor, void* C,
                        int64_t ldc, int32_t c_f32, float alpha, const void* bias, int32_t accumulate,
                        void* ws, size_t ws_bytes, void* stream);

/* O = softmax(q k^T / sqrt(head_dim)) v for every (sample b, head h), no mask
 * (Sec. III-A). Row t = b*L + l of q holds head h at q[t*ldq + h*head_dim];
 * likewise k, v, o. lse [B, H, L] float32 receives the natural-log
 * normaliser of each softmax row (needed by the backward). o32 (may be NULL,
 * leading dimension ldo32) receives a float32 copy of O. Leading dimensions
 * are at least H*head_dim and multiples of 8. In bf16 mode the kernels
 * address one (sample, head) slice with 32-bit byte offsets: (L + 256) times
 * the largest leading dimension times 4 must stay below 2^31 (and B*H*L
 * below 2^31), else ORBIT_E_UNSUPPORTED; the backward has the same limits. */
orbit_status orbit_attention_fwd(int32_t dtype, int32_t B, int32_t H, int32_t L, int32_t head_dim,
                                 const void* q, int64_t ldq, const void* k, int64_t ldk,
                                 const void* v, int64_t ldv, void* o, int64_t ldo, float* lse,
                                 float* o32, int64_t ldo32, void* stream);
/* Gradients dq, dk, dv (same row layout, leading dimension ldg) from dO and
 * the forward's O and lse. O is float32 when o_f32 (the forward's o32 copy:
 * its row sums against dO stay consistent with the recomputed probabilities
 * in bf16 mode), else dtype. Workspace: orbit_attention_bwd_workspace_bytes. */
size_t orbit_attention_bwd_workspace_bytes(int32_t B, int32_t H, int32_t L, int32_t head_dim);
orbit_status orbit_attention_bwd(int32_t dtype, int32_t B, int32_t H, int32_t L, int32_t head_dim,
                                 const void* q, int64_t ldq, const void* k, int64_t ldk,
                                 const void* v, int64_t ldv, const void* o, int64_t ldo,
                                 int32_t o_f32, const float* lse, const void* dO, int64_t lddo,
                                 void* dq, void* dk, void* dv, int64_t ldg, void* ws, size_t ws_bytes,
                                 void* stream);

/* orbit_attention_bwd without a workspace argument, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation). The same kernels and results (bitwise)
 * as orbit_attention_bwd; their scratch lives in a device array the library
 * holds per GPU (ORBIT_ATTN_BWD_NOALLOC_MAX_SCRATCH bytes on each GPU the
 * library runs on, until the process ends). The call allocates nothing.
 * Sizes whose orbit_attention_bwd_workspace_bytes exceeds that maximum return
 * ORBIT_E_UNSUPPORTED. Every call on one GPU shares that GPU's array, so calls
 * that overlap on one GPU (concurrent streams or host threads) race: order
 * them on one stream. The array needs no clearing: every call writes the
 * scratch it reads. */
#define ORBIT_ATTN_BWD_NOALLOC_MAX_SCRATCH ((size_t)160 << 20)
orbit_status orbit_attention_bwd_noalloc(int32_t dtype, int32_t B, int32_t H, int32_t L, int32_t head_dim,
                                         const void* q, int64_t ldq, const void* k, int64_t ldk,
                                         const void* v, int64_t ldv, const void* o, int64_t ldo,
                                         int32_t o_f32, const float* lse, const void* dO, int64_t lddo,
                                         void* dq, void* dk, void* dv, int64_t ldg, void* stream);

/* LayerNorm over rows of length n (biased variance): y = g (x - mean) rstd + b;
 * mean, rstd [rows] float32 (may be NULL). n <= 16384, multiple of 8. */
orbit_status orbit_layernorm_fwd(int32_t dtype, int32_t rows, int32_t n, const void* x, const void* g,
                                 const void* b, float eps, void* y, float* mean, float* rstd,
                                 void* stream);

/* ------------------------------------------------------------------------ */
/* Diagnostics and measurement support                                       */
/* ------------------------------------------------------------------------ */

const char* orbit_status_string(orbit_status s);
/* Detail of the last failure on the calling thread ("" if none). */
const char* orbit_last_error(void);
int orbit_abi_version(void);

/* Kernel timing. While enabled, every kernel the library enqueues is
 * bracketed by a pair of HIP events on the caller's stream, and its name,
 * algorithmic flop count and algorithmic HBM byte count are recorded (up to
 * an internal limit of launches; later launches are not recorded).
 * orbit_timing_enable(1) clears previous records. orbit_timing_summary()
 * waits for the recorded events and, for launches of kernels whose name
 * starts with `prefix` (NULL or "" = all), returns the number of launches,
 * their summed duration in milliseconds, summed flops and summed bytes.
 * Not for concurrent use from several threads. */
orbit_status orbit_timing_enable(int on);
/* Record only kernels whose name starts with `prefix` (NULL or "" = all).
 * Applies to launches enqueued after the call. */
orbit_status orbit_timing_filter(const char* prefix);
orbit_status orbit_timing_summary(const char* prefix, int64_t* launches, double* total_ms,
                                  double* flops, double* bytes);
/* Name of the i-th distinct kernel recorded (NULL past the end). */
const char* orbit_timing_kernel_name(int i);

/* Matrix-core throughput probe, for measuring the sustained bf16 peak and
 * clock of the GPU the library runs on (not a step of the model). Launches
 * `blocks` blocks of 4 waves; each wave keeps 8 independent bf16 32x32x16
 * matrix products in flight for `iters` rounds, which is
 * blocks * 4 * iters * 8 * 32768 flops; the caller times the launch on
 * `stream`. Both operands of every product are the lane's 8-element
 * fragment: with seed 0 every element is bf16(x); otherwise element i of
 * lane l is bf16(x * p) with p = ((h & 255) - 128) / 64 and h the 32-bit
 * hash h0 = (seed ^ (8 l + i)) * 0x9E3779B1, h1 = h0 ^ (h0 >> 15),
 * h2 = h1 * 0x85EBCA77, h = h2 ^ (h2 >> 13) (varied operand bits, as in real
 * data; the clock is lower then). out (device, float32, blocks * 4 elements,
 * caller owned) receives per wave 8 iters (s0 + s32), s_l the sum of the
 * squares of lane l's fragment elements (accumulated in float32). blocks in
 * [1, 2^20], iters in [1, 2^20]; otherwise ORBIT_E_ARG. */
orbit_status orbit_mfma_probe(int32_t blocks, int32_t iters, uint32_t seed, float x, float* out, void* stream);

#ifdef __cplusplus
}
#endif
#endif /* ORBIT_H */
