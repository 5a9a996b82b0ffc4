/*
 * layerdrop.h -- C ABI of the MI355X (gfx950) layer-dropout training hot path.
 *
 * What is computed (paper: "Don't Drop Dropout: Optimizing Layer Sparsity for
 * Efficient LLM Training and Inference", Preliminary section):
 *   for layer l at training step t, per sequence b of the batch,
 *     Z       = X + r * M[b] * f_attn(X)
 *     X^{l+1} = Z + r * M[b] * f_ffn(Z)
 *   with the mask M ~ Bernoulli(1 - p^{l,t}) drawn once per sequence and
 *   shared by both sub-blocks (layer granularity, per-sequence tensor
 *   granularity; Dropout Granularity section), r = res_scale / (1 - p) when
 *   rescaling (the paper's r_train = 1/rho; Hyperparameters section, "Dropout
 *   Scale"), and f executed only on the kept sequences (the efficient form
 *   described right after the per-sequence case form), so a dropped sequence
 *   costs no FLOPs and its rows are never touched.
 *   f_attn(X) = MHA_causal(RMSNorm(X; g_attn) W_qkv^T) W_o^T
 *   f_ffn(Z)  = (silu(U) * V) W_down^T,  [U V] = RMSNorm(Z; g_mlp) W_gate_up^T
 *
 * Conventions shared by every entry point
 *   - Every function returns an ld_status (int).  On any error nothing has
 *     been enqueued; ld_last_error() (thread-local) says why.
 *   - "device" pointers are HIP device memory owned by the caller; "host"
 *     pointers are ordinary host memory read before the call returns.
 *     The library allocates no device memory on any call below.
 *   - stream is a hipStream_t passed as void*; NULL means the null stream.
 *     Calls only enqueue work; results are valid once the stream has reached
 *     them.  Exception: while profiling is on (ld_prof_start), mask counts are
 *     read back to the host after each mask launch (one stream sync).
 *   - Tensors are row-major.  Activations are [B, S, d] (sequence-major,
 *     token rows of d contiguous elements).  Weights are [out, in] and applied
 *     as x W^T.  w_qkv rows are [q | k | v], head h owning rows
 *     h*dh .. h*dh+dh-1 of each part; w_gate_up rows [0, d_ff) are the gate,
 *     [d_ff, 2 d_ff) the up projection.
 *   - Element type of activations and weights is cfg->dtype (LD_F32 or
 *     LD_BF16); weight gradients are always float32.
 *   - Repeated calls with equal inputs give bitwise equal outputs (no float
 *     atomics; all reductions run in a fixed order).
 *   - Calls that share a workspace, ctx or output buffer and overlap on
 *     different streams race; the library adds no locking.
 */
#ifndef LAYERDROP_H
#define LAYERDROP_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  LD_OK = 0,
  LD_E_INVALID = 1,     /* bad argument value (NULL pointer, p outside [0,1], NaN) */
  LD_E_SHAPE = 2,       /* inconsistent or unsupported shape                        */
  LD_E_UNSUPPORTED = 3, /* valid request the library does not implement             */
  LD_E_WORKSPACE = 4,   /* workspace smaller than the matching *_bytes query       */
  LD_E_HIP = 5          /* a HIP runtime call failed                                */
} ld_status;

typedef enum { LD_F32 = 0, LD_BF16 = 1 } ld_dtype;

/* Shape and options of one decoder layer.
 *   batch B, seq S, d_model d, n_heads H (d % H == 0), d_ff f.
 *   LD_BF16 requires d_head = d/H in {64, 128}, d % 8 == 0, f % 8 == 0,
 *   S % 64 == 0.  LD_F32 requires d_head in {16, 32, 64}, d % 4 == 0, f % 4 == 0.
 *   d <= 4096 (bf16) or d <= 2048 (fp32).
 *   rms_eps: RMSNorm epsilon (the paper fixes none; 1e-5 is the default).
 *   rescale: 1 -> r = res_scale / (1 - p); 0 -> r = res_scale.
 *   res_scale: constant residual-branch multiplier (the depth multiplier of
 *   the paper's parameterisation table); 1 for plain layer dropout.
 *   block_kind: LD_BLOCK_SWIGLU (0): pre-norm RMSNorm, causal multi-head
 *   attention, SwiGLU feed-forward.  LD_BLOCK_ALIBI_RELU2 (1): the block of
 *   the paper's experiments (Experimental Setup: ALiBi position bias,
 *   squared-ReLU activation): pre-norm RMSNorm, causal attention whose
 *   scaled scores get the ALiBi bias -m_h (i - j) (query i, key j <= i, head
 *   slope m_h of ld_alibi_slope), and the feed-forward relu(h W_up^T)^2 W_down^T.
 *   granularity: which masks are drawn (Dropout Granularity section), two bits:
 *   LD_GRAN_SUBLAYER: model granularity "sub-layer": the attention and FFN
 *     sub-blocks get independent masks M_attn, M_ffn (both Bernoulli(1 - p)
 *     with the layer's p, one r for both):
 *       Z = X + r M_attn f_attn(X),  X^{l+1} = Z + r M_ffn f_ffn(Z);
 *     without it one mask serves both (layer dropout, the paper's choice).
 *   LD_GRAN_PER_BATCH: tensor granularity "per batch": one draw per
 *     (layer, step) shared by every sequence, so a layer (or sub-block) is
 *     kept or skipped for the whole batch; a skipped one reads no weights
 *     and its weight gradients are zero-filled.  Without it the draws are per
 *     sequence (the paper's choice).
 *   Masks per layer: n_masks = 2 under LD_GRAN_SUBLAYER (attention, then
 *   FFN), else 1. */
typedef enum { LD_BLOCK_SWIGLU = 0, LD_BLOCK_ALIBI_RELU2 = 1 } ld_block_kind;
typedef enum {
  LD_GRAN_LAYER_SEQ = 0,
  LD_GRAN_SUBLAYER = 1,
  LD_GRAN_PER_BATCH = 2,
  LD_GRAN_SUBLAYER_SEQ = 1,
  LD_GRAN_LAYER_BATCH = 2,
  LD_GRAN_SUBLAYER_BATCH = 3
} ld_granularity;

typedef struct {
  int32_t batch, seq, d_model, n_heads, d_ff;
  int32_t dtype;
  float rms_eps;
  int32_t rescale;
  float res_scale;
  int32_t block_kind;
  int32_t granularity;
} ld_config;

/* Device pointers to one layer's parameters (element type cfg->dtype):
 * g_attn [d], w_qkv [3d, d], w_o [d, d], g_mlp [d], w_down [d, f], and
 * w_gate_up [2f, d] (gate rows then up rows) for LD_BLOCK_SWIGLU or [f, d]
 * (W_up) for LD_BLOCK_ALIBI_RELU2.  Read only. */
typedef struct {
  const void *g_attn, *w_qkv, *w_o, *g_mlp, *w_gate_up, *w_down;
} ld_weights;

/* Device pointers to one layer's float32 gradients, same shapes as
 * ld_weights.  Overwritten (not accumulated) with sums over kept rows. */
typedef struct {
  float *g_attn, *w_qkv, *w_o, *g_mlp, *w_gate_up, *w_down;
} ld_grads;

/* ---------------------------------------------------------------- errors */

/* Static string naming a status code. */
const char* ld_status_string(int status);
/* Detail of the last error on the calling thread ("" if none). */
const char* ld_last_error(void);

/* -------------------------------------------------------------- schedule */

/* p^{l,t} = depth(l) * time(t), computed in double and rounded to float
 * (Dropout Configurations section).
 *   dist:  0 uniform p_max; 1 ILD l/(L-1) p_max (0 when L = 1);
 *          2 ALD p_max for odd l, 0 for even l.
 *   sched: 0 constant; 1 ITS t/(T-1); 2 DTS 1 - t/(T-1); t is clamped to
 *          [0, T-1] and t/(T-1) is 0 when T = 1.
 * p_out: host float.  Errors: LD_E_INVALID for unknown dist/sched, p_max
 * outside [0,1] or NaN, layer outside [0, n_layers), n_layers < 1, T < 1. */
int ld_schedule_p(int32_t dist, int32_t sched, float p_max, int32_t layer, int32_t n_layers,
                  int64_t t, int64_t n_steps, float* p_out);

/* ----------------------------------------------------- masks / compaction */

/* Bernoulli(1 - p) keep masks and ascending kept lists for layers
 * first_layer .. first_layer + n_layers - 1 at `step` (per-sequence mask of
 * the layer-dropout training equation; the kept list is the set of sequences
 * f is executed on).  The draw for (sample b, layer l, step t) is word 0 of
 * Philox4x64-10 (Salmon et al., SC'11) with counter (b, l, t, 0) and key
 * (seed, 0); sample b drops iff p >= 1 or (p > 0 and word < floor(p 2^64)).
 *   p:     host float[n_layers], each in [0, 1].
 *   keep:  device uint8[n_layers][batch], 1 = kept.
 *   idx:   device int32[n_layers][batch], kept samples ascending, then -1.
 *   count: device int32[n_layers], number of kept samples.
 * n_layers in [1, 128], batch >= 1.  One kernel launch. */
int ld_masks(int32_t n_layers, int32_t batch, const float* p, int32_t first_layer, uint64_t seed,
             uint64_t step, uint8_t* keep, int32_t* idx, int32_t* count, void* stream);

/* ld_masks for any ld_granularity (Dropout Granularity section).  Per
 * sequence, mask m of layer l uses word m of the Philox block with counter
 * (b, l, t, 0); per batch, word m of the block (0, l, t, 1) decides every
 * sample; key (seed, 0) and the threshold rule as in ld_masks.  Mask 0 is the
 * attention (or whole-layer) mask, mask 1 the FFN mask of sub-layer dropout,
 * so the attention mask of LD_GRAN_SUBLAYER_SEQ is the ld_masks mask.
 *   keep, idx: device [n_layers][n_masks][batch]; count: device
 *   [n_layers][n_masks].  Errors as ld_masks, plus LD_E_INVALID for an
 *   unknown granularity. */
int ld_masks_granular(int32_t granularity, int32_t n_layers, int32_t batch, const float* p,
                      int32_t first_layer, uint64_t seed, uint64_t step, uint8_t* keep, int32_t* idx,
                      int32_t* count, void* stream);

/* Gather the rows of the kept sequences into a contiguous block:
 * xk[j*S + s, :] = x[idx[j]*S + s, :] for j < *count (bit copy).  This is
 * the first half of the efficient form of the layer-dropout training
 * equation (Preliminary section, right after the per-sequence case form):
 * f is executed on the kept sequences only, stacked contiguously.
 *   idx, count: device, as produced by ld_masks for one layer.
 *   x: device [B, S, d]; xk: device [B*S, d] (rows past count*S untouched). */
int ld_gather_rows(const ld_config* cfg, const int32_t* idx, const int32_t* count, const void* x,
                   void* xk, void* stream);

/* Residual scatter-add of kept rows, in place:
 * x[idx[j]*S + s, c] = round(fmaf(r, yk[j*S + s, c], x[idx[j]*S + s, c]))
 * for j < *count, with one round-to-nearest-even to cfg->dtype.  Rows of
 * dropped sequences are not read or written.  This is the second half of
 * the efficient form (Preliminary section): H^{l+1} = H^l + r M f(H^l)
 * with the branch output of the kept sequences added back at their rows and
 * the dropped rows left as they are (M = 0); r is r_train (Hyperparameters
 * section, "Dropout Scale").
 *   yk: device [B*S, d] compacted branch output; x: device [B, S, d]. */
int ld_scatter_add_rows(const ld_config* cfg, const int32_t* idx, const int32_t* count, float r,
                        const void* yk, void* x, void* stream);

/* ------------------------------------------------------ layer and stack */

/* Bytes of the per-layer context ld_layer_fwd saves for ld_layer_bwd
 * (kept-row activations sized for the whole batch, plus the mask). */
size_t ld_layer_ctx_bytes(const ld_config* cfg);
/* Bytes of scratch workspace ld_layer_fwd / ld_layer_bwd need. */
size_t ld_layer_ws_bytes(const ld_config* cfg);
/* Bytes of workspace ld_stack_step needs for n_layers layers
 * (n_layers contexts + masks + backward scratch). */
size_t ld_stack_ws_bytes(const ld_config* cfg, int32_t n_layers);

/* Forward of global layer `layer` at step `step` (Preliminary section,
 * transformer form of the training equation).
 *   x:   device [B, S, d], X^l in, X^{l+1} out, in place; rows of dropped
 *        sequences are not touched.
 *   ctx: device, ld_layer_ctx_bytes(cfg) bytes, written (mask, kept lists,
 *        saved activations); consumed by ld_layer_bwd.
 *   ws:  device scratch of ws_bytes >= ld_layer_ws_bytes(cfg).
 *   keep_override: NULL, or device uint8[n_masks][B] used instead of the
 *        Philox masks (test hook for forcing kept counts 0, 1, all, ragged).
 * p in [0, 1]; with p = 1 (or no kept sample) x is left unchanged.  Under
 * LD_GRAN_PER_BATCH without an override the host takes the draw itself and
 * launches nothing for a dropped sub-block (the masks in ctx still say so). */
int ld_layer_fwd(const ld_config* cfg, const ld_weights* w, int32_t layer, float p, uint64_t seed,
                 uint64_t step, void* x, void* ctx, void* ws, size_t ws_bytes,
                 const uint8_t* keep_override, void* stream);

/* Backward of the layer whose forward wrote ctx.
 *   dx: device [B, S, d], dL/dX^{l+1} in, dL/dX^l out, in place; rows of
 *       dropped sequences pass through untouched.
 *   dw: host struct of device float32 gradient pointers, overwritten with
 *       sums over kept rows (zero when no sequence is kept).  The kept
 *       counts are read on the device (every launch is made). */
int ld_layer_bwd(const ld_config* cfg, const ld_weights* w, const void* ctx, void* dx,
                 const ld_grads* dw, void* ws, size_t ws_bytes, void* stream);

/* One training step of an n_layers stack: masks for all layers (one
 * launch), forward through layers 0..L-1, backward through L-1..0.
 *   w, dw: host arrays of n_layers structs (device pointers inside).
 *   p:     host float[n_layers].
 *   x:     device [B, S, d], X^0 in, X^L out (in place).
 *   dx:    device [B, S, d], dL/dX^L in, dL/dX^0 out (in place).
 *   ws:    device, ws_bytes >= ld_stack_ws_bytes(cfg, n_layers).
 *   keep_override: NULL or device uint8[n_layers][n_masks][B] (test hook).
 *   keep_out, idx_out, count_out: NULL or device buffers shaped as in
 *        ld_masks_granular, receiving this step's masks (device-to-device
 *        copies).
 * Under LD_GRAN_PER_BATCH without an override, a layer or sub-block whose
 * draw drops it launches nothing but the zero fill of its weight gradients.
 * n_layers in [1, 1024]. */
int ld_stack_step(const ld_config* cfg, int32_t n_layers, const ld_weights* w, const float* p,
                  uint64_t seed, uint64_t step, void* x, void* dx, const ld_grads* dw, void* ws,
                  size_t ws_bytes, const uint8_t* keep_override, uint8_t* keep_out,
                  int32_t* idx_out, int32_t* count_out, void* stream);

/* ------------------------------------------------ evaluation and decoding
 * Depth-elastic inference (Preliminary section, evaluation equation;
 * Inference Optimizations section).  An active layer applies
 *   Z = X + r_eval f_attn(X),  X' = Z + r_eval f_ffn(Z)
 * to every sequence (no masks); an inactive layer is skipped (identity).
 * Static early exit at l' is active[l] = (l < l'); intermediate layer
 * skipping is any active set; a self-speculative draft decodes with a subset
 * of the layers over the caches the full model wrote.
 *   active: host uint8[n_layers], NULL = every layer.
 *   r_eval: host float[n_layers], NULL = 1 for every layer (the paper's
 *           r_eval = 1, Hyperparameters section).
 *   kv:     host array of n_layers device pointers, each a bf16 cache
 *           [B, s_max, 2 d] holding per position the keys (columns 0..d-1,
 *           head h at h*dh) then the values, as projected by that layer.
 *           Only active layers' caches are read or written. */

/* Bytes of scratch ld_stack_eval needs (one layer's activations). */
size_t ld_eval_ws_bytes(const ld_config* cfg);

/* Forward-only pass of the evaluation form over positions 0..S-1
 * (cfg->seq = S) of every sequence, x [B, S, d] in place.  With kv non-NULL
 * (bf16 only, s_max >= S) each active layer's keys and values of positions
 * 0..S-1 are written to its cache.  fp32 and bf16 configurations. */
int ld_stack_eval(const ld_config* cfg, int32_t n_layers, const ld_weights* w, const uint8_t* active,
                  const float* r_eval, void* x, void* const* kv, int32_t s_max, void* ws,
                  size_t ws_bytes, void* stream);

/* Bytes of scratch ld_stack_decode needs for n_new rows per sequence and
 * caches of s_max positions (0 on invalid arguments). */
size_t ld_decode_ws_bytes(const ld_config* cfg, int32_t n_new, int32_t s_max);

/* Incremental decoding of n_new rows per sequence at positions
 * pos..pos+n_new-1 (the same for every sequence): x [B, n_new, d] in place
 * holds their layer-0 input and receives the output of the last layer.
 * Each active layer first writes the rows' keys/values into its cache at
 * those positions, then attends over positions 0..pos+n_new-1 (causal within
 * the new rows; ALiBi for block kind 1), so positions 0..pos-1 of every
 * active layer's cache must hold valid keys/values (from ld_stack_eval or
 * earlier decoding steps).  The result equals the evaluation form's rows at
 * those positions.  bf16 only; 1 <= n_new <= 8; pos + n_new <= s_max;
 * cfg->seq is not used (it must still form a valid configuration). */
int ld_stack_decode(const ld_config* cfg, int32_t n_layers, const ld_weights* w, const uint8_t* active,
                    const float* r_eval, void* x, void* const* kv, int32_t s_max, int32_t pos,
                    int32_t n_new, void* ws, size_t ws_bytes, void* stream);

/* ------------------------------------------- kernel-level entry points
 * The single kernels the layer is built from, exposed for isolated parity
 * tests and roofline measurements.  dtype is an ld_dtype; all row counts are
 * host values. */

/* y = x * rsqrt(mean_d(x^2) + eps) * g; rstd[row] = that rsqrt (float32).
 * x, y: device [rows, d]; g: device [d].  d <= 4096 (bf16) / 2048 (fp32). */
int ld_rmsnorm_fwd(int32_t dtype, int32_t rows, int32_t d, float eps, const void* x, const void* g,
                   void* y, float* rstd, void* stream);

/* Backward of ld_rmsnorm_fwd given gy:
 *   gx = gres + rstd*(g*gy) - x*rstd^3*mean_d(x*g*gy)   (gres may be NULL)
 *   dg = sum_rows gy*x*rstd   (float32 [d], fixed-order reduction)
 * ws: device scratch of ld_rmsnorm_bwd_ws_bytes(rows, d) bytes. */
size_t ld_rmsnorm_bwd_ws_bytes(int32_t rows, int32_t d);
int ld_rmsnorm_bwd(int32_t dtype, int32_t rows, int32_t d, const void* x, const void* g,
                   const float* rstd, const void* gy, const void* gres, void* gx, float* dg,
                   void* ws, size_t ws_bytes, void* stream);

/* s = relu(u)^2, u and s device [rows, f] (squared ReLU, cited in the
 * paper's Experimental Setup). */
int ld_relu2_fwd(int32_t dtype, int32_t rows, int32_t f, const void* u, void* s, void* stream);
/* gu = gs * 2 relu(u), device [rows, f]. */
int ld_relu2_bwd(int32_t dtype, int32_t rows, int32_t f, const void* u, const void* gs, void* gu,
                 void* stream);

/* s = silu(u) * v with uv = [u | v] device [rows, 2f], s device [rows, f]. */
int ld_swiglu_fwd(int32_t dtype, int32_t rows, int32_t f, const void* uv, void* s, void* stream);
/* guv = [gs * v * silu'(u) | gs * silu(u)], device [rows, 2f]. */
int ld_swiglu_bwd(int32_t dtype, int32_t rows, int32_t f, const void* uv, const void* gs,
                  void* guv, void* stream);

/* C[m, n] = (R ? R[m, n] : 0) + alpha * sum_k A(m, k) * B(n, k)
 *   A(m, k) = A[m*lda + k] if a_kcontig else A[k*lda + m]
 *   B(n, k) = B[n*ldb + k] if b_kcontig else B[k*ldb + n]
 * C (and R) are [M, N] with leading dimension ldc (ldr); C is float32 when
 * c_f32 (R must then be NULL), else dtype.  Forward projections use
 * (1, 1); input gradients (1, 0); weight gradients (0, 0) with c_f32.
 * K may be 0 (C = R or 0).  For LD_BF16, K, lda, ldb must be multiples of 8,
 * and M (N) too when A (B) is not k-contiguous.
 * ws: NULL, or device scratch of ws_bytes; with at least
 * ld_gemm_ws_bytes(...) bytes a float32 GEMM without R may be split along K
 * (partials summed in a fixed order).  Kernel-level diagnostics only. */
size_t ld_gemm_ws_bytes(int32_t dtype, int32_t a_kcontig, int32_t b_kcontig, int32_t M, int32_t N,
                        int32_t K, int32_t ldc, int32_t c_f32);
int ld_gemm(int32_t dtype, int32_t a_kcontig, int32_t b_kcontig, int32_t M, int32_t N, int32_t K,
            const void* A, int32_t lda, const void* B, int32_t ldb, void* C, int32_t ldc,
            int32_t c_f32, float alpha, const void* R, int32_t ldr, void* ws, size_t ws_bytes,
            void* stream);

/* ALiBi slope of head h of n_heads (ALiBi paper, Press et al. 2022, §3):
 * with n the largest power of two <= n_heads, m_h = 2^(-8(h+1)/n) for
 * h < n, and m_h = 2^(-4(2(h-n)+1)/n) for the remaining heads (every other
 * slope of the 2n-head sequence).  Host function; returns 0 for h outside
 * [0, n_heads) or n_heads < 1. */
float ld_alibi_slope(int32_t h, int32_t n_heads);

/* Skinny GEMM of decoding, bf16: C[m, n] = (R ? R[m, n] : 0) + alpha *
 * sum_k A[m, k] W[n, k] for 1 <= M <= 64 rows (A [M, K] and W [N, K] both
 * k-contiguous, 16-byte aligned, lda and ldw multiples of 8, K % 8 == 0).
 * ws: device scratch of ld_gemm_skinny_ws_bytes(M, N, K) bytes (may be 0,
 * then ws may be NULL). */
size_t ld_gemm_skinny_ws_bytes(int32_t M, int32_t N, int32_t K);
int ld_gemm_skinny(int32_t M, int32_t N, int32_t K, const void* A, int32_t lda, const void* W, int32_t ldw,
                   void* C, int32_t ldc, float alpha, const void* R, int32_t ldr, void* ws, size_t ws_bytes,
                   void* stream);

/* Fused projection of a decoding step, bf16, for 1 <= M <= 8 rows (one new
 * row per sequence): the pre-norm, the projection and the feed-forward
 * activation of an active layer of the evaluation form (Preliminary section,
 * evaluation equation; Inference Optimizations section) in one launch,
 *   C[m, n] = act(R[m, n] + alpha * sum_k A'[m, k] W[n, k]),
 * A' = A when g is NULL, else the RMSNorm of A's rows with gain g [K]:
 * A'[m, k] = bf16(A[m, k] * rstd_m * g[k]), rstd_m = 1/sqrt(mean_k A[m, k]^2 + eps).
 *   act 0: none (R optional, [M, N] with leading dimension ldr);
 *   act 1: SwiGLU; W holds 2N rows (gate rows 0..N-1, then up rows N..2N-1)
 *          and C = silu(u) v for u, v = bf16(alpha * A' W_gate^T), likewise
 *          with W_up (R must be NULL);
 *   act 2: squared ReLU, C = relu(bf16(alpha * A' W^T))^2 (R must be NULL).
 * A [M, K], W and C (bf16 [M, N], leading dimension ldc) are device
 * pointers; A, W (and g) 16-byte aligned, lda and ldw multiples of 8,
 * K % 8 == 0.  The rows of A are staged in LDS: K <= 4096 with g, K <= 9664
 * without; LD_E_UNSUPPORTED beyond.  No workspace; deterministic. */
int ld_gemm_dec(int32_t M, int32_t N, int32_t K, const void* A, int32_t lda, const void* g, float eps,
                const void* W, int32_t ldw, void* C, int32_t ldc, float alpha, const void* R, int32_t ldr,
                int32_t act, void* stream);

/* Keys and values of qkv rows (device bf16 [n_seq * n_new, 3 d], row
 * b*n_new + j) into the cache kv (device bf16 [n_seq, s_max, 2 d]) at
 * position pos + j of sequence b. */
int ld_kv_store(int32_t n_seq, int32_t n_new, int32_t d_model, int32_t pos, const void* qkv, void* kv,
                int32_t s_max, void* stream);

/* Decode attention, bf16: the queries of qkv rows b*n_new + j (device
 * [n_seq * n_new, 3 H dh], position pos + j) over positions 0..pos+j of the
 * cache kv (device [n_seq, s_max, 2 H dh], which must already hold the new
 * rows' keys/values), causal, with the ALiBi bias when alibi = 1.
 *   o: device bf16 [n_seq * n_new, H dh].  d_head 64 or 128; n_new <= 8.
 *   ws: device scratch of ld_attn_decode_ws_bytes(n_seq, n_heads, d_head,
 *   s_max) bytes. */
size_t ld_attn_decode_ws_bytes(int32_t n_seq, int32_t n_heads, int32_t d_head, int32_t s_max);
int ld_attn_decode(int32_t n_seq, int32_t n_heads, int32_t d_head, int32_t alibi, int32_t pos, int32_t n_new,
                   const void* qkv, const void* kv, int32_t s_max, void* o, void* ws, size_t ws_bytes,
                   void* stream);

/* Causal multi-head attention over n_seq independent sequences.
 *   qkv: device [n_seq*S, 3*H*dh] as produced by x W_qkv^T;
 *   o:   device [n_seq*S, H*dh]; o[s, h] = softmax_j<=s(q_s.k_j / sqrt(dh)
 *        - alibi * m_h (s - j)) v
 *   lse: device float32 [n_seq, H, S], natural-log sum-exp of the biased
 *        scaled scores of each row (saved for the backward).
 *   alibi: 0 or 1. */
int ld_attn_fwd(int32_t dtype, int32_t n_seq, int32_t seq, int32_t n_heads, int32_t d_head,
                int32_t alibi, const void* qkv, void* o, float* lse, void* stream);

/* Backward of ld_attn_fwd: gqkv (device [n_seq*S, 3*H*dh]) from go
 * (device [n_seq*S, H*dh]); the probabilities are recomputed from lse.
 * ws: device scratch of ld_attn_bwd_ws_bytes(n_seq, seq, n_heads) bytes. */
size_t ld_attn_bwd_ws_bytes(int32_t n_seq, int32_t seq, int32_t n_heads);
int ld_attn_bwd(int32_t dtype, int32_t n_seq, int32_t seq, int32_t n_heads, int32_t d_head,
                int32_t alibi, const void* qkv, const void* o, const float* lse, const void* go,
                void* gqkv, void* ws, size_t ws_bytes, void* stream);

/* ld_attn_bwd with no workspace argument and no allocation, for callers
 * that cannot allocate device memory (code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc).  The delta rows live in a
 * fixed scratch array built into the library: 8 MiB on each GPU it runs on,
 * held until the process ends, so n_seq * n_heads * seq <= 2^21 (larger
 * requests return LD_E_UNSUPPORTED before anything is launched).  Every call
 * on a GPU shares that GPU's array, so calls that overlap on one GPU
 * (other streams or threads) race.  The first call on a device looks up the
 * array's address there.  Arguments and results as ld_attn_bwd. */
int ld_attn_bwd_noalloc(int32_t dtype, int32_t n_seq, int32_t seq, int32_t n_heads, int32_t d_head,
                        int32_t alibi, const void* qkv, const void* o, const float* lse, const void* go,
                        void* gqkv, void* stream);

/* ------------------------------------------------------------- profiling
 * Per-kernel timing with HIP events recorded on the launch stream around
 * every launch of the named kernel (its __global__ name, e.g.
 * "ld_gemm_bf16_nt"), with the launch's algorithmic FLOPs and HBM bytes
 * computed from the kept counts.  Process-wide, not thread-safe; meant for
 * benchmarks.  At most 1 << 16 launches are recorded. */
int ld_prof_start(const char* kernel_name);
int ld_prof_stop(void);
/* Synchronises on the recorded events.  Outputs: number of launches, summed
 * event time in ms, summed algorithmic FLOPs and bytes. */
int ld_prof_result(int64_t* launches, double* total_ms, double* flops, double* bytes);

#ifdef __cplusplus
}
#endif

#endif /* LAYERDROP_H */
