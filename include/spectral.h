/*
 * spectral.h -- C ABI of the per-head spectral-norm estimator and the
 * per-layer FP8 E4M3 scale factor for MI355X (gfx950).
 *
 * What it computes (arXiv 2602.18851):
 *   For every layer l and query head h, sigma_h estimates
 *   ||W^Q_h W^{K T}_{g(h)}||_2 by implicit power iteration (Sec. 4.1 and
 *   App. E, "Power Iteration for Spectral Norm Estimation"): with one
 *   persistent vector v per head,
 *       z = W^{K T} v,  u' = W^Q z,  sigma = ||u'||,  u = u'/sigma,
 *       y = W^{Q T} u,  v' = W^K y,  v = v'/||v'||,
 *   never forming the d x d product.  Grouped-query attention uses the
 *   unexpanded key weights (Sec. 4.2, Prop. "Implicit GQA power iteration"):
 *   query head h reads key head g(h) = floor(h / g), g = n_q / n_kv, and each
 *   key head's weights are read once per sweep for its whole group.
 *   The per-layer scale is Eq. "scale" (Sec. 3.4):
 *       scale_l = alpha * max_h sigma_h * (d / sqrt(d_h)) / (eta_fp8 * r_max).
 *
 * Weight layout (per layer, PyTorch Linear): wq is [n_q*d_h rows][ld],
 * wk is [n_kv*d_h rows][ld], row-major, only the first d_model columns of a
 * row are read.  Rows of head h are h*d_h .. h*d_h+d_h-1, i.e. the transpose
 * of the paper's W^Q_h in R^{d x d_h}.
 *
 * Memory and ownership: every pointer passed to spectral_step is device
 * memory owned by the caller and must stay valid until the work queued on the
 * context's stream has finished.  The library owns only the context and its
 * workspace (allocated in spectral_init, freed in spectral_destroy).
 *
 * Errors: functions return SN_OK (0) or a negative code; spectral_last_error
 * returns a thread-local message for the last failure on the calling thread.
 * Argument and shape errors are detected before anything is queued.
 * Numerical degeneracy is reported per head through sigma and iters.
 *
 * Threading: a context may be used by one host thread at a time.  Distinct
 * contexts are independent.
 */
#ifndef SPECTRAL_H
#define SPECTRAL_H

#include <stdint.h>

#if defined(__GNUC__)
#define SN_API __attribute__((visibility("default")))
#else
#define SN_API
#endif

#ifdef __cplusplus
extern "C" {
#endif

#define SN_OK 0
#define SN_EINVAL (-1)   /* bad shape, parameter, size or alignment            */
#define SN_ENULL (-2)    /* a required pointer is NULL                          */
#define SN_EDTYPE (-3)   /* dtype is neither SN_F32 nor SN_BF16                 */
#define SN_EHIP (-4)     /* a HIP runtime call failed (message has its text)    */
#define SN_ESTATE (-5)   /* context not usable (e.g. no device)                 */

typedef enum { SN_F32 = 0, SN_BF16 = 1 } sn_dtype;

typedef struct {
  int32_t n_layers;    /* L >= 1                                                  */
  int32_t d_model;     /* d >= 1: model width (LayerNorm/RMSNorm width, Sec. 3.1) */
  int32_t n_q_heads;   /* n_q >= 1                                                */
  int32_t n_kv_heads;  /* n_kv >= 1, divides n_q (n_kv == n_q: multi-head)        */
  int32_t head_dim;    /* d_h: one of 8, 16, 32, 64, 128; d_h * ld * element size
                          must stay below 2^31 bytes                              */
  int32_t dtype;       /* sn_dtype of the weights; vectors are always float32     */
  int64_t ld;          /* row stride of wq and wk in elements; 0 means d_model.
                          ld * element size must be a multiple of 16 bytes.       */
} sn_shape;

typedef struct {
  float alpha;         /* calibration factor alpha > 0 (Eq. "calibrated_bound")   */
  float eta_fp8;       /* FP8 margin, 0 < eta_fp8 (the paper uses 0.8)            */
  float r_max;         /* largest finite FP8 magnitude, 448 for OCP E4M3          */
  float tol;           /* 0: run exactly n_iter iterations.  > 0: stop a head
                          after step k >= 2 once |sigma_k - sigma_{k-1}| <=
                          tol * sigma_k, with n_iter as the cap.  With
                          head_dim >= 16 the workspace then also holds the
                          Gram matrices of the tail (see spectral_step; 240 MB
                          at 80 x 64 heads of d_h 128, d 8192).                   */
  int32_t q_strips;    /* column strips per head in the W_Q sweep; 0 = automatic  */
  int32_t k_strips;    /* column strips per KV head in the W_K sweep; 0 = auto    */
  int32_t flags;       /* SN_FLAG_* bits; 0 for the defaults                      */
} sn_params;

/* Run the W_K sweeps of grouped heads on the vector ALUs even where the
 * matrix-core kernel applies (bf16 weights, d_h 64 or 128, >= 3 query heads
 * per KV head).  Results agree to rounding; the flag exists for comparison. */
#define SN_FLAG_VALU_K_SWEEP 1

/* Gram form of the same iteration.  For one head, ||W^Q z||^2 = z^T G_Q z
 * with G_Q = Q_h Q_h^T (d_h x d_h), and ||W^K y||^2 = y^T G_K y with
 * G_K = K_j K_j^T, so the step maps of Sec. 4.1 factor through the two Gram
 * matrices:  y = G_Q z / sigma,  z_next = G_K y / ||v'||.  With this flag one
 * sweep over all weights forms G_Q for every query head and G_K for every
 * key head on the matrix cores, the iteration runs in d_h-space, and one
 * final W_K sweep (plus one W_Q sweep when u is requested) maps the last y
 * (z) back to v (u).  The iterates, sigma, u and v are those of the default
 * path up to rounding; the weights are read about four times per call
 * instead of twice per iteration.  Needs head_dim >= 16.  The workspace
 * grows by the Gram partials, 2 d_h (d_h + 16) bytes per query or key head
 * and column strip (spectral_workspace_bytes gives the total). */
#define SN_FLAG_GRAM 2

/* Reserve the workspace of the layer-level form (spectral_step_layer): the
 * row-sweep partials, one d_h-vector per query head, the column sums (one row
 * of d_model rounded up to 64 per layer and row split, up to n_q splits on
 * small shapes) and per-layer vectors; spectral_workspace_bytes gives the
 * total.  spectral_step itself is unaffected. */
#define SN_FLAG_LAYER 4


typedef struct sn_ctx sn_ctx;

/* Creates a context for one model shape on the current HIP device and
 * allocates its workspace and a device table of the layer pointers.
 * hip_stream is a hipStream_t (NULL = the default stream) on which every
 * later spectral_step is queued.  On success *ctx receives the handle.
 * Errors: SN_ENULL, SN_EINVAL, SN_EDTYPE, SN_EHIP. */
SN_API int spectral_init(sn_ctx** ctx, const sn_shape* shape, const sn_params* params,
                         void* hip_stream);

/* One estimation call over all layers and heads (Sec. 4.1; App. E).
 *   wq_layers  host array of n_layers device pointers, layer l -> wq of l
 *              (16-byte aligned).
 *   wk_layers  host array of n_layers device pointers to wk.
 *   v          device float32 [n_layers][n_q][d_model], in/out: the
 *              persistent right vectors.  Read as the start vectors (any
 *              nonzero finite vectors; normalised on entry), overwritten with
 *              the unit vector after the last step of each head.
 *   u          device float32 [n_layers][n_q][d_model] or NULL: receives the
 *              unit left vector u of each head's last step.
 *   n_iter     >= 1: iterations (tol == 0) or the cap (tol > 0).
 *   sigma      device float32 [n_layers][n_q]: the estimate of the last step,
 *              sigma = ||M v|| taken before v moves.
 *   scale      device float32 [n_layers]: Eq. "scale" with max_h sigma_h;
 *              NaN if any head of the layer is NaN.
 *   iters      device int32 [n_layers][n_q] or NULL: steps run per head;
 *              -1 if the start vector is zero or not finite (sigma = NaN,
 *              v unchanged, u = 0); -2 if M v = 0 (sigma = 0, v normalised
 *              start vector, u = 0).
 * The call is queued asynchronously on the context's stream and never waits
 * on the host.  With tol > 0 and head_dim >= 16, the first two steps (the
 * fewest the stopping rule allows) run as sweeps over all heads; then one
 * fixed sequence of launches lists the heads still running on the device,
 * forms their Gram matrices G_Q = Q_h Q_h^T and G_K = K_j K_j^T (see
 * SN_FLAG_GRAM), continues their iteration in d_h-space to the tolerance or
 * the cap, and maps the last vectors back to v (and u) with sweeps over the
 * listed heads only; the iterates are those of the sweeps up to rounding.
 * (With head_dim 8 every step runs as sweeps over all heads; stopped heads
 * leave them at once.)  The layer pointers reach the kernels through a
 * device table written by a small kernel whose launch arguments carry them:
 * an eager call rewrites it only when the pointers change; a call being
 * captured into a HIP graph always writes its own copy, so every replay
 * uses the pointers of its capture (graphs captured from one context must
 * not replay concurrently).  Every form and mode can be captured.  Weights
 * and vectors must not alias the outputs.  Errors: SN_ENULL, SN_EINVAL,
 * SN_EHIP. */
SN_API int spectral_step(sn_ctx* ctx, const void* const* wq_layers, const void* const* wk_layers,
                         float* v, float* u, int32_t n_iter, float* sigma, float* scale,
                         int32_t* iters);

/* Allocation-free variant of spectral_step, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc).  It needs no context: shape, params
 * (SN_FLAG_LAYER ignored) and hip_stream as for spectral_init, the other
 * arguments as for spectral_step, whose results it gives bit for bit.  Its
 * workspace and layer-pointer table live in a static device array of
 * 32 MiB that each device holds from the first call on it until the process
 * ends; a shape whose workspace (spectral_workspace_bytes) plus 4 n_layers
 * pointers, rounded up to 256 bytes, does not fit is rejected with
 * SN_EINVAL before anything is queued.  The call allocates nothing (no
 * hipMalloc, hipFree, event or allocating library routine).  Every call on
 * a device shares that device's array, which keeps the last call's
 * contents: calls that overlap on one device (queued on different streams,
 * or from several threads without ordering) race and give wrong results.
 * Errors: SN_ENULL, SN_EINVAL, SN_EDTYPE, SN_ESTATE, SN_EHIP. */
SN_API int spectral_step_noalloc(const sn_shape* shape, const sn_params* params, const void* const* wq_layers,
                                 const void* const* wk_layers, float* v, float* u, int32_t n_iter, float* sigma,
                                 float* scale, int32_t* iters, void* hip_stream);

/* The layer-level estimator exactly as the paper prints it (App. E,
 * "Implicit GQA Power Iteration"; g = 1 is the multi-head algorithm of
 * Sec. 4.1): one pair u, v in R^d per layer for the concatenated
 * W^Q = [W^Q_1 .. W^Q_{n_q}] and the key weights expanded implicitly,
 *     z = RepeatBlocks(W^{K T} v, g),  u' = W^Q z,  sigma = ||u'||,
 *     y = W^{Q T} u,  v' = W^K SumGroups(y, g),  v = v'/||v'||,
 * so sigma estimates || sum_h W^Q_h W^{K T}_{g(h)} ||_2 for the whole layer
 * (not max_h of the per-head norms that spectral_step returns).  Needs a
 * context created with SN_FLAG_LAYER (else SN_ESTATE).
 *   wq_layers, wk_layers  as for spectral_step.
 *   v      device float32 [n_layers][d_model], in/out: the persistent right
 *          vector of each layer (normalised on entry, unit vector on exit).
 *   u      device float32 [n_layers][d_model] or NULL: the unit left vector.
 *   n_iter >= 1 iterations (fixed count; params.tol does not apply).
 *   sigma  device float32 [n_layers]: the estimate of the last step.
 *   scale  device float32 [n_layers]: Eq. "scale" with that sigma.
 * A layer whose start vector is zero or not finite gets sigma = scale = NaN,
 * v unchanged and u = 0; one with M v = 0 gets sigma = scale = 0, v the
 * normalised start vector and u = 0.  Queued on the context's stream; never
 * waits.  Errors: SN_ENULL, SN_EINVAL, SN_ESTATE, SN_EHIP. */
SN_API int spectral_step_layer(sn_ctx* ctx, const void* const* wq_layers, const void* const* wk_layers,
                               float* v, float* u, int32_t n_iter, float* sigma, float* scale);

/* ---- FP8 E4M3 consumer of the scale ----------------------------------
 *
 * Stage 3 of the geometry-aware forward pass (Sec. 3.4, Algorithm
 * "Geometry-Aware Attention Forward Pass") up to the quantised logits, for
 * every layer l and query head h:
 *     Q = X_l W^Q,  K = X_l W^K,  S_h = Q_h K_{g(h)}^T / sqrt(d_h),
 *     S~_h = S_h / scale_l  ->  OCP E4M3FN codes (round to nearest even;
 *                              |S~| > 464 gives NaN, 0x7F | sign),
 * with the statistics of Sec. 1 (overflow when |S~| > 448) and Table
 * "pretrained" (largest scaled logit).  Key heads are not expanded.  The
 * projections accumulate in fp32 and the logits are formed to about 2^-15
 * relative precision (three bf16 matrix-core products on hi/lo halves).
 * Needs bf16 weights and tokens and head_dim 16, 32, 64 or 128.
 *
 * spectral_logits_workspace_bytes: device scratch the call needs: a table
 * of 3 n_layers device pointers (padded to 256 bytes), then the Q and K of
 * every layer as hi and lo bf16 planes (n_layers * seq_len * (n_q + n_kv) *
 * head_dim * 4 bytes).  One launch of each kernel covers all layers.
 *
 * spectral_logits_fp8:
 *   x_layers   host array of n_layers device pointers: tokens of layer l,
 *              bf16 [seq_len][ld_x] (ld_x = 0: d_model), 16-byte aligned.
 *   wq_layers, wk_layers  as for spectral_step.
 *   scale      device float32 [n_layers] (e.g. spectral_step's output).
 *   workspace  device scratch of >= workspace_bytes bytes, 256-byte aligned,
 *              owned by the caller; contents are overwritten.
 *   codes      device uint8 [n_layers][n_q][seq_len][seq_len] or NULL
 *              (16-byte aligned): E4M3 codes of S~, row i, column j.
 *   max_abs    device float32 [n_layers][n_q]: max |S~| per head.
 *   n_over     device int32 [n_layers][n_q]: #{(i, j): |S~_ij| > 448}.
 * A scaled logit that is not finite (a NaN or zero scale) counts as an
 * overflow and makes max_abs non-finite (NaN for a NaN scale).
 * Queued on the context's stream; allocates nothing; seq_len <= 46340, and
 * one layer's W_Q (n_q * head_dim rows of ld bf16) below 4 GiB (else
 * SN_EINVAL).  The layer pointer table is written into the workspace by a
 * kernel whose launch arguments carry the pointers, so the call can be
 * captured into a HIP graph.
 * Errors: SN_ENULL, SN_EINVAL, SN_EDTYPE, SN_ESTATE. */
SN_API int spectral_logits_workspace_bytes(const sn_shape* shape, int32_t seq_len, int64_t* bytes);
SN_API int spectral_logits_fp8(sn_ctx* ctx, const void* const* x_layers, int64_t ld_x, int32_t seq_len,
                               const void* const* wq_layers, const void* const* wk_layers, const float* scale,
                               void* workspace, int64_t workspace_bytes, uint8_t* codes, float* max_abs,
                               int32_t* n_over);

/* Redirects later calls to another hipStream_t.  Unless either stream is
 * being captured, the new stream is first made to wait for all work queued
 * on the previous one (they share the workspace and the pointer table). */
SN_API int spectral_set_stream(sn_ctx* ctx, void* hip_stream);

/* Frees the context and its workspace (waits for its queued work first). */
SN_API void spectral_destroy(sn_ctx* ctx);

/* Thread-local text of the last error ("" if none). */
SN_API const char* spectral_last_error(void);

/* Bytes of device workspace spectral_init allocates for this shape. */
SN_API int spectral_workspace_bytes(const sn_shape* shape, const sn_params* params,
                                    int64_t* bytes);

/* Per-kernel timing.  With enable != 0 every later launch is bracketed by
 * HIP events on the context's stream.  spectral_profile_read waits for the
 * stream and returns, per kernel kind (0 = first W_K sweep from v,
 * 1 = W_Q sweep, 2 = W_K sweep, 3 = finalize, 4 = Gram sweep, 5 = d_h-space
 * iteration, 6 = final sweeps of the Gram form, 7 = row sweeps of the
 * layer-level form, 8 = its column sweeps, 9 = its reductions and
 * finalize, 10 = projections of the logit consumer, 11 = its logit
 * kernels, 12 = the running-head lists of tolerance mode), the summed
 * device time in
 * milliseconds and the number of launches since the previous read, then
 * resets both.  ms and launches point to SN_PROFILE_KINDS host elements
 * each. */
#define SN_PROFILE_KINDS 13
SN_API int spectral_profile(sn_ctx* ctx, int32_t enable);
SN_API int spectral_profile_read(sn_ctx* ctx, double* ms, int64_t* launches);

/* ---- host-side calibration helpers (no GPU involved) ------------------
 *
 * spectral_alpha_select: the selection rule of Sec. 3.2.  gamma is the
 * smallest gamma > 1 with gamma - 1 - ln(gamma) >= (2 / d_h) ln(2 N L / delta)
 * (Eq. "gamma_selection"), and alpha_min = sqrt(2 gamma d_h) / d *
 * sqrt(ln(4 N L^2 / delta)) (Eq. "alpha_selection"), with N = n_heads_total
 * (layers x query heads) and L = seq_len.  Writes both to host doubles.
 * Errors: SN_ENULL, SN_EINVAL (sizes < 1, delta outside (0, 1)). */
SN_API int spectral_alpha_select(int32_t d_model, int32_t head_dim, int64_t n_heads_total, int64_t seq_len,
                                 double delta, double* gamma, double* alpha_min);

/* T1 = L exp(-(d_h / 2)(gamma - 1 - ln gamma)), T2 = 2 L^2 exp(-d^2 alpha^2 /
 * (2 gamma d_h)) of Prop. "Rank-aware overflow probability bound", for one
 * head.  Errors: SN_ENULL, SN_EINVAL (alpha <= 0, gamma <= 1, sizes < 1). */
SN_API int spectral_overflow_terms(int32_t d_model, int32_t head_dim, int64_t seq_len, double alpha,
                                   double gamma, double* t1, double* t2);

/* Auto-alpha (Sec. 3.5, App. M): alpha = Quantile_q(slack) * kappa over n
 * burn-in slack ratios (host array), the quantile interpolating linearly
 * between order statistics at position q (n - 1).  Errors: SN_ENULL,
 * SN_EINVAL (n < 1, q outside [0, 1], kappa < 1, a negative or non-finite
 * ratio). */
SN_API int spectral_auto_alpha(const double* slack, int64_t n, double quantile, double kappa, double* alpha);

/* Slack ratio r = max|S| / B_max with B_max = sigma_layer * d / sqrt(d_h)
 * (Sec. 3.5, Eq. "bound"). */
SN_API double spectral_slack_ratio(double max_abs_logit, double sigma_layer, int32_t d_model, int32_t head_dim);

#ifdef __cplusplus
}
#endif

#endif /* SPECTRAL_H */
