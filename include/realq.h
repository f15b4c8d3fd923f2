/*
 * realq.h - C ABI of the REAL-Q per-layer quantization sweep on MI355X (gfx950).
 *
 * The library quantizes one linear module W (m x n, row = output channel) to
 * asymmetric group-wise integers with GPTQ-style compensation, and after every
 * column block runs Block-wise Gradient Descent on the not-yet-quantized columns
 * (REAL-Q, Sec. 3-4 and Alg. 1 of Appendix A).
 *
 * Conventions shared by every entry point:
 *   - All array arguments are DEVICE pointers owned by the caller, row-major and
 *     contiguous unless a leading dimension says otherwise.  bf16 arrays are passed
 *     as uint16_t bit patterns.  The library never frees caller memory.
 *   - Work is enqueued on the HIP stream given to realq_ctx_create and is
 *     asynchronous unless stated; caller buffers must stay alive until the stream
 *     has passed the work.
 *   - Return value: REALQ_OK (0) or a negative REALQ_ERR_* code.  Arguments are
 *     validated before anything is launched, so an error return from validation
 *     leaves all outputs untouched.  An error detected after launch (a HIP error,
 *     a non-positive-definite Hessian) leaves outputs undefined.
 *     realq_last_error(ctx) returns a message for the last failure on that context.
 *   - A context is not thread-safe; use one context per host thread / stream.
 *
 * Shapes: m output channels, n input channels (columns), T calibration tokens.
 * Calibration inputs are token-major: X[t*n + j].
 */
#ifndef REALQ_H
#define REALQ_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define REALQ_OK               0
#define REALQ_ERR_INVALID_ARG (-1) /* NULL where not allowed, bad parameter value           */
#define REALQ_ERR_SHAPE       (-2) /* inconsistent or unsupported sizes                     */
#define REALQ_ERR_NOT_SPD     (-3) /* damped Hessian not positive definite                  */
#define REALQ_ERR_HIP         (-4) /* HIP runtime error (launch, copy, event)               */
#define REALQ_ERR_OOM         (-5) /* device allocation failed                              */
#define REALQ_ERR_NONFINITE   (-6) /* non-finite value found in an input checked on device  */

typedef struct realq_ctx realq_ctx;             /* stream (borrowed), workspaces, last error */
typedef struct realq_bgd_state realq_bgd_state; /* per-module BGD state, see realq_bgd_state_create */

/* Quantizer and GPTQ parameters.
 *   bits  : code width, 2..4 (codes are 0 .. 2^bits-1)                     [4]
 *   group : columns sharing one (scale, zero) per row, >= 1; 0 = one group
 *           per row (per-row quantization, the paper's W4A16 setting)      [128]
 *   block : GPTQ column block B (Sec. 3.2), 1..128; BGD runs after each    [128]
 *   grid  : number of shrink factors p_k = 1 - k/100, k = 0..grid-1, 1..100 [80]
 *   damp  : relative damping, lambda = damp * mean(diag H), > 0            [0.01]
 *   sym   : 0 = asymmetric (range [min(0, x), max(0, x)], zero searched);
 *           1 = symmetric (Sec. 6.1: range [-max|x|, max|x|], zero fixed at
 *           2^(bits-1), only the shrink factor searched)                  [0]
 * With group > 0 either block % group == 0 or group % block == 0 must hold. */
typedef struct realq_qparams {
    int32_t bits, group, block, grid;
    float damp;
    int32_t sym;
} realq_qparams;

/* Block-GD parameters (Sec. 4.3, Eq. block_gd_update; Adam constants of Appendix D.1).
 *   steps     : Adam steps after every column block (0 = plain GPTQ)
 *   lr        : learning rate eta
 *   beta1, beta2, eps : Adam constants [0.9, 0.999, 1e-8]
 *   tok_chunk : tokens per streamed chunk of the residual/gradient GEMMs (0 = all T)
 *   form      : REALQ_BGD_TOKENS or REALQ_BGD_GRAM (below) [REALQ_BGD_TOKENS]
 *   loss_clip : output-perturbation clip quantile q in (0, 1], 0 = off [0] (Appendix D.1,
 *               a_loss_clip): each step scales every token's channels whose |R| exceeds
 *               the token's nearest-rank q-quantile over the m channels down to it, the
 *               factor c = tau_t / |R| held fixed (loss sum s (cR)^2, gradient through
 *               c^2 R).  Needs the identity metric (no M, no window partner P).
 *   batch     : tokens per BGD step, 0 = all T [0] (Sec. 4.3, calibration mini-batch):
 *               Adam step t of the module (1-based) uses the consecutive token batch
 *               (t - 1) mod ceil(T / batch); loss and gradient are normalised by its
 *               size.  The final loss is always over all T tokens and unclipped.
 *   resid_increment : 1 = allowed [1], 0 = never.  Residual, gradient and loss are
 *               linear or quadratic in the weights, so within one column block step k > 0
 *               can take them from the block's first step (residual R_0, gradient G_0, loss
 *               L_0) and the weight change Delta = bf16(W_k - W_0)_J: R_k = R_0 + Q_k with
 *               Q_k = Delta Xhat_J^T, G_k = G_0 + M_a bf16(Q_k o s) Xhat_J / T and, for
 *               M_a = I, loss L_0 + <G_0, Delta> + sum s Q_k^2 / 2T.  One bf16 MFMA pass over
 *               Delta for Q_k and one over Q_k for the gradient, instead of two over the
 *               float32 D = W - W0 and R o s; R_0 itself is never stored.  Token form, no
 *               clip, batch = T, and only where the change is small enough that its bf16
 *               rounding stays below what the sweep's decisions resolve: the weights cannot
 *               move by more than rms(W0) / 32 within a block ((steps - 1) lr (1 - beta1) /
 *               sqrt((1 - beta2)(1 - beta1^2/beta2)) bounds that move: the Adam step's
 *               supremum over every gradient history; needs beta1^2 < beta2), n <= 8192 (at
 *               most 64 column blocks carry the rounding forward) and T >= 16 n (the
 *               gradient's rounding averages over at least 16 tokens per input column).
 *               Costs [m, n] arrays (two float32, one bf16).
 *   The Gram form takes neither a clip nor a batch smaller than T. */
typedef struct realq_bgd_params {
    int32_t steps;
    float lr, beta1, beta2, eps;
    int64_t tok_chunk;
    int32_t form;
    float loss_clip;
    int64_t batch;
    int32_t resid_increment;
} realq_bgd_params;

/* realq_bgd_params.form: how the loss and gradient of a BGD step are evaluated.
 *   REALQ_BGD_TOKENS  residual and gradient GEMMs streamed over all T tokens every step
 *                     (R = B + D_J Xhat_J^T, G = M_a (R o s) Xhat_J / T).
 *   REALQ_BGD_GRAM    the same loss and gradient through the calibration Gram matrices,
 *                     which exist because the surrogate at the module output is quadratic
 *                     in W: with D = W - W0, Delta = Xhat - X, G_ab = a^T diag(s) b,
 *                       gradient = M_a (W0 G_dh + D G_hh)[:, J] / T,
 *                       2T L     = <W0 G_dd, W0> + 2 <W0 G_dh, D> + <D G_hh, D>   (M_a = I),
 *                     one m x n x n product per step instead of two m x T x |J| ones and no
 *                     [m, T] residual base. */
#define REALQ_BGD_TOKENS 0
#define REALQ_BGD_GRAM 1

/* Fill *q / *b with the defaults given above. */
void realq_qparams_default(realq_qparams* q);
void realq_bgd_params_default(realq_bgd_params* b);

/* ------------------------------------------------------------------ context */

/* Create a context bound to hip_stream (a hipStream_t; NULL = the null stream) on
 * the current device.  The stream is borrowed, not owned. */
int realq_ctx_create(realq_ctx** out, void* hip_stream);
void realq_ctx_destroy(realq_ctx* ctx);
const char* realq_last_error(const realq_ctx* ctx);

/* Kernel timing: when enabled, the library brackets the launches of its main
 * kernels with HIP events on its stream and accumulates their durations, read with
 * realq_ctx_kernel_time after the stream has drained.  Names: "hessian",
 * "chol", "quantize", "obs", "lock", "resid", "grad", "resid_inc" and "grad_inc" (the
 * residual and gradient GEMMs of the Block-GD steps that take increments, see
 * resid_increment), "adam", "init", "gram" (Gram
 * matrices of the input perturbation), "gram_step" (the per-step product of the
 * Gram form), "dense_loss" (final loss with a dense metric), "saliency", "block_init" and
 * "block_step" (the block sweeps: the fixed forwards, one Block-GD step) and "attention"
 * (realq_decoder_block_sweep: each attention forward or backward with its rotary embeddings),
 * "metric" (the dense-metric product of a Block-GD step).
 * Returns REALQ_ERR_INVALID_ARG for an unknown name.  Independently of this switch, each of
 * these phases (and each column block of realq_quantize_layer) is a roctx range of the same
 * name around its launches, visible with `rocprofv3 --marker-trace`. */
int realq_ctx_set_timing(realq_ctx* ctx, int enable);
int realq_ctx_kernel_time(realq_ctx* ctx, const char* name, int64_t* launches, double* total_ms);
int realq_ctx_reset_timing(realq_ctx* ctx);

/* ------------------------------------------------------------------ a0: Stage-0 accumulators
 * Stage 0 of Alg. 1 derives two per-module quantities from the per-token gradients
 * g_t = dL/dy_t of the module's output, G: [T, m] bf16, token-major (G[t*m + i]).
 *
 * Aggregated Fisher (Eq. fisher_full): F = (1/T) sum_t g_t g_t^T.  realq_fisher_accum adds
 * sum_t g_t g_t^T over the T tokens given to F_acc ([m,m] float64, caller-initialised,
 * typically zeroed), one call per token chunk (the same MFMA contraction as the Hessian, bf16
 * products accumulated in float32 per tile and in float64 across tiles).  realq_fisher_finish
 * writes F = F_acc / T_total as the float32 [m,m] metric that realq_bgd_state_create and
 * realq_layer_desc take as M.  T == 0 is a no-op; T_total must be > 0. */
int realq_fisher_accum(realq_ctx* ctx, const uint16_t* G /*[T,m]*/, int64_t T, int64_t m, double* F_acc /*[m,m]*/);
int realq_fisher_finish(realq_ctx* ctx, const double* F_acc, int64_t m, int64_t T_total, float* F /*[m,m]*/);

/* Saliency per row group (Sec. 3.3, Eq. saliency_hessian).  The m output channels are cut into
 * n_groups contiguous row groups of r = ceil(m / n_groups) channels (the last one shorter; a
 * group that would start at or past m is empty), and
 *   s_out[g*T + t] = sum over the channels i of group g of G[t, i]^2
 * (squares and sums in float64, stored as float32).  clip_q in (0, 1] then clips every group's
 * row at its nearest-rank clip_q quantile over the T tokens, the k-th smallest value with
 * k = ceil(clip_q * T) evaluated in double from the float32 clip_q (Appendix D.1's Hessian-side
 * saliency clipping uses 0.99); clip_q = 0 disables the clip.  s_out is [n_groups, T] float32;
 * rows of empty groups are written as zeros.  G must be finite.  1 <= n_groups <= m.  All T
 * tokens are passed in one call, since the clip is a quantile over them.  T == 0 is a no-op. */
int realq_saliency(realq_ctx* ctx, const uint16_t* G /*[T,m]*/, int64_t T, int64_t m, int32_t n_groups, float clip_q,
                   float* s_out /*[n_groups,T]*/);

/* ------------------------------------------------------------------ diagnostics (not part of the method)
 * The bf16 MFMA rate the GPU sustains on a register-resident loop (v_mfma_f32_32x32x16_bf16,
 * eight independent accumulator chains per wave, two waves per SIMD, four blocks per CU; no
 * memory traffic in the loop), in TFLOP/s written to *tflops (host).  The sweep's MFMA fraction is
 * reported against it beside the data-sheet peak.  iters in 1 .. 2^24 rounds per wave (2^16 takes
 * about 50 ms).  Synchronises the stream. */
int realq_mfma_peak(realq_ctx* ctx, int64_t iters, double* tflops);

/* ------------------------------------------------------------------ a1: Hessian
 * Sec. 3.2 (H = (2/T) sum_t x_t x_t^T) and Eq. saliency_hessian (per-token weights).
 * H_acc[n*n] (float64, caller-initialised, typically zeroed) += sum_t s_t xhat_t xhat_t^T
 * over the T tokens given.  Call once per token chunk; the 2/T scale is applied by
 * realq_chol_inverse with the total token count.  s may be NULL (all ones).
 * T == 0 is a no-op.  The full symmetric matrix is written.  Precision: the bf16 products
 * are exact; s_t xhat_t is formed in float32 and carried as three bf16 terms (all of its
 * 24 bits); tiles accumulate in float32 over a token chunk and in float64 across chunks. */
int realq_hessian_accum(realq_ctx* ctx, const uint16_t* Xhat /*[T,n]*/, const float* s /*[T]|NULL*/,
                        int64_t T, int64_t n, double* H_acc /*[n,n]*/);

/* For callers that cannot allocate device memory (code under HIP graph capture, tight serving
 * loops, harnesses that forbid hipMalloc): the same accumulation as realq_hessian_accum, with the
 * token chunks staged in a fixed scratch array of REALQ_NOALLOC_SCRATCH_BYTES that the library
 * holds on each GPU it runs on (from the first call on that GPU until the process ends) instead of
 * context workspaces; it calls no device allocator.  Chunks are shorter than realq_hessian_accum's,
 * so float64 sums across chunks may differ from it in the last bits.  n > REALQ_NOALLOC_MAX_N gives
 * REALQ_ERR_SHAPE.  Every call on one GPU shares that GPU's scratch array: calls that overlap on one
 * GPU (from several streams or threads) race and must be serialised by the caller.  Nothing in the
 * array needs clearing between calls. */
#define REALQ_NOALLOC_SCRATCH_BYTES (64ll << 20)
#define REALQ_NOALLOC_MAX_N 32768
int realq_hessian_accum_noalloc(realq_ctx* ctx, const uint16_t* Xhat /*[T,n]*/, const float* s /*[T]|NULL*/,
                                int64_t T, int64_t n, double* H_acc /*[n,n]*/);

/* ------------------------------------------------------------------ a2: inverse factor
 * H = (2/T_total) H_acc is written to H_out (float32) when H_out != NULL.  Dead
 * columns (H_jj == 0) get H_jj = 1 and are flagged in dead[j] (when non-NULL);
 * then H_d = H + damp*mean(diag H) I, and U (upper triangular, positive diagonal,
 * float32, lower triangle zero) with H_d^{-1} = U^T U is written.  Row j of U
 * over U_jj is the compensation direction of Eq. gptq_update (Sec. 3.2) with the
 * sequentially eliminated inverse.  Computed in float64.  Synchronises the stream
 * once to read two flags: REALQ_ERR_NONFINITE if H_acc holds a NaN or an infinity (a
 * non-finite Xhat or s reached the Hessian), else REALQ_ERR_NOT_SPD if the factorisation
 * fails (retry with a larger damp). */
int realq_chol_inverse(realq_ctx* ctx, const double* H_acc, int64_t n, int64_t T_total, float damp,
                       float* H_out /*[n,n]|NULL*/, float* U /*[n,n]*/, uint8_t* dead /*[n]|NULL*/);

/* ------------------------------------------------------------------ BGD state
 * Per-module state of Block-GD (Sec. 4.3): the residual base
 *   B = W0 (Xhat - X)^T + (W_locked - W0_locked) Xhat_locked^T      ([m,T] float32),
 * the Adam moments (m, v, [m,n] float32), the step counter, a transposed copy of
 * Xhat and the split of W - W0 the GEMMs consume.  W0, X, Xhat, s, M and P are
 * borrowed and must stay valid for the state's lifetime.
 *   X    : inputs of the full-precision model ([T,n] bf16); Xhat: inputs the
 *          partially quantized model feeds this module ([T,n] bf16); X == Xhat
 *          (same pointer) is allowed.
 *   s    : per-token weights [T] or NULL (all ones).
 *   M    : surrogate output metric [m,m] float32 (symmetric) or NULL (identity):
 *          the aggregated Fisher of Eq. fisher_full / fisher_loss.
 *   P    : consumer's pulled-back metric [m,m] float32 or NULL, blended with M by
 *          the sliding window (Eq. slide_window).
 * The state assumes the caller's working weights start equal to W0 and are only
 * changed through realq_quantize_block / realq_bgd_step afterwards.  When the other
 * conditions of resid_increment hold, creation synchronises the stream once to read
 * rms(W0). */
int realq_bgd_state_create(realq_ctx* ctx, realq_bgd_state** out, const float* W0 /*[m,n]*/,
                           const uint16_t* X /*[T,n]*/, const uint16_t* Xhat /*[T,n]*/,
                           const float* s /*[T]|NULL*/, const float* M /*[m,m]|NULL*/,
                           const float* P /*[m,m]|NULL*/, int64_t m, int64_t n, int64_t T,
                           const realq_bgd_params* params);
void realq_bgd_state_destroy(realq_bgd_state* st);

/* ------------------------------------------------------------------ a3-a6: one column block
 * W is the caller's float64 working copy of the weights [m, n] (device, row-major),
 * started from W0 and changed only by these calls: every column takes many small
 * updates before it is quantized, and float64 keeps its rounding decisions those of
 * exact arithmetic.
 * Quantize columns [c0, c0+bs) of W (in place; the block is written back
 * dequantized) following Alg. 1's inner loop: dead columns of the block are zeroed,
 * group (scale, zero) parameters are searched when a group starts, each column is
 * quantized and its error compensated on the block's remaining columns
 * (Eq. gptq_update), then all columns >= c0+bs get the batch update W -= E_b U_{b,:}
 * (Sec. 3.2).  Writes codes (uint8, 0..2^bits-1), scales ([m, ceil(n/group)] float32)
 * and zeros ([m, ceil(n/group)] uint8, one column when group = 0) for the groups touched.  Group parameters of a
 * group that started in an earlier block are read back from scales/zeros.
 * U and dead come from realq_chol_inverse.  When st != NULL the residual base of
 * the state is also advanced by the locked block (Sec. 4.3: quantized weights stay
 * locked).  Requirements: c0 is a multiple of qp->block, bs == qp->block except for
 * the last block (c0 + bs == n), bs <= 128, and blocks are quantized in column order;
 * otherwise REALQ_ERR_SHAPE. */
int realq_quantize_block(realq_ctx* ctx, double* W /*[m,n]*/, int64_t m, int64_t n, int64_t c0, int64_t bs,
                         const float* U /*[n,n]*/, const uint8_t* dead /*[n]|NULL*/, const realq_qparams* qp,
                         uint8_t* codes /*[m,n]*/, float* scales, uint8_t* zeros, realq_bgd_state* st);

/* Row groups (Eq. saliency_hessian): each group of output rows is quantized with its own inverse
 * factor.  realq_quantize_block_rows does what realq_quantize_block does for rows [r0, r1) only
 * (W, codes, scales and zeros are the full [m, ...] arrays; U and dead are the group's), and
 * with st != NULL refreshes the state's copy of W - W0 on those rows, but does not advance the
 * residual base.  After every row group of a block has been quantized, realq_bgd_lock_block
 * folds the block [c0, c0 + bs) into the state (the lock realq_quantize_block performs itself).
 * Requirements as for realq_quantize_block, plus 0 <= r0 < r1 <= m; the lock takes the blocks in
 * column order (c0 equal to the columns already locked), else REALQ_ERR_SHAPE. */
int realq_quantize_block_rows(realq_ctx* ctx, double* W /*[m,n]*/, int64_t m, int64_t n, int64_t r0, int64_t r1,
                              int64_t c0, int64_t bs, const float* U /*[n,n]*/, const uint8_t* dead /*[n]|NULL*/,
                              const realq_qparams* qp, uint8_t* codes /*[m,n]*/, float* scales, uint8_t* zeros,
                              realq_bgd_state* st);
int realq_bgd_lock_block(realq_ctx* ctx, realq_bgd_state* st, int64_t c0, int64_t bs);

/* ------------------------------------------------------------------ a7-a9: one BGD step
 * One Adam step (Eq. block_gd_update) on the trailing columns W[:, c1:n] against
 *   L = (1/2T) sum_t s_t R_t^T M_a R_t,  R = W Xhat^T - W0 X^T,  M_a = alpha M + (1-alpha) P
 * (Eq. fisher_loss at the module output; Eq. slide_window for alpha).  The gradient
 * (1/T) M_a R diag(s) Xhat[:, c1:] is formed with token-streamed GEMMs.
 * loss_out (device float64 scalar, may be NULL) receives L before the update; it
 * is computed for M_a = identity only and set to NaN otherwise.  c1 == n is a no-op.
 * With increments (realq_bgd_params.resid_increment and its gate), the state keeps the
 * loss and gradient of the first step at a given c1 and up to steps - 1 later steps at the
 * same c1 start from them; realq_quantize_block(_rows) and realq_bgd_lock_block restart
 * that, as does a step at another c1 or the steps-th step after a first one. */
int realq_bgd_step(realq_ctx* ctx, realq_bgd_state* st, double* W /*[m,n]*/, int64_t c1, float alpha,
                   double* loss_out);

/* Final surrogate loss with the module's own metric (alpha = 1) at the current W,
 * written to *loss_out (device float64).  M = identity only (else REALQ_ERR_SHAPE). */
int realq_bgd_loss(realq_ctx* ctx, realq_bgd_state* st, const double* W /*[m,n]*/, double* loss_out);

/* ------------------------------------------------------------------ a10: window partner and hand-off
 * Sec. 4.4 (Eq. slide_window) blends this module's objective with the next stage's.  For a
 * linear consumer y' = W_next y of this module's output, a perturbation dy costs
 * dy^T P dy with P = W_next^T M_next W_next (M_next = NULL: identity).
 *   W_next : [m_next, m] float32;  M_next : [m_next, m_next] float32 | NULL;
 *   P      : [m, m] float32 output; accumulate != 0 adds to P (several consumers, e.g. gate and up).
 * Computed in float32. */
int realq_pullback_metric(realq_ctx* ctx, const float* W_next, const float* M_next, int64_t m_next, int64_t m,
                          int accumulate, float* P);

/* Hand-off to the next module of a layer: the inputs the next module sees.
 *   Wb == NULL : Y[t, i] = bf16( sum_j Wa[i, j] X[t, j] )                  (q -> o, o -> gate/up)
 *   Wb != NULL : Y[t, i] = bf16( silu(sum_j Wa[i,j] X[t,j]) * sum_j Wb[i,j] X[t,j] ),
 *                silu(g) = g / (1 + e^-g)                                     (gate, up -> down)
 * Wa, Wb: [m, n] float32 (quantized or original weights); X: [T, n] bf16; Y: [T, m] bf16,
 * rounded to nearest even.  Products are accumulated in float32 (weights carried as bf16
 * hi/lo pairs against the bf16 activations).  T == 0 is a no-op. */
int realq_handoff(realq_ctx* ctx, const float* Wa, const float* Wb, const uint16_t* X, int64_t T, int64_t n,
                  int64_t m, uint16_t* Y);

/* ------------------------------------------------------------------ a1-a11: whole module
 * The whole sweep for one module: Hessian over all tokens, inverse factor, then for
 * every column block realq_quantize_block followed (when steps > 0 and columns
 * remain) by `steps` realq_bgd_step calls, and the final loss.
 * Window: when window_total > 0, column block b of this module is step
 * b_global = window_offset + b + 1 of window_total and alpha follows Eq. slide_window;
 * otherwise alpha = 1.
 * Row groups: with s_groups != NULL ([n_groups, T] float32, e.g. from realq_saliency) row group g
 * (as in realq_saliency) is quantized with its own Hessian (2/T) sum_t s_groups[g, t] xhat_t xhat_t^T,
 * damping, dead columns and inverse factor (Eq. saliency_hessian, Alg. 1 Stage 1), while s keeps
 * weighting the tokens of the Block-GD surrogate; then H, U and dead of the output are
 * [n_groups, n, n] / [n_groups, n] (entries of empty groups untouched).  s_groups == NULL needs
 * n_groups == 0 (one Hessian built from s); otherwise 1 <= n_groups <= m. */
typedef struct realq_layer_desc {
    int64_t m, n, T;
    const float* W0;          /* [m,n] float32                                 */
    const uint16_t* X;        /* [T,n] bf16                                     */
    const uint16_t* Xhat;     /* [T,n] bf16                                     */
    const float* s;           /* [T] | NULL                                     */
    const float* M;           /* [m,m] | NULL (identity)                        */
    const float* P;           /* [m,m] | NULL                                   */
    int32_t window_offset, window_total;
    realq_qparams q;
    realq_bgd_params bgd;
    const float* s_groups;    /* [n_groups,T] | NULL (one Hessian from s)       */
    int32_t n_groups;         /* 0 with s_groups == NULL, else 1..m             */
} realq_layer_desc;

typedef struct realq_layer_out {
    uint8_t* codes;           /* [m,n]                     required             */
    float* scales;            /* [m,ceil(n/group)]         required             */
    uint8_t* zeros;           /* [m,ceil(n/group)]         required             */
    float* W_hat;             /* [m,n] final dequantized weights, required      */
    float* H;                 /* [n,n] float32 Hessian before damping | NULL
                                 ([n_groups,n,n] with row groups)               */
    float* U;                 /* [n,n] inverse factor | NULL (workspace used)
                                 ([n_groups,n,n] with row groups)               */
    uint8_t* dead;            /* [n] | NULL ([n_groups,n] with row groups)      */
    double* loss_trace;       /* [nblocks*steps] device float64 | NULL; entries of
                                 steps with a dense metric M_a are NaN          */
    double loss_final;        /* host: final loss with the module's own metric M
                                 (alpha = 1); with a dense M it is evaluated
                                 through the calibration Gram matrices         */
    double ms_total;          /* host: wall time of the call between events on the stream */
} realq_layer_out;

/* Synchronises the stream (after the inverse factor, and at the end to read the
 * final loss).  Returns the first error of any stage; REALQ_ERR_NONFINITE when the Hessian
 * (non-finite Xhat or s) or the final loss (non-finite W0, X, s or metric) is not finite, in
 * which case the outputs are undefined. */
int realq_quantize_layer(realq_ctx* ctx, const realq_layer_desc* desc, realq_layer_out* out);

/* ------------------------------------------------------------------ NEXT: block-output surrogate
 * Sec. 4.2-4.4 put the Block-GD surrogate at the transformer block's output (Eq. fisher_loss),
 * take its gradient through a forward and backward pass of the block, and blend in the next
 * block over the column blocks of all modules of the block (Eq. slide_window).  For the MLP
 * half of a pre-norm decoder block
 *     u = bf16(rmsnorm(h) * gamma),  z = bf16(silu(u Wg^T) * (u Wu^T)),  y = h + bf16(z Wd^T)
 * (rmsnorm(h) = h / sqrt(mean h^2 + eps); products accumulated in float32 from bf16 hi/lo
 * weights; normalisation and SwiGLU in float64 before the bf16 rounding; y float32),
 * realq_mlp_block_sweep quantizes gate, up and down in that order (Alg. 1).  Each module gets
 * GPTQ on its own input in the quantized path (u for gate and up; z with the quantized gate
 * and up for down) and, after every column block but its last, `bgd.steps` Adam steps
 * (Eq. block_gd_update) on its trailing columns against
 *     L = (1/2T) sum_t (y_t - y*_t)^T F (y_t - y*_t),
 * y* the full-precision block on X, y the partially quantized block on Xhat, the gradient
 * taken through the block with the bf16 roundings as the identity.  With window != 0 and a
 * next block, column block b_global (gate's blocks, then up's, then down's; B_total in all)
 * descends alpha L + (1 - alpha) L_next with alpha of Eq. slide_window and L_next the next
 * block's loss on y against the next block applied to y*.  Attention is not part of the block.
 *   X, Xhat   : [T, d] bf16 block inputs of the full-precision and the quantized model
 *   gamma     : [d] float32;  Wg, Wu: [f, d] float32;  Wd: [d, f] float32 (original weights)
 *   F         : [d, d] float32 symmetric Fisher at the block output, or NULL (identity)
 *   next      : the next block, same shapes; next.Wg == NULL when there is none
 *   q         : quantizer as for realq_quantize_layer (group = 0: one group per row)
 *   bgd       : steps, lr, the Adam constants and batch; form and loss_clip must be 0.
 *               With 0 < batch < T, Adam step t of a module (1-based) evaluates L (and
 *               L_next) on token batch (t - 1) mod ceil(T / batch) only, normalised by its
 *               token count (Sec. 4.3 mini-batch); loss_final is over all T tokens
 *   start_module, n_modules, W_fixed : quantize modules start_module .. start_module +
 *               n_modules - 1 only (n_modules = 0: through the last; [0, 0] is the whole
 *               block).  The modules before start_module are taken as already quantized, with
 *               W_fixed[k] their float32 quantized weights (required, copied to W_hat[k]; their
 *               codes, scales and zeros are not written); the modules after the range keep their
 *               original weights, also in loss_final.  b_global and the window's alpha count
 *               every module's column blocks, as in a whole-block sweep, so a module swept alone
 *               on the upstream modules' quantized weights follows the steps it takes in the
 *               whole sweep.  loss_trace entries of modules not swept stay NaN.
 *   X_fixed   : the start module's input in the quantized path ([T, cols] bf16: u for gate
 *               and up, z for down) taken as given instead of computed by the block from the
 *               fixed weights, or NULL.  With X_fixed and W_fixed from a reference sweep, the
 *               start module sees exactly the reference's inputs (a bf16 rounding of an
 *               activation can fall either way between two correct implementations).
 * Outputs per module (0 gate, 1 up, 2 down): codes [rows, cols] (gate, up: [f, d]; down:
 * [d, f]), scales and zeros [rows, ceil(cols/group)], W_hat [rows, cols] float32 (all
 * required); loss_trace [B_total * steps] device float64, entry (b_global - 1) * steps + k,
 * NaN for the last column block of each module, or NULL; loss_final (host) = L at the
 * quantized weights; ms_total (host).  Needs d, f >= 1, T >= 1, d and f multiples of 8.
 * Synchronises the stream (after each inverse factor and at the end). */
typedef struct realq_mlp_block {
    const float* gamma;
    const float* Wg;
    const float* Wu;
    const float* Wd;
    const float* F;
} realq_mlp_block;

typedef struct realq_mlp_desc {
    int64_t T, d, f;
    const uint16_t* X;
    const uint16_t* Xhat;
    realq_mlp_block blk;
    realq_mlp_block next;
    float eps;
    int32_t window;
    realq_qparams q;
    realq_bgd_params bgd;
    int32_t start_module, n_modules;
    const float* W_fixed[3];
    const uint16_t* X_fixed;
} realq_mlp_desc;

typedef struct realq_mlp_out {
    uint8_t* codes[3];
    float* scales[3];
    uint8_t* zeros[3];
    float* W_hat[3];
    double* loss_trace;
    double loss_final;
    double ms_total;
} realq_mlp_out;

int realq_mlp_block_sweep(realq_ctx* ctx, const realq_mlp_desc* desc, realq_mlp_out* out);

/* The full decoder block: the attention half in front of the MLP half,
 *     h1 = bf16(rmsnorm(x) * gamma1),  q/k/v = bf16(h1 W^T),  qr/kr = bf16(rope(q/k)),
 *     O = bf16(softmax_causal(qr kr^T / sqrt(hd)) v),  x2 = x + bf16(O Wo^T),
 *     then y = the MLP half of realq_mlp_block_sweep applied to x2,
 * with n_heads query heads and n_kv key/value heads of head_dim (query head h reads key/value
 * head h / (n_heads / n_kv)), the rotary embedding over pairs (i, i + hd/2) at angle
 * (t mod seq_len) rope_base^(-2i/hd) (positions counted within each sequence of seq_len
 * tokens), and causal attention within each sequence: scores as float32 sums of the exact
 * bf16 products, the softmax's maxima, sums and exponents in float64 (each exponential in
 * float32), the value sums with the probabilities in full float32 precision.  realq_decoder_block_sweep quantizes q, k, v, o, gate, up and down
 * in that order (Alg. 1), each with GPTQ on its own input in the quantized path (h1; O; u;
 * z) and Block-GD on the block-output Fisher loss as described for realq_mlp_block_sweep,
 * b_global running over the column blocks of all seven modules; the window partner is the
 * next decoder block.  Shapes: Wq [H hd, d], Wk and Wv [Hkv hd, d], Wo [d, H hd]; seq_len a
 * multiple of 32 and at most 4096, T a multiple of seq_len, H a multiple of Hkv, head_dim a
 * multiple of 32 and at most 256, d and f multiples of 8, bgd.batch a multiple of seq_len, so
 * that a mini-batch holds whole sequences (REALQ_ERR_SHAPE otherwise).  The
 * attention forward keeps the row log-sum-exp (the backward recomputes the probabilities from
 * it); its backward keeps six bf16 arrays of T n_heads seq_len entries.  Outputs per
 * module in the order q, k, v, o, gate, up, down; loss_trace entry (b_global - 1) * steps + k.
 * start_module, n_modules, W_fixed[7] and X_fixed select the modules swept as for
 * realq_mlp_desc (module indices in the order above; X_fixed is h1 for q, k and v, O for o, u
 * for gate and up, z for down). */
typedef struct realq_decoder_block {
    const float* gamma1;
    const float* Wq;
    const float* Wk;
    const float* Wv;
    const float* Wo;
    realq_mlp_block mlp;   /* gamma (the second norm), Wg, Wu, Wd, F (the block-output metric) */
} realq_decoder_block;

typedef struct realq_decoder_desc {
    int64_t T, d, f, seq_len;
    int32_t n_heads, n_kv, head_dim;
    float rope_base, eps;
    const uint16_t* X;
    const uint16_t* Xhat;
    realq_decoder_block blk;
    realq_decoder_block next;   /* next.Wq == NULL: none */
    int32_t window;
    realq_qparams q;
    realq_bgd_params bgd;
    int32_t start_module, n_modules;
    const float* W_fixed[7];
    const uint16_t* X_fixed;
} realq_decoder_desc;

typedef struct realq_decoder_out {
    uint8_t* codes[7];
    float* scales[7];
    uint8_t* zeros[7];
    float* W_hat[7];
    double* loss_trace;
    double loss_final;
    double ms_total;
} realq_decoder_out;

int realq_decoder_block_sweep(realq_ctx* ctx, const realq_decoder_desc* desc, realq_decoder_out* out);

/* One forward of the decoder block above on desc->X with desc->blk's weights (desc->Xhat, next,
 * window, q and bgd are not read): the block output y, which is the next block's input in
 * Alg. 1's block-by-block pass (run it on X with the full-precision weights and on Xhat with
 * the quantized ones), and, where the pointer is not NULL, the intermediates h1, q, k, v
 * (before the rotary embedding), O (the o projection's input) and x2, laid out as in the
 * formulas above, token-major.  All device memory owned by the caller; y is required.
 * Errors as for realq_decoder_block_sweep; the call returns after the stream has finished. */
typedef struct realq_decoder_fwd_out {
    uint16_t* h1;   /* [T, d] bf16 */
    uint16_t* q;    /* [T, n_heads head_dim] bf16 */
    uint16_t* k;    /* [T, n_kv head_dim] bf16 */
    uint16_t* v;    /* [T, n_kv head_dim] bf16 */
    uint16_t* O;    /* [T, n_heads head_dim] bf16 */
    float* x2;      /* [T, d] */
    float* y;       /* [T, d] */
} realq_decoder_fwd_out;

int realq_decoder_forward(realq_ctx* ctx, const realq_decoder_desc* desc, realq_decoder_fwd_out* out);

#ifdef __cplusplus
}
#endif
#endif /* REALQ_H */
