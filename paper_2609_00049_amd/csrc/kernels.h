// Internal launchers of the REAL-Q gfx950 library (not part of the C ABI).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace realq {

// ---------------------------------------------------------------- bf16 MFMA NT GEMM
// acc[i][j] = sum_k (Ahi[i*lda+k] + Alo[i*lda+k]) * B[j*ldb+k], i < M, j < N, k < K;
// Alo may be NULL.  splits > 1 partitions K into equal BK-aligned ranges (gridDim.z).
struct GemmArgs {
    const uint16_t* Ahi;
    const uint16_t* Alo;
    int64_t lda;
    const uint16_t* B;
    int64_t ldb;
    int64_t M, N, K;
    int64_t splits;
    int64_t group_m = 0;  // row tiles walked together per XCD (0 = chosen from the shape)
    int tile = 0;         // 0: chosen from the shape, 1: 256x256 tile, 2: 128x128 tile
    int a_blocked = 0;    // A in the blocked hi/lo layout of gemm_resid (Alo = Ahi + 32): element
                          // (i, k) at i*lda + (k/32)*64 + k%32
};
int64_t gemm_effective_splits(int64_t K, int64_t splits);
int64_t gemm_num_blocks(int64_t M, int64_t N, int tile = 0);
hipError_t gemm_store_f32(const GemmArgs& g, float* C, int64_t ldc, int64_t split_stride, float alpha, hipStream_t st);
// Split-K gradient slices C[z][i][j] = acc, always on the 256x256 tile; gemm_grad_blocks gives its tile count.
int64_t gemm_grad_blocks(int64_t M, int64_t N);
hipError_t gemm_grad(const GemmArgs& g, float* C, int64_t ldc, int64_t split_stride, hipStream_t st);
hipError_t gemm_acc_f32(const GemmArgs& g, float* C, int64_t ldc, float alpha, hipStream_t st);
hipError_t gemm_acc_f64(const GemmArgs& g, double* C, int64_t ldc, hipStream_t st);
// Residual R = B0 + acc with split(R o s) stored either as two arrays Rhi/Rlo [i*ldr + t]
// (blocked = false) or in one array of 128-byte lines holding 32 tokens' hi then their lo
// (blocked = true: hi at Rhi[i*ldr + (t/32)*64 + t%32], lo 32 further, ldr a multiple of 64;
// Rlo unused), the A layout of a_blocked gradient launches.
hipError_t gemm_resid(const GemmArgs& g, const float* B0, int64_t ldb0, const float* s, uint16_t* Rhi, uint16_t* Rlo,
                      int64_t ldr, double* partials, hipStream_t st, bool blocked = false);
// Later step of a column block (A = the weight change since its first step): Q = bf16(acc * s_t)
// [i*ldq + t] and partial sums of s_t acc^2.
hipError_t gemm_resid_inc(const GemmArgs& g, const float* s, uint16_t* Q, int64_t ldq, double* partials,
                          hipStream_t st);
hipError_t gemm_loss(const GemmArgs& g, const float* B0, int64_t ldb0, const float* s, double* partials,
                     hipStream_t st);
// Token-major stores for the module hand-off: out[j*ld + i] = bf16(acc[i][j] + add[j*ld + i]);
// float32 variant (add may be NULL, and for the float32 variant equal to out);
// SwiGLU variant out[j*ld + i] = bf16(silu(G[j*ldg + i]) * acc[i][j]).
hipError_t gemm_store_bf16_t(const GemmArgs& g, uint16_t* out, int64_t ld, hipStream_t st, const float* add = nullptr);
hipError_t gemm_store_f32_t(const GemmArgs& g, float* out, int64_t ld, hipStream_t st, const float* add = nullptr);
hipError_t gemm_swiglu_t(const GemmArgs& g, const float* G, int64_t ldg, uint16_t* out, int64_t ld, hipStream_t st);
// out[c*ldo + r] = in[r*ldi + c] (float32)
hipError_t transpose_f32(const float* in, int64_t ldi, float* out, int64_t ldo, int64_t rows, int64_t cols,
                         hipStream_t st);

// ---------------------------------------------------------------- elementwise / layout
hipError_t fill_f32(float* p, float v, int64_t count, hipStream_t st);
hipError_t fill_f64(double* p, double v, int64_t count, hipStream_t st);
hipError_t fill_u16(uint16_t* p, uint16_t v, int64_t count, hipStream_t st);
// out[c*ldo + r] = in[r*ldi + c] for r < rows, c < cols (bf16 bit patterns)
hipError_t transpose_u16(const uint16_t* in, int64_t ldi, uint16_t* out, int64_t ldo, int64_t rows, int64_t cols,
                         hipStream_t st);
// Transposed, weighted split: hi/lo[c*ldo + r] = split(s[r] * bf16(in[r*ldi + c]))   (s may be NULL);
// lo2 (may be NULL) receives the bf16 of the float32 remainder, so hi + lo + lo2 is the product.
hipError_t transpose_scale_split(const uint16_t* in, int64_t ldi, const float* s, uint16_t* hi, uint16_t* lo,
                                 uint16_t* lo2, int64_t ldo, int64_t rows, int64_t cols, hipStream_t st);
// hi/lo[i*ld + j] = split(A[i*lda + j] - (Bm ? Bm[i*ldb + j] : 0)) for j < cols (float32 inputs)
hipError_t split_diff_f32(const float* A, int64_t lda, const float* Bm, int64_t ldb, uint16_t* hi, uint16_t* lo,
                          int64_t ld, int64_t rows, int64_t cols, hipStream_t st);
// hi/lo[i*ld + j] = split(float(A[i*lda + j] - Bm[i*ldb + j])) for j < cols (float64 A, float32 Bm)
hipError_t split_diff_f64(const double* A, int64_t lda, const float* Bm, int64_t ldb, uint16_t* hi, uint16_t* lo,
                          int64_t ld, int64_t rows, int64_t cols, hipStream_t st);
// Transposed input perturbation of a token chunk: delta = bf16(Xh) - bf16(X) ([rows = tokens,
// cols]); sdh/sdl = split(s[r] * delta), dh/dl = split(delta), all written as [cols][ldo].
hipError_t transpose_delta_split(const uint16_t* Xh, const uint16_t* X, int64_t ldi, const float* s, uint16_t* sdh,
                                 uint16_t* sdl, uint16_t* dh, uint16_t* dl, int64_t ldo, int64_t rows, int64_t cols,
                                 hipStream_t st);
// hi/lo = split(float(in))
hipError_t split_f64(const double* in, uint16_t* hi, uint16_t* lo, int64_t count, hipStream_t st);
// Three-term splits that carry all 24 bits of a float32: hi = bf16(x), lo = bf16(x - hi),
// lo2 = bf16(x - hi - lo), so hi + lo + lo2 equals x to float32 precision (x = float(in) for the
// float64 input).
hipError_t split3_f64(const double* in, uint16_t* hi, uint16_t* lo, uint16_t* lo2, int64_t count, hipStream_t st);
hipError_t split3_f32(const float* A, int64_t lda, uint16_t* hi, uint16_t* lo, uint16_t* lo2, int64_t ld,
                      int64_t rows, int64_t cols, hipStream_t st);
// *flag |= 1 when any of p[0 .. count) is a nonzero bf16 value (the caller clears *flag)
hipError_t any_nonzero_u16(const uint16_t* p, int64_t count, int* flag, hipStream_t st);
// G[i][j] = C0[i][c1+j] + P[i][c1+j], i < m, j < w
hipError_t gram_grad(const float* C0, const float* P, int64_t ld, int64_t c1, int64_t m, int64_t w, float* G,
                     hipStream_t st);
// partials = fixed-order partial sums of (2 C0 + P) (W - W0) over count elements
hipError_t dot_gram(const float* C0, const float* P, const double* W, const float* W0, int64_t count,
                    double* partials, hipStream_t st);
// out = A - double(B)
hipError_t sub_f64_f32(const double* A, const float* B, double* out, int64_t count, hipStream_t st);
// partials[0 .. dot_f64_partials()) = fixed-order partial sums of X . Y
hipError_t dot_f64(const double* X, const double* Y, int64_t count, double* partials, hipStream_t st);
int64_t dot_f64_partials();
// out[i] = double(in[i]) / float(in[i])
hipError_t widen_f32(const float* in, double* out, int64_t count, hipStream_t st);
hipError_t narrow_f64(const double* in, float* out, int64_t count, hipStream_t st);
// hi/lo[i] = split(bf16(a[i]) - bf16(b[i]))
hipError_t split_diff_bf16(const uint16_t* a, const uint16_t* b, uint16_t* hi, uint16_t* lo, int64_t count,
                           hipStream_t st);
// hi/lo[i*m + k] = split(alpha (M ? M : I)[i][k] + (1 - alpha) (P ? P[i][k] : 0)), m x m float32 inputs
hipError_t blend_split(const float* M, const float* P, float alpha, int64_t m, uint16_t* hi, uint16_t* lo,
                       hipStream_t st);
// out = sum of partials (fixed order) * scale, written to *out (device)
hipError_t reduce_partials(const double* partials, int64_t count, double scale, double* out, hipStream_t st);
// Adam on W[:, c1:n] with G = gscale * sum_z Gp[z][i][j - c1]; refreshes Dhi/Dlo = split(W - W0) there
// (skipped when Dhi is NULL).  With Dacc, the block's weight change since its first step is kept
// too: Dacc = (reset ? 0 : Dacc) + the step (float32), Dinc = bf16(Dacc).
struct AdamArgs {
    double* W;
    const float* W0;
    float* mA;
    float* vA;
    uint16_t* Dhi;
    uint16_t* Dlo;
    int64_t m, n, c1;
    const float* Gp;  // [splits][m][n - c1]
    int64_t splits;
    float gscale, lr, beta1, beta2, eps, bc1, bc2;  // bc1 = 1/(1-beta1^t), bc2 = 1/(1-beta2^t)
    float* Dacc = nullptr;     // [m, n]
    uint16_t* Dinc = nullptr;  // [m, n]
    int inc_reset = 0;
    // the block's first gradient, [m][n - c1], unscaled: g0_mode 1 stores sum_z Gp there,
    // 2 adds it to sum_z Gp (later steps, whose Gp holds the change only)
    float* G0 = nullptr;
    int g0_mode = 0;
};
hipError_t adam_update(const AdamArgs& a, hipStream_t st);
// Loss of a later step of a column block from the block's first loss L0 and first gradient sum
// G0 [m][w] (unscaled, over the T tokens), the bf16 weight change Dinc [i*ldd + j] and the partial
// sums of s_t acc^2: *out = *L0 + <G0, Dinc> / T + 0.5 / T * sum(parts).  dots: inc_loss_partials()
// doubles of workspace.
hipError_t inc_loss(const double* L0, const float* G0, const uint16_t* Dinc, int64_t ldd, int64_t m, int64_t w,
                    const double* parts, int64_t nparts, double T, double* dots, double* out, hipStream_t st);
int64_t inc_loss_partials();
// G[i][j] = (accumulate ? G[i][j] : 0) + gscale * sum_z Gp[z][i][j]  (m x w), z in order
hipError_t reduce_splits(const float* Gp, int64_t splits, int64_t m, int64_t w, float gscale, float* G,
                         bool accumulate, hipStream_t st);
// Adam with a ready gradient G (m x (n-c1)).
hipError_t adam_update_dense(const AdamArgs& a, const float* G, hipStream_t st);

// ---------------------------------------------------------------- fp32 GEMM (VALU): C = beta*C + alpha*A*B
// A [M,K] lda, B [K,N] ldb, C [M,N] ldc, all float32 row-major.
struct SgemmArgs {
    const float* A;
    int64_t lda;
    const float* B;
    int64_t ldb;
    float* C;
    int64_t ldc;
    int64_t M, N, K;
    float alpha, beta;
};
hipError_t sgemm(const SgemmArgs& a, hipStream_t st);
// float64 VALU GEMM: C = A B (accumulate = false) or C += A B; A [M,K] lda, B [K,N] ldb,
// C [M,N] ldc, all float64 row-major.
hipError_t dgemm(const double* A, int64_t lda, const double* B, int64_t ldb, double* C, int64_t ldc, int64_t M,
                 int64_t N, int64_t K, bool accumulate, hipStream_t st);

// ---------------------------------------------------------------- output-perturbation clip
// tau[t] = k-th smallest |R[i][t]| over i < m (t < cur, R row stride ldr), 1 <= k <= m
hipError_t clip_select(const float* R, int64_t ldr, int64_t m, int64_t cur, int64_t k, float* tau, hipStream_t st);
// c = min(1, tau_t / |R|): Rhi/Rlo = split(c^2 s_t R), partials[0 .. clip_apply_partials()) =
// fixed-order partial sums of s_t (c R)^2
hipError_t clip_apply(const float* R, int64_t ldr, int64_t m, int64_t cur, const float* tau, const float* s,
                      uint16_t* Rhi, uint16_t* Rlo, double* partials, hipStream_t st);
int64_t clip_apply_partials();
// R[i][t] = B0[i][t] + (split(D) Xhat^T)[i][t] in float32 (the residual kept whole for the clip)
hipError_t gemm_resid_f32(const GemmArgs& g, const float* B0, int64_t ldb0, float* R, int64_t ldr, hipStream_t st);

// ---------------------------------------------------------------- Stage-0 accumulators
// Row group g = channels [g r, min(m, (g+1) r)), r = ceil(m / n_groups).  s64 [n_groups][T]
// (work) = float64 sums of G[t][i]^2 over the group's channels; k > 0: tau[g] = k-th smallest
// of group g's row (nearest rank, 1 <= k <= T) and out = float(min(s64, tau)); k == 0: out =
// float(s64).  Rows of empty groups (g r >= m) are written as zeros.  sel: work of
// saliency_select_bytes(n_groups) bytes (8-byte aligned).
hipError_t saliency(const uint16_t* G, int64_t T, int64_t m, int64_t n_groups, int64_t k, double* s64, double* tau,
                    void* sel, float* out, hipStream_t st);
int64_t saliency_select_bytes(int64_t n_groups);
// out[e] = float(a[e] / d)
hipError_t div_narrow(const double* a, double d, float* out, int64_t count, hipStream_t st);

// ---------------------------------------------------------------- block-output surrogate (MLP block)
// u[t, :] = bf16(h[t, :] gamma / sqrt(mean h[t, :]^2 + eps)) (statistics in float64)
hipError_t rmsnorm_bf16(const uint16_t* h, int64_t T, int64_t d, const float* gamma, double eps, uint16_t* u,
                        hipStream_t st);
hipError_t rmsnorm_f32(const float* h, int64_t T, int64_t d, const float* gamma, double eps, uint16_t* u,
                       hipStream_t st);
// z = bf16(silu(a) b) elementwise
hipError_t swiglu_fwd(const float* a, const float* b, uint16_t* z, int64_t count, hipStream_t st);
// y = h + out, dy = y - ystar (y, dy may be NULL)
hipError_t residual_out_bf16(const uint16_t* h, const uint16_t* out, const float* ystar, float* y, float* dy,
                             int64_t count, hipStream_t st);
hipError_t residual_out_f32(const float* h, const uint16_t* out, const float* ystar, float* y, float* dy,
                            int64_t count, hipStream_t st);
// out = s x (out may be NULL), hi/lo = split(s x) (may be NULL)
hipError_t scale_split(const float* x, float s, float* out, uint16_t* hi, uint16_t* lo, int64_t count,
                       hipStream_t st);
// partials[0 .. dot_f32_partials()) = scale * fixed-order partial sums of x . y
hipError_t dot_f32(const float* x, const float* y, int64_t count, double scale, double* partials, hipStream_t st);
int64_t dot_f32_partials();
// SwiGLU backward to the gate (which 0) or up (which 1) input from dz [T, f], split to hi/lo,
// transposed ([f][ldo]) or row-major ([T][ldo])
hipError_t swiglu_bwd(const float* dz, const float* a, const float* b, int which, int64_t T, int64_t f,
                      int transposed, uint16_t* hi, uint16_t* lo, int64_t ldo, hipStream_t st);
// Both row-major outputs (gate: hi0/lo0, up: hi1/lo1) of swiglu_bwd in one pass over dz, a, b.
hipError_t swiglu_bwd_pair(const float* dz, const float* a, const float* b, int64_t T, int64_t f, uint16_t* hi0,
                           uint16_t* lo0, uint16_t* hi1, uint16_t* lo1, int64_t ldo, hipStream_t st);
// hi/lo[c * ldo + r] = split(in[r * ldi + c])
hipError_t transpose_split_f32(const float* in, int64_t ldi, uint16_t* hi, uint16_t* lo, int64_t ldo, int64_t rows,
                               int64_t cols, hipStream_t st);
// g = alpha g + (1 - alpha) (g2 + RMSNorm backward of du at h); alpha == 0 does not read g
hipError_t rmsnorm_bwd_blend(const float* h, const float* g2, const float* du, const float* gamma, double eps,
                             double alpha, int64_t T, int64_t d, float* g, hipStream_t st);

// ---------------------------------------------------------------- attention half of a decoder block
// rotary embedding: forward on bf16 [T][n hd] (rounded), inverse rotation on float32 (backward),
// with the cos/sin table cs [L][hd/2][2] (float64) that rope_table fills for (L, hd, base)
hipError_t rope_table(double* cs, int64_t L, int64_t hd, double base, hipStream_t st);
hipError_t rope_fwd(const uint16_t* in, uint16_t* out, const double* cs, int64_t T, int64_t n, int64_t hd, int64_t L,
                    hipStream_t st);
hipError_t rope_inv(const float* in, float* out, const double* cs, int64_t T, int64_t n, int64_t hd, int64_t L,
                    hipStream_t st);
// Causal attention per sequence of L tokens (L and hd multiples of 32): O32 = softmax(qr kr^T /
// sqrt(hd)) v [T][H hd] float32, O = bf16(O32), LSE [T][H] the row log-sum-exp (float64) that the
// backward recomputes the probabilities from; vt receives v^T [Hkv hd][T].
hipError_t attn_fwd(const uint16_t* qr, const uint16_t* kr, const uint16_t* v, int64_t T, int64_t H, int64_t Hkv,
                    int64_t hd, int64_t L, double* LSE, float* O32, uint16_t* O, uint16_t* vt, hipStream_t st);
// Scratch of the attention backward: D [T][H] float64; dS, dS^T and P^T as bf16 hi/lo pairs,
// each [T/L][H][L][L]; kr^T [Hkv hd][T], qr^T [H hd][T], dO^T hi/lo [H hd][T]; partial dK/dV.
struct AttnScratch {
    double* D;
    uint16_t *dSh, *dSl, *dSth, *dStl, *Pth, *Ptl;
    uint16_t *kt, *qt, *dOth, *dOtl;
    float* part;  // [attn_dkv_chunks(L)][2][T][Hkv hd] partial dK/dV sums
};
// number of query-tile chunks whose partial dK/dV sums the backward keeps
int64_t attn_dkv_chunks(int64_t L);
// From dO [T][H hd] float32 and the forward's LSE and O32: dq [T][H hd] (gradient at the rotated
// queries), dk [T][Hkv hd] (at the rotated keys) and dv [T][Hkv hd], float32.
hipError_t attn_bwd(const double* LSE, const float* O32, const float* dO, const uint16_t* qr, const uint16_t* kr,
                    const uint16_t* v, int64_t T, int64_t H, int64_t Hkv, int64_t hd, int64_t L, const AttnScratch& w,
                    float* dq, float* dk, float* dv, hipStream_t st);

// ---------------------------------------------------------------- quantize one column block
struct QuantArgs {
    double* W;
    int64_t m, n, c0, bs;
    const float* U;
    const uint8_t* dead;
    int bits, group, grid;
    int sym;  // symmetric range, zero fixed at (maxq + 1) / 2
    uint8_t* codes;
    float* scales;
    uint8_t* zeros;
    int64_t ngroups;
    double* E;  // [m][bs]
    const float* W0;  // may be NULL (no split written)
    uint16_t* Dhi;
    uint16_t* Dlo;
};
hipError_t quantize_block(const QuantArgs& q, hipStream_t st);
// W[i][j] -= sum_k E[i][k] U[k][j] in float64 (M x N, K <= block width); when Dhi != NULL
// also Dhi/Dlo[i*ldd + j] = split(W[i][j] - W0[i*ldw0 + j]).
struct ObsArgs {
    const double* E;
    int64_t lde;
    const float* U;
    int64_t ldu;
    double* W;
    int64_t ldw;
    int64_t M, N, K;
    const float* W0;
    int64_t ldw0;
    uint16_t* Dhi;
    uint16_t* Dlo;
    int64_t ldd;
};
hipError_t obs_update(const ObsArgs& a, hipStream_t st);

// ---------------------------------------------------------------- float64 factorisation
// Prepares A = J (H + lambda I) J (index-reversed, padded to np with identity) from H_acc,
// writes H_out and dead; lambda computed on device.  Then Cholesky + triangular inverse.
struct CholArgs {
    const double* Hacc;
    int64_t n, np;
    double scale;  // 2 / T_total
    double damp;
    float* Hout;
    uint8_t* dead;
    double* A;     // [np][np] work (becomes L, lower)
    double* Linv;  // [np][np] work
    double* diaginv;  // [np/64][64][64]
    double* tmp;   // [64][np]
    int* flag;     // device int: 0 ok, 1 not SPD
    double* scratch;  // small: >= 8 doubles
    float* U;      // [n][n] output
};
hipError_t chol_inverse(const CholArgs& c, hipStream_t st);

}  // namespace realq
