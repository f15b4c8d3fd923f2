// Inverse factor of the damped Hessian in float64 (Sec. 3.2; Alg. 1 "its inverse").
//
// GPTQ's compensation for column j uses row j of the inverse of H restricted to the
// columns not yet quantized.  Those rows, scaled, are the rows of the upper factor U
// with H_d^{-1} = U^T U.  With J the index reversal, A = J H_d J = L L^T (lower
// Cholesky) gives H_d^{-1} = (J L^{-1} J)^T (J L^{-1} J), so U = J L^{-1} J.
//
// Steps (all float64):
//   prep     H = scale * H_acc; dead columns (H_jj == 0) get H_jj = 1; lambda = damp * mean(diag);
//            A = J (H + lambda I) J, padded to a multiple of 64 with identity.
//   Cholesky right-looking, 64-wide panels: factor the diagonal block in one
//            workgroup (and invert it), triangular-solve the panel below, update the
//            trailing lower triangle.
//   inverse  X = L^{-1} by recursive doubling: with the aligned diagonal blocks of size s already
//            inverted (s = 64: the diagonal factor's own inverses), each aligned block of size 2s
//            [[L_A, 0], [L_CA, L_C]] gets its lower-left block X_CA = -X_C (L_CA X_A), two batched
//            float64 tile products per level that skip the tiles where a triangular operand is
//            zero; the intermediate L_CA X_A is parked, transposed, in the unused upper triangle of
//            the factor's work array.
//   U        U[i][j] = X[n-1-i][n-1-j] (j >= i), stored as float32.
#include "common.h"
#include "kernels.h"

namespace realq {

namespace {
constexpr int NB = 64;

// 256 threads; thread (ty, tx) owns rows ty*4..+3 and columns tx*4..+3 of a 64x64 tile.
// acc += A * B^T   (A, B in LDS, [64][NB+1])
__device__ __forceinline__ void tile_mac_nt(double (&acc)[4][4], const double (*sa)[NB + 1],
                                            const double (*sb)[NB + 1]) {
    const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
    for (int k = 0; k < NB; ++k) {
        double a[4], b[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) a[i] = sa[ty * 4 + i][k];
#pragma unroll
        for (int j = 0; j < 4; ++j) b[j] = sb[tx * 4 + j][k];
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j) acc[i][j] = fma(a[i], b[j], acc[i][j]);
    }
}
// acc += A * B   (B indexed [k][col])
__device__ __forceinline__ void tile_mac_nn(double (&acc)[4][4], const double (*sa)[NB + 1],
                                            const double (*sb)[NB + 1]) {
    const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
    for (int k = 0; k < NB; ++k) {
        double a[4], b[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) a[i] = sa[ty * 4 + i][k];
#pragma unroll
        for (int j = 0; j < 4; ++j) b[j] = sb[k][tx * 4 + j];
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j) acc[i][j] = fma(a[i], b[j], acc[i][j]);
    }
}
__device__ __forceinline__ void load_tile(double (*s)[NB + 1], const double* g, int64_t ld) {
    for (int e = threadIdx.x; e < NB * NB; e += 256) s[e / NB][e % NB] = g[(e / NB) * ld + (e % NB)];
}
__device__ __forceinline__ void zero_acc(double (&acc)[4][4]) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = 0.0;
}
}  // namespace

// ---------------------------------------------------------------- prep
// scratch[0] = lambda.  One block: deterministic mean of the fixed diagonal.
__global__ __launch_bounds__(256) void chol_diag_kernel(const double* __restrict__ Hacc, int64_t n, double scale,
                                                        double damp, uint8_t* dead, double* scratch) {
    __shared__ double red[256];
    double acc = 0.0;
    for (int64_t j = threadIdx.x; j < n; j += 256) {
        double d = scale * Hacc[j * n + j];
        bool dd = d == 0.0;
        if (dead) dead[j] = dd ? 1 : 0;
        acc += dd ? 1.0 : d;
    }
    red[threadIdx.x] = acc;
    __syncthreads();
    for (int s = 128; s > 0; s >>= 1) {
        if (threadIdx.x < s) red[threadIdx.x] += red[threadIdx.x + s];
        __syncthreads();
    }
    if (threadIdx.x == 0) scratch[0] = damp * (red[0] / (double)n);
}

// A = the index-reversed damped Hessian (padded with the identity); nonfinite[0] = 1 when an entry
// of the accumulator is NaN or infinite (a non-finite input reached the Hessian).
__global__ void chol_fill_kernel(const double* __restrict__ Hacc, int64_t n, int64_t np, double scale,
                                 const double* __restrict__ scratch, double* __restrict__ A, float* Hout,
                                 int* nonfinite) {
    const double lam = scratch[0];
    const int64_t total = np * np;
    for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < total; e += (int64_t)gridDim.x * blockDim.x) {
        const int64_t r = e / np, c = e % np;
        double v;
        if (r < n && c < n) {
            const int64_t hr = n - 1 - r, hc = n - 1 - c;
            double h = scale * Hacc[hr * n + hc];
            if (!isfinite(h)) *nonfinite = 1;
            if (Hout) Hout[hr * n + hc] = (float)h;
            if (hr == hc) v = (h == 0.0 ? 1.0 : h) + lam;
            else v = h;
        } else {
            v = (r == c) ? 1.0 : 0.0;
        }
        A[e] = v;
    }
}

// ---------------------------------------------------------------- diagonal block: factor + invert
__global__ __launch_bounds__(256) void chol_potrf_kernel(double* A, int64_t np, int64_t k0, double* diaginv,
                                                         double* X, int* flag) {
    __shared__ double T[NB][NB + 1];
    __shared__ double V[NB][NB + 1];
    double* Ad = A + k0 * np + k0;
    load_tile(T, Ad, np);
    __syncthreads();
    for (int k = 0; k < NB; ++k) {
        if (threadIdx.x == 0) {
            double d = T[k][k];
            if (!(d > 0.0)) {  // not positive definite (or NaN): flag it and keep values finite
                *flag = 1;
                d = 1.0;
            }
            T[k][k] = sqrt(d);
        }
        __syncthreads();
        const double piv = T[k][k];
        for (int i = k + 1 + threadIdx.x; i < NB; i += 256) T[i][k] /= piv;
        __syncthreads();
        const int rem = NB - k - 1;
        for (int e = threadIdx.x; e < rem * rem; e += 256) {
            const int i = k + 1 + e / rem, j = k + 1 + e % rem;
            if (j <= i) T[i][j] -= T[i][k] * T[j][k];
        }
        __syncthreads();
    }
    // inverse of the lower factor, one column per thread (forward substitution)
    if (threadIdx.x < NB) {
        const int c = threadIdx.x;
        for (int i = 0; i < NB; ++i) V[i][c] = 0.0;
        V[c][c] = 1.0 / T[c][c];
        for (int i = c + 1; i < NB; ++i) {
            double s = 0.0;
            for (int k = c; k < i; ++k) s = fma(T[i][k], V[k][c], s);
            V[i][c] = -s / T[i][i];
        }
    }
    __syncthreads();
    double* D = diaginv + (k0 / NB) * NB * NB;
    double* Xd = X + k0 * np + k0;
    for (int e = threadIdx.x; e < NB * NB; e += 256) {
        const int i = e / NB, j = e % NB;
        Ad[i * np + j] = (j <= i) ? T[i][j] : 0.0;
        D[e] = V[i][j];
        Xd[i * np + j] = V[i][j];
    }
}

// ---------------------------------------------------------------- panel solve: L21 = A21 L_kk^{-T}
__global__ __launch_bounds__(256) void chol_trsm_kernel(double* A, int64_t np, int64_t k0,
                                                        const double* __restrict__ diaginv) {
    __shared__ double sa[NB][NB + 1];
    __shared__ double sl[NB][NB + 1];
    const int64_t r0 = k0 + NB + (int64_t)blockIdx.x * NB;
    double* P = A + r0 * np + k0;
    load_tile(sa, P, np);
    load_tile(sl, diaginv + (k0 / NB) * NB * NB, NB);
    __syncthreads();
    double acc[4][4];
    zero_acc(acc);
    tile_mac_nt(acc, sa, sl);
    const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) P[(ty * 4 + i) * np + tx * 4 + j] = acc[i][j];
}

// ---------------------------------------------------------------- trailing update: A22 -= L21 L21^T (lower tiles)
__global__ __launch_bounds__(256) void chol_syrk_kernel(double* A, int64_t np, int64_t k0) {
    __shared__ double sa[NB][NB + 1];
    __shared__ double sb[NB][NB + 1];
    const int64_t t = blockIdx.x;
    int64_t ti = (int64_t)((sqrt(8.0 * (double)t + 1.0) - 1.0) * 0.5);
    while ((ti + 1) * (ti + 2) / 2 <= t) ++ti;
    while (ti * (ti + 1) / 2 > t) --ti;
    const int64_t tj = t - ti * (ti + 1) / 2;
    const int64_t base = k0 + NB;
    const int64_t ri = base + ti * NB, rj = base + tj * NB;
    load_tile(sa, A + ri * np + k0, np);
    load_tile(sb, A + rj * np + k0, np);
    __syncthreads();
    double acc[4][4];
    zero_acc(acc);
    tile_mac_nt(acc, sa, sb);
    const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
    double* C = A + ri * np + rj;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) C[(ty * 4 + i) * np + tx * 4 + j] -= acc[i][j];
}

// ---------------------------------------------------------------- triangular inverse, one doubling level
// C (M x N) = alpha * A (M x K) * B (K x N) for every pair p of the level, all dimensions multiples
// of 64.  Element (i, k) of A sits at A[i * lda + k] (A_KC) or A[i + k * lda]; element (k, j) of B at
// B[k + j * ldb] (B_KC) or B[k * ldb + j]; element (i, j) of C at C[i * ldc + j] (C_ROW) or
// C[i + j * ldc].  Pair p offsets every base by p * 2s (1 + ld) and has M_p = min(s, np - p*2s - s)
// rows.  TRI_B: B is lower triangular, so output column tile jt needs k >= 64 jt; TRI_A: A is lower
// triangular, so row tile it needs k < 64 (it + 1).  A 64 x 64 output tile per block, 4 x 4 per
// thread, K in slices of 16 through two LDS buffers.
namespace {
constexpr int KS = 16;
constexpr int SP = 64 + 2;  // padded LDS row: 16-byte aligned, transposed stores spread over banks

// one 64 x 16 operand slice: outer index o (row of A, column of B) and k.  KC: consecutive k adjacent.
template <bool KC>
__device__ __forceinline__ void slice_load(double (&r)[4], const double* __restrict__ p, int64_t ld) {
    const int t = threadIdx.x;
    if constexpr (KC) {
        const double2* q = reinterpret_cast<const double2*>(p + (int64_t)(t >> 2) * ld + (t & 3) * 4);
        const double2 u = q[0], v = q[1];
        r[0] = u.x; r[1] = u.y; r[2] = v.x; r[3] = v.y;
    } else {
        const double2* q = reinterpret_cast<const double2*>(p + (int64_t)(t >> 4) * ld + (t & 15) * 4);
        const double2 u = q[0], v = q[1];
        r[0] = u.x; r[1] = u.y; r[2] = v.x; r[3] = v.y;
    }
}
template <bool KC>
__device__ __forceinline__ void slice_store(double (*sx)[SP], const double (&r)[4]) {
    const int t = threadIdx.x;
    if constexpr (KC) {
#pragma unroll
        for (int q = 0; q < 4; ++q) sx[(t & 3) * 4 + q][t >> 2] = r[q];
    } else {
        double2* d = reinterpret_cast<double2*>(&sx[t >> 4][(t & 15) * 4]);
        d[0] = make_double2(r[0], r[1]);
        d[1] = make_double2(r[2], r[3]);
    }
}
}  // namespace

template <bool A_KC, bool B_KC, bool C_ROW, bool TRI_A, bool TRI_B>
__global__ __launch_bounds__(256) void chol_pair_gemm_kernel(const double* __restrict__ A, int64_t lda,
                                                             const double* __restrict__ B, int64_t ldb,
                                                             double* __restrict__ C, int64_t ldc, int64_t np,
                                                             int64_t s, int64_t N, int64_t Kfull, bool k_is_m,
                                                             double alpha) {
    __shared__ __attribute__((aligned(16))) double sa[2][KS][SP];
    __shared__ __attribute__((aligned(16))) double sb[2][KS][SP];
    const int64_t p = blockIdx.z;
    const int64_t off = p * 2 * s;
    const int64_t Mp = np - off - s < s ? np - off - s : s;  // rows of this pair's C block
    const int64_t it = blockIdx.y, jt = blockIdx.x;
    if (it * 64 >= Mp || jt * 64 >= N) return;
    const int64_t K = k_is_m ? Mp : Kfull;
    int64_t k_lo = 0, k_hi = K;
    if constexpr (TRI_B) k_lo = jt * 64;
    if constexpr (TRI_A) k_hi = (it + 1) * 64 < K ? (it + 1) * 64 : K;
    const double* Ap = A + off * (lda + 1) + (A_KC ? it * 64 * lda : it * 64);
    const double* Bp = B + off * (ldb + 1) + (B_KC ? jt * 64 * ldb : jt * 64);
    auto a_at = [&](int64_t k) { return A_KC ? Ap + k : Ap + k * lda; };
    auto b_at = [&](int64_t k) { return B_KC ? Bp + k : Bp + k * ldb; };
    const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
    double acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = 0.0;
    double ra[4], rb[4];
    if (k_lo < k_hi) {
        slice_load<A_KC>(ra, a_at(k_lo), lda);
        slice_load<B_KC>(rb, b_at(k_lo), ldb);
        slice_store<A_KC>(sa[0], ra);
        slice_store<B_KC>(sb[0], rb);
    }
    __syncthreads();
    int cur = 0;
    for (int64_t k = k_lo; k < k_hi; k += KS) {
        const bool more = k + KS < k_hi;
        if (more) {
            slice_load<A_KC>(ra, a_at(k + KS), lda);
            slice_load<B_KC>(rb, b_at(k + KS), ldb);
        }
#pragma unroll 4
        for (int kk = 0; kk < KS; ++kk) {
            const double2* pa = reinterpret_cast<const double2*>(&sa[cur][kk][ty * 4]);
            const double2* pb = reinterpret_cast<const double2*>(&sb[cur][kk][tx * 4]);
            const double2 a01 = pa[0], a23 = pa[1], b01 = pb[0], b23 = pb[1];
            const double a[4] = {a01.x, a01.y, a23.x, a23.y};
            const double b[4] = {b01.x, b01.y, b23.x, b23.y};
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) acc[i][j] = fma(a[i], b[j], acc[i][j]);
        }
        if (more) {
            slice_store<A_KC>(sa[cur ^ 1], ra);
            slice_store<B_KC>(sb[cur ^ 1], rb);
        }
        __syncthreads();
        cur ^= 1;
    }
    double* Cp = C + off * (ldc + 1);
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int64_t r = it * 64 + ty * 4 + i, c = jt * 64 + tx * 4 + j;
            Cp[C_ROW ? r * ldc + c : r + c * ldc] = alpha * acc[i][j];
        }
}

__global__ void chol_extract_u_kernel(const double* __restrict__ X, int64_t np, int64_t n, float* __restrict__ U) {
    const int64_t total = n * n;
    for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < total; e += (int64_t)gridDim.x * blockDim.x) {
        const int64_t i = e / n, j = e % n;
        U[e] = (j >= i) ? (float)X[(n - 1 - i) * np + (n - 1 - j)] : 0.f;
    }
}

__global__ void chol_zero_kernel(double* p, int64_t count) {
    for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < count; e += (int64_t)gridDim.x * blockDim.x)
        p[e] = 0.0;
}

hipError_t chol_inverse(const CholArgs& c, hipStream_t st) {
    const int64_t n = c.n, np = c.np;
    const int64_t nb = np / NB;
    auto grid_of = [](int64_t count) {
        int64_t b = (count + 255) / 256;
        return (unsigned)(b < 1 ? 1 : (b > 65536 ? 65536 : b));
    };
    hipLaunchKernelGGL(chol_diag_kernel, dim3(1), dim3(256), 0, st, c.Hacc, n, c.scale, c.damp, c.dead, c.scratch);
    hipLaunchKernelGGL(chol_fill_kernel, dim3(grid_of(np * np)), dim3(256), 0, st, c.Hacc, n, np, c.scale, c.scratch,
                       c.A, c.Hout, c.flag + 1);
    hipLaunchKernelGGL(chol_zero_kernel, dim3(grid_of(np * np)), dim3(256), 0, st, c.Linv, np * np);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    for (int64_t kb = 0; kb < nb; ++kb) {
        const int64_t k0 = kb * NB;
        hipLaunchKernelGGL(chol_potrf_kernel, dim3(1), dim3(256), 0, st, c.A, np, k0, c.diaginv, c.Linv, c.flag);
        const int64_t rem = nb - kb - 1;
        if (rem > 0) {
            hipLaunchKernelGGL(chol_trsm_kernel, dim3((unsigned)rem), dim3(256), 0, st, c.A, np, k0, c.diaginv);
            hipLaunchKernelGGL(chol_syrk_kernel, dim3((unsigned)(rem * (rem + 1) / 2)), dim3(256), 0, st, c.A, np,
                               k0);
        }
        e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    // X = L^{-1}: the diagonal 64-blocks came out of the factorisation; level s completes every
    // aligned 2s block (the last one cut at np) from its two inverted halves
    for (int64_t sz = NB; sz < np; sz *= 2) {
        const unsigned t = (unsigned)(sz / NB);
        const unsigned pairs = (unsigned)((np - sz + 2 * sz - 1) / (2 * sz));
        // T1 = L_CA X_A, stored transposed above the diagonal of the factor's array
        hipLaunchKernelGGL((chol_pair_gemm_kernel<true, false, false, false, true>), dim3(t, t, pairs), dim3(256), 0,
                           st, c.A + sz * np, np, c.Linv, np, c.A + sz, np, np, sz, sz, sz, false, 1.0);
        // X_CA = -X_C T1
        hipLaunchKernelGGL((chol_pair_gemm_kernel<true, true, true, true, false>), dim3(t, t, pairs), dim3(256), 0,
                           st, c.Linv + sz * np + sz, np, c.A + sz, np, c.Linv + sz * np, np, np, sz, sz, 0, true,
                           -1.0);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    hipLaunchKernelGGL(chol_extract_u_kernel, dim3(grid_of(n * n)), dim3(256), 0, st, c.Linv, np, n, c.U);
    return hipGetLastError();
}

}  // namespace realq
