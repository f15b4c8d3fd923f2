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
//   inverse  block rows of X = L^{-1}: X_ii = L_ii^{-1}, X_ij = -L_ii^{-1} sum_{j<=k<i} L_ik X_kj.
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

// ---------------------------------------------------------------- block row ib of X = L^{-1}
// X[ib][jb] = -Linv_ib * sum_{kb=jb}^{ib-1} L[ib][kb] X[kb][jb], one block per jb < ib.
__global__ __launch_bounds__(256) void chol_inv_row_kernel(const double* __restrict__ A, double* X, int64_t np,
                                                           int64_t ib, const double* __restrict__ diaginv) {
    __shared__ double sa[NB][NB + 1];
    __shared__ double sb[NB][NB + 1];
    const int64_t jb = blockIdx.x;
    double acc[4][4];
    zero_acc(acc);
    for (int64_t kb = jb; kb < ib; ++kb) {
        __syncthreads();
        load_tile(sa, A + ib * NB * np + kb * NB, np);
        load_tile(sb, X + kb * NB * np + jb * NB, np);
        __syncthreads();
        tile_mac_nn(acc, sa, sb);
    }
    __syncthreads();
    const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) sb[ty * 4 + i][tx * 4 + j] = acc[i][j];
    load_tile(sa, diaginv + ib * NB * NB, NB);
    __syncthreads();
    zero_acc(acc);
    tile_mac_nn(acc, sa, sb);
    double* C = X + ib * NB * np + jb * NB;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) C[(ty * 4 + i) * np + tx * 4 + j] = -acc[i][j];
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
    for (int64_t ib = 1; ib < nb; ++ib) {
        hipLaunchKernelGGL(chol_inv_row_kernel, dim3((unsigned)ib), dim3(256), 0, st, c.A, c.Linv, np, ib,
                           c.diaginv);
    }
    hipLaunchKernelGGL(chol_extract_u_kernel, dim3(grid_of(n * n)), dim3(256), 0, st, c.Linv, np, n, c.U);
    return hipGetLastError();
}

}  // namespace realq
