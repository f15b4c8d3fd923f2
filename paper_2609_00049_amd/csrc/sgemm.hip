// VALU GEMMs, all row-major, 64x64 output tile per 256-thread block, 4x4 per thread, K
// staged through LDS.
//   sgemm  C = beta*C + alpha*A*B in float32: the dense surrogate metric M_a G
//          (Eq. fisher_loss) and the window partner W_next^T M_next W_next (Eq.
//          slide_window).
//   dgemm  C (+)= A*B in float64: the products of the final loss with a dense metric,
//          written through the calibration Gram matrices.
#include "common.h"
#include "kernels.h"

namespace realq {

namespace {
constexpr int TM = 64, TN = 64, TK = 16;
}

__global__ __launch_bounds__(256) void sgemm_kernel(SgemmArgs a, int64_t tiles_n) {
    __shared__ float sA[TK][TM + 4];
    __shared__ float sB[TK][TN + 4];
    const int64_t tm = blockIdx.x / tiles_n, tn = blockIdx.x % tiles_n;
    const int64_t m0 = tm * TM, n0 = tn * TN;
    const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;  // 16 x 16 threads, 4x4 each
    float acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = 0.f;

    for (int64_t k0 = 0; k0 < a.K; k0 += TK) {
        // A tile: 64 rows x 16 k -> 1024 values, 4 per thread
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            int e = threadIdx.x + r * 256;
            int row = e / TK, kk = e % TK;
            int64_t gi = m0 + row, gk = k0 + kk;
            sA[kk][row] = (gi < a.M && gk < a.K) ? a.A[gi * a.lda + gk] : 0.f;
        }
        // B tile: 16 k x 64 cols
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            int e = threadIdx.x + r * 256;
            int kk = e / TN, col = e % TN;
            int64_t gk = k0 + kk, gj = n0 + col;
            sB[kk][col] = (gk < a.K && gj < a.N) ? a.B[gk * a.ldb + gj] : 0.f;
        }
        __syncthreads();
#pragma unroll
        for (int kk = 0; kk < TK; ++kk) {
            float av[4], bv[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) av[i] = sA[kk][ty * 4 + i];
#pragma unroll
            for (int j = 0; j < 4; ++j) bv[j] = sB[kk][tx + 16 * j];
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(av[i], bv[j], acc[i][j]);
        }
        __syncthreads();
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        int64_t gi = m0 + ty * 4 + i;
        if (gi >= a.M) continue;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            int64_t gj = n0 + tx + 16 * j;
            if (gj >= a.N) continue;
            float* c = a.C + gi * a.ldc + gj;
            float v = a.alpha * acc[i][j];
            if (a.beta != 0.f) v = fmaf(a.beta, *c, v);
            *c = v;
        }
    }
}

// float64 counterpart (C = A B or C += A B), same tiling with double operands in LDS.
__global__ __launch_bounds__(256) void dgemm_kernel(const double* __restrict__ A, int64_t lda,
                                                    const double* __restrict__ B, int64_t ldb, double* __restrict__ C,
                                                    int64_t ldc, int64_t M, int64_t N, int64_t K, int accumulate,
                                                    int64_t tiles_n) {
    __shared__ double sA[TK][TM + 1];
    __shared__ double sB[TK][TN + 1];
    const int64_t tm = blockIdx.x / tiles_n, tn = blockIdx.x % tiles_n;
    const int64_t m0 = tm * TM, n0 = tn * TN;
    const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
    double acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = 0.0;
    for (int64_t k0 = 0; k0 < K; k0 += TK) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int e = threadIdx.x + r * 256;
            const int row = e / TK, kk = e % TK;
            const int64_t gi = m0 + row, gk = k0 + kk;
            sA[kk][row] = (gi < M && gk < K) ? A[gi * lda + gk] : 0.0;
        }
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int e = threadIdx.x + r * 256;
            const int kk = e / TN, col = e % TN;
            const int64_t gk = k0 + kk, gj = n0 + col;
            sB[kk][col] = (gk < K && gj < N) ? B[gk * ldb + gj] : 0.0;
        }
        __syncthreads();
#pragma unroll
        for (int kk = 0; kk < TK; ++kk) {
            double av[4], bv[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) av[i] = sA[kk][ty * 4 + i];
#pragma unroll
            for (int j = 0; j < 4; ++j) bv[j] = sB[kk][tx + 16 * j];
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) acc[i][j] = fma(av[i], bv[j], acc[i][j]);
        }
        __syncthreads();
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int64_t gi = m0 + ty * 4 + i;
        if (gi >= M) continue;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int64_t gj = n0 + tx + 16 * j;
            if (gj >= N) continue;
            double* c = C + gi * ldc + gj;
            *c = accumulate ? *c + acc[i][j] : acc[i][j];
        }
    }
}

hipError_t dgemm(const double* A, int64_t lda, const double* B, int64_t ldb, double* C, int64_t ldc, int64_t M,
                 int64_t N, int64_t K, bool accumulate, hipStream_t st) {
    if (M <= 0 || N <= 0) return hipSuccess;
    const int64_t tiles_m = (M + TM - 1) / TM, tiles_n = (N + TN - 1) / TN;
    hipLaunchKernelGGL(dgemm_kernel, dim3((unsigned)(tiles_m * tiles_n)), dim3(256), 0, st, A, lda, B, ldb, C, ldc,
                       M, N, K, (int)accumulate, tiles_n);
    return hipGetLastError();
}

hipError_t sgemm(const SgemmArgs& a, hipStream_t st) {
    if (a.M <= 0 || a.N <= 0) return hipSuccess;
    int64_t tiles_m = (a.M + TM - 1) / TM, tiles_n = (a.N + TN - 1) / TN;
    hipLaunchKernelGGL(sgemm_kernel, dim3((unsigned)(tiles_m * tiles_n)), dim3(256), 0, st, a, tiles_n);
    return hipGetLastError();
}

}  // namespace realq
