// float32 VALU GEMM, C = beta*C + alpha*A*B (all row-major), used where the sweep
// needs full float32 products of two non-bf16 operands with a short contraction:
// the trailing OBS update W[:, c1:] -= E_b U[b, c1:] (Sec. 3.2, K = block width)
// and the dense surrogate metric M_a G (Eq. fisher_loss).  Optionally refreshes the
// bf16 hi/lo split of C - W0 that the MFMA GEMMs consume.
// 64x64 output tile per 256-thread block, 4x4 per thread, K staged through LDS.
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
            if (a.Dhi) {
                uint16_t h, l;
                split_bf16(v - a.W0[gi * a.ldw + gj], h, l);
                a.Dhi[gi * a.ldd + gj] = h;
                a.Dlo[gi * a.ldd + gj] = l;
            }
        }
    }
}

hipError_t sgemm(const SgemmArgs& a, hipStream_t st) {
    if (a.M <= 0 || a.N <= 0) return hipSuccess;
    int64_t tiles_m = (a.M + TM - 1) / TM, tiles_n = (a.N + TN - 1) / TN;
    hipLaunchKernelGGL(sgemm_kernel, dim3((unsigned)(tiles_m * tiles_n)), dim3(256), 0, st, a, tiles_n);
    return hipGetLastError();
}

}  // namespace realq
