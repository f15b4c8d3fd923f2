// Output-perturbation clip of a BGD step (a_loss_clip, Appendix D.1): for every token t
// (column of R), the channels whose |R[i][t]| exceeds the token's q-quantile over the m
// channels are scaled down to it with the factor c = tau_t / |R| held fixed, so the step
// uses the loss sum s_t (c R)^2 and the gradient through c^2 R.
//
// clip_select_kernel finds tau_t exactly: the k-th smallest |R[:, t]| (k = ceil(q m),
// nearest rank) by a radix select on the float bit patterns (|R| >= 0, so their uint32
// order is the value order), four 8-bit digits from the top, one block per 64 consecutive
// tokens.  A wave reads 64 consecutive tokens of one row (256 coalesced bytes) and each
// lane counts its own token's digit into an LDS histogram.
#include "common.h"
#include "kernels.h"

namespace realq {

namespace {
constexpr int CT = 64;   // tokens per block
constexpr int CW = 4;    // waves per block
}  // namespace

__global__ __launch_bounds__(256) void clip_select_kernel(const float* __restrict__ R, int64_t ldr, int64_t m,
                                                          int64_t cur, int64_t k, float* __restrict__ tau) {
    __shared__ uint32_t hist[CT][256];
    __shared__ uint32_t prefix[CT];
    __shared__ uint32_t krem[CT];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int64_t t = (int64_t)blockIdx.x * CT + lane;
    const bool live = t < cur;
    if (threadIdx.x < CT) {
        prefix[threadIdx.x] = 0u;
        krem[threadIdx.x] = (uint32_t)k;
    }
    for (int pass = 0; pass < 4; ++pass) {
        const int shift = 24 - 8 * pass;
        for (int e = threadIdx.x; e < CT * 256; e += 256) (&hist[0][0])[e] = 0u;
        __syncthreads();
        const uint32_t pre = prefix[lane];
        for (int64_t i = wave; i < m; i += CW) {
            if (!live) continue;
            const uint32_t u = __float_as_uint(fabsf(R[i * ldr + t]));
            // digits above this pass must match the prefix found so far
            if (pass == 0 || (u >> (shift + 8)) == pre) atomicAdd(&hist[lane][(u >> shift) & 255u], 1u);
        }
        __syncthreads();
        if (threadIdx.x < CT) {
            const int c = threadIdx.x;
            uint32_t need = krem[c], acc = 0u, bin = 255u;
            for (uint32_t b = 0; b < 256u; ++b) {
                const uint32_t h = hist[c][b];
                if (acc + h >= need) {
                    bin = b;
                    break;
                }
                acc += h;
            }
            krem[c] = need - acc;
            prefix[c] = (prefix[c] << 8) | bin;
        }
        __syncthreads();
    }
    if (wave == 0 && live) tau[t] = __uint_as_float(prefix[lane]);
}

hipError_t clip_select(const float* R, int64_t ldr, int64_t m, int64_t cur, int64_t k, float* tau, hipStream_t st) {
    if (m <= 0 || cur <= 0) return hipSuccess;
    if (k < 1 || k > m) return hipErrorInvalidValue;
    const unsigned grid = (unsigned)((cur + CT - 1) / CT);
    hipLaunchKernelGGL(clip_select_kernel, dim3(grid), dim3(256), 0, st, R, ldr, m, cur, k, tau);
    return hipGetLastError();
}

// Apply: rs = c^2 s_t r written as the hi/lo bf16 pair the gradient GEMM reads, and fixed-order
// partial sums of s_t (c r)^2 (one per block; grid-stride over rows of the chunk).
constexpr int APPLY_BLOCKS = 1024;
__global__ __launch_bounds__(256) void clip_apply_kernel(const float* __restrict__ R, int64_t ldr, int64_t m,
                                                         int64_t cur, const float* __restrict__ tau,
                                                         const float* __restrict__ s, uint16_t* __restrict__ Rhi,
                                                         uint16_t* __restrict__ Rlo, double* __restrict__ partials) {
    __shared__ double red[256];
    double acc = 0.0;
    const int64_t total = m * cur;
    for (int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x; e < total; e += (int64_t)APPLY_BLOCKS * 256) {
        const int64_t i = e / cur, t = e % cur;
        const float r = R[i * ldr + t];
        const float a = fabsf(r), tt = tau[t];
        const float c = a > tt ? tt / a : 1.f;
        const float w = s ? s[t] : 1.f;
        const float cr = c * r;
        uint16_t h, l;
        split_bf16(c * cr * w, h, l);
        Rhi[i * ldr + t] = h;
        Rlo[i * ldr + t] = l;
        acc += (double)(w * cr) * (double)cr;
    }
    red[threadIdx.x] = acc;
    __syncthreads();
    for (int st = 128; st > 0; st >>= 1) {
        if (threadIdx.x < st) red[threadIdx.x] += red[threadIdx.x + st];
        __syncthreads();
    }
    if (threadIdx.x == 0) partials[blockIdx.x] = red[0];
}

hipError_t clip_apply(const float* R, int64_t ldr, int64_t m, int64_t cur, const float* tau, const float* s,
                      uint16_t* Rhi, uint16_t* Rlo, double* partials, hipStream_t st) {
    hipLaunchKernelGGL(clip_apply_kernel, dim3(APPLY_BLOCKS), dim3(256), 0, st, R, ldr, m, cur, tau, s, Rhi, Rlo,
                       partials);
    return hipGetLastError();
}
int64_t clip_apply_partials() { return APPLY_BLOCKS; }

}  // namespace realq
