// Stage-0 accumulators (Alg. 1, Stage 0): per-token saliency restricted to the row groups of
// Eq. saliency_hessian, with the Hessian-side clip of Appendix D.1, and the 1/T scaling of the
// aggregated Fisher of Eq. fisher_full (its token contraction runs on the Hessian's MFMA GEMM).
//
// Row group g covers output channels [g r, min(m, (g+1) r)), r = ceil(m / n_groups).
#include "common.h"
#include "kernels.h"

namespace realq {

// s[g*T + t] = sum over the channels i of group g of G[t*m + i]^2, squares and sum in float64.
// One wave per (group, token) item, grid-stride over the items in group-major order; the lanes
// read consecutive channels of the group's contiguous segment (128 bytes per wave load) and the
// wave reduces in a fixed butterfly order, so the result does not depend on the launch.
constexpr int SAL_BLOCKS = 2048;
__global__ __launch_bounds__(256) void saliency_sums_kernel(const uint16_t* __restrict__ G, int64_t T, int64_t m,
                                                            int64_t r, int64_t ng, double* __restrict__ s) {
    const int lane = threadIdx.x & 63;
    const int64_t nw = (int64_t)gridDim.x * 4;
    const int64_t items = T * ng;
    for (int64_t it = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6); it < items; it += nw) {
        const int64_t g = it / T, t = it - g * T;
        const int64_t i0 = g * r, i1 = i0 + r < m ? i0 + r : m;
        const uint16_t* row = G + t * m;
        double a0 = 0.0, a1 = 0.0;
        int64_t i = i0 + lane;
        for (; i + 64 < i1; i += 128) {
            const double v0 = (double)bf2f(row[i]), v1 = (double)bf2f(row[i + 64]);
            a0 += v0 * v0;
            a1 += v1 * v1;
        }
        if (i < i1) {
            const double v0 = (double)bf2f(row[i]);
            a0 += v0 * v0;
        }
        double acc = a0 + a1;
        for (int off = 32; off > 0; off >>= 1) acc += __shfl_xor(acc, off);
        if (lane == 0) s[it] = acc;
    }
}

// tau[g] = the k-th smallest of s[g*T .. g*T + T) (nearest rank), found exactly: non-negative
// doubles order like their uint64 bit patterns, so a radix select over eight 8-bit digits from
// the top, one block per group.
__global__ __launch_bounds__(1024) void saliency_select_kernel(const double* __restrict__ s, int64_t T, int64_t k,
                                                               double* __restrict__ tau) {
    __shared__ uint32_t hist[256];
    __shared__ unsigned long long prefix;
    __shared__ long long krem;
    const double* v = s + (int64_t)blockIdx.x * T;
    if (threadIdx.x == 0) {
        prefix = 0ull;
        krem = k;
    }
    for (int pass = 0; pass < 8; ++pass) {
        const int shift = 56 - 8 * pass;
        if (threadIdx.x < 256) hist[threadIdx.x] = 0u;
        __syncthreads();
        const unsigned long long pre = prefix;
        for (int64_t t = threadIdx.x; t < T; t += 1024) {
            const unsigned long long u = (unsigned long long)__double_as_longlong(v[t]);
            // digits above this pass must match the prefix found so far
            if (pass == 0 || (u >> (shift + 8)) == pre) atomicAdd(&hist[(u >> shift) & 255ull], 1u);
        }
        __syncthreads();
        if (threadIdx.x == 0) {
            long long need = krem, acc = 0;
            unsigned bin = 255u;
            for (unsigned b = 0; b < 256u; ++b) {
                const long long h = hist[b];
                if (acc + h >= need) {
                    bin = b;
                    break;
                }
                acc += h;
            }
            krem = need - acc;
            prefix = (prefix << 8) | bin;
        }
        __syncthreads();
    }
    if (threadIdx.x == 0) tau[blockIdx.x] = __longlong_as_double((long long)prefix);
}

// out[e] = float(min(s[e], tau[e / T])) for e < live (tau NULL: no clip); out[e] = 0 for the rows
// of empty groups, e in [live, total).
constexpr int APPLY_SAL_BLOCKS = 1024;
__global__ __launch_bounds__(256) void saliency_apply_kernel(const double* __restrict__ s, int64_t T, int64_t live,
                                                             int64_t total, const double* __restrict__ tau,
                                                             float* __restrict__ out) {
    for (int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x; e < total; e += (int64_t)APPLY_SAL_BLOCKS * 256) {
        double x = 0.0;
        if (e < live) {
            x = s[e];
            if (tau) x = fmin(x, tau[e / T]);
        }
        out[e] = (float)x;
    }
}

hipError_t saliency(const uint16_t* G, int64_t T, int64_t m, int64_t n_groups, int64_t k, double* s64, double* tau,
                    float* out, hipStream_t st) {
    if (T <= 0 || m <= 0 || n_groups <= 0) return hipSuccess;
    const int64_t r = (m + n_groups - 1) / n_groups;
    const int64_t ng = (m + r - 1) / r;  // groups that hold at least one row
    const int64_t items = T * ng;
    const unsigned grid = (unsigned)(items / 4 + 1 < SAL_BLOCKS ? items / 4 + 1 : SAL_BLOCKS);
    hipLaunchKernelGGL(saliency_sums_kernel, dim3(grid), dim3(256), 0, st, G, T, m, r, ng, s64);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (k > 0) {
        if (k > T) return hipErrorInvalidValue;
        hipLaunchKernelGGL(saliency_select_kernel, dim3((unsigned)ng), dim3(1024), 0, st, s64, T, k, tau);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    hipLaunchKernelGGL(saliency_apply_kernel, dim3(APPLY_SAL_BLOCKS), dim3(256), 0, st, s64, T, items, T * n_groups,
                       k > 0 ? tau : nullptr, out);
    return hipGetLastError();
}

// out[e] = float(a[e] / d)
__global__ __launch_bounds__(256) void div_narrow_kernel(const double* __restrict__ a, double d, float* __restrict__ out,
                                                         int64_t count) {
    for (int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x; e < count; e += (int64_t)gridDim.x * 256)
        out[e] = (float)(a[e] / d);
}

hipError_t div_narrow(const double* a, double d, float* out, int64_t count, hipStream_t st) {
    if (count <= 0) return hipSuccess;
    const int64_t blocks = (count + 255) / 256;
    hipLaunchKernelGGL(div_narrow_kernel, dim3((unsigned)(blocks < 4096 ? blocks : 4096)), dim3(256), 0, st, a, d, out,
                       count);
    return hipGetLastError();
}

}  // namespace realq
