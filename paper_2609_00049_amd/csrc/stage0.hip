// Stage-0 accumulators (Alg. 1, Stage 0): per-token saliency restricted to the row groups of
// Eq. saliency_hessian, with the Hessian-side clip of Appendix D.1, and the 1/T scaling of the
// aggregated Fisher of Eq. fisher_full (its token contraction runs on the Hessian's MFMA GEMM).
//
// Row group g covers output channels [g r, min(m, (g+1) r)), r = ceil(m / n_groups).
#include "common.h"
#include "kernels.h"

namespace realq {

// s[g*T + t] = sum over the channels i of group g of G[t*m + i]^2, squares and sum in float64.
// One wave per (group, token) item, grid-stride over the items in group-major order.  Lanes read
// 16-byte runs of 8 channels from the 16-byte-aligned middle of the group's segment and single
// channels at its ragged ends; the wave reduces in a fixed butterfly order, so the result does
// not depend on the launch.
constexpr int SAL_BLOCKS = 2048;
__global__ __launch_bounds__(256) void saliency_sums_kernel(const uint16_t* __restrict__ G, int64_t T, int64_t m,
                                                            int64_t r, int64_t ng, double* __restrict__ s) {
    const int lane = threadIdx.x & 63;
    const int64_t nw = (int64_t)gridDim.x * 4;
    const int64_t items = T * ng;
    const bool rows16 = (m & 7) == 0 && (reinterpret_cast<uintptr_t>(G) & 15) == 0;
    for (int64_t it = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6); it < items; it += nw) {
        const int64_t g = it / T, t = it - g * T;
        const int64_t i0 = g * r, i1 = i0 + r < m ? i0 + r : m;
        const uint16_t* row = G + t * m;
        // aligned middle [a0, a1) in runs of 8; the ends element by element
        int64_t a0 = i0, a1 = i0;
        if (rows16) {
            a0 = (i0 + 7) & ~(int64_t)7;
            a1 = i1 & ~(int64_t)7;
            if (a1 < a0) a1 = a0 = i0;
        }
        double acc = 0.0;
        for (int64_t c = a0 + 8 * lane; c < a1; c += 512) {
            const u16x8 v = *reinterpret_cast<const u16x8*>(row + c);
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const double x = (double)bf2f(v[e]);
                acc += x * x;
            }
        }
        for (int64_t i = i0 + lane; i < a0; i += 64) {
            const double x = (double)bf2f(row[i]);
            acc += x * x;
        }
        const int64_t tail0 = a1 > a0 ? a1 : a0;
        for (int64_t i = tail0 + lane; i < i1; i += 64) {
            const double x = (double)bf2f(row[i]);
            acc += x * x;
        }
        for (int off = 32; off > 0; off >>= 1) acc += __shfl_xor(acc, off);
        if (lane == 0) s[it] = acc;
    }
}

// tau[g] = the k-th smallest of s[g*T .. g*T + T) (nearest rank), found exactly: non-negative
// doubles order like their uint64 bit patterns, so a radix select over eight 8-bit digits from
// the top.  Each digit takes two launches: SEL_SPLIT blocks per group count the values that
// match the prefix found so far into a global histogram (LDS histogram per block, then one
// global add per nonzero bin), and one block per group picks the digit where the running
// count reaches the remaining rank and clears the histogram for the next digit.
constexpr int SEL_SPLIT = 64;
struct SelState {
    unsigned long long prefix;
    long long krem;
};
__global__ __launch_bounds__(256) void select_init_kernel(SelState* st, uint32_t* hist, int64_t ng, int64_t k) {
    const int64_t g = blockIdx.x;
    if (threadIdx.x == 0) {
        st[g].prefix = 0ull;
        st[g].krem = k;
    }
    hist[g * 256 + threadIdx.x] = 0u;
    (void)ng;
}
__global__ __launch_bounds__(256) void select_count_kernel(const double* __restrict__ s, int64_t T, int pass,
                                                           const SelState* __restrict__ st, uint32_t* hist) {
    __shared__ uint32_t h[256];
    const int64_t g = blockIdx.x / SEL_SPLIT, part = blockIdx.x % SEL_SPLIT;
    const int64_t per = (T + SEL_SPLIT - 1) / SEL_SPLIT;
    const int64_t t0 = part * per, t1 = t0 + per < T ? t0 + per : T;
    const int shift = 56 - 8 * pass;
    const unsigned long long pre = st[g].prefix;
    h[threadIdx.x] = 0u;
    __syncthreads();
    const double* v = s + g * T;
    for (int64_t t = t0 + threadIdx.x; t < t1; t += 256) {
        const unsigned long long u = (unsigned long long)__double_as_longlong(v[t]);
        if (pass == 0 || (u >> (shift + 8)) == pre) atomicAdd(&h[(u >> shift) & 255ull], 1u);
    }
    __syncthreads();
    const uint32_t c = h[threadIdx.x];
    if (c) atomicAdd(&hist[g * 256 + threadIdx.x], c);
}
__global__ __launch_bounds__(256) void select_pick_kernel(SelState* st, uint32_t* hist, double* tau, int last) {
    __shared__ uint32_t h[256];
    const int64_t g = blockIdx.x;
    h[threadIdx.x] = hist[g * 256 + threadIdx.x];
    hist[g * 256 + threadIdx.x] = 0u;
    __syncthreads();
    if (threadIdx.x == 0) {
        const long long need = st[g].krem;
        long long acc = 0;
        unsigned bin = 255u;
        for (unsigned b = 0; b < 256u; ++b) {
            if (acc + (long long)h[b] >= need) {
                bin = b;
                break;
            }
            acc += h[b];
        }
        st[g].krem = need - acc;
        st[g].prefix = (st[g].prefix << 8) | bin;
        if (last) tau[g] = __longlong_as_double((long long)st[g].prefix);
    }
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
                    void* sel, float* out, hipStream_t st) {
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
        SelState* ss = reinterpret_cast<SelState*>(sel);
        uint32_t* hist = reinterpret_cast<uint32_t*>(ss + ng);
        hipLaunchKernelGGL(select_init_kernel, dim3((unsigned)ng), dim3(256), 0, st, ss, hist, ng, k);
        for (int pass = 0; pass < 8; ++pass) {
            hipLaunchKernelGGL(select_count_kernel, dim3((unsigned)(ng * SEL_SPLIT)), dim3(256), 0, st, s64, T, pass,
                               ss, hist);
            hipLaunchKernelGGL(select_pick_kernel, dim3((unsigned)ng), dim3(256), 0, st, ss, hist, tau,
                               pass == 7 ? 1 : 0);
        }
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

int64_t saliency_select_bytes(int64_t n_groups) { return n_groups * (int64_t)(sizeof(SelState) + 256 * 4); }

}  // namespace realq
