// Elementwise and per-token kernels of the block-output surrogate for a pre-norm SwiGLU MLP
// block (Sec. 4.2-4.4: the surrogate sits at the transformer block's output and Block-GD
// takes its gradient through the block):
//
//   u = bf16(rmsnorm(h) * gamma),  z = bf16(silu(u Wg^T) * (u Wu^T)),  y = h + bf16(z Wd^T).
//
// The products of the block run on the bf16 MFMA GEMM; the kernels here are HBM-bound
// (rows of d or f values per token), with the normalisation statistics and the SwiGLU in
// float64 so that the bf16 roundings fall where exact arithmetic puts them.
#include "common.h"
#include "kernels.h"

namespace realq {

namespace {
constexpr int TB = 256;
typedef uint16_t u16x4 __attribute__((ext_vector_type(4)));
inline unsigned grid_for(int64_t count) {
    int64_t b = (count + TB * 4 - 1) / (TB * 4);
    if (b < 1) b = 1;
    if (b > 65536) b = 65536;
    return (unsigned)b;
}
__device__ __forceinline__ float ld_act(const uint16_t* p, int64_t i) { return bf2f(p[i]); }
__device__ __forceinline__ float ld_act(const float* p, int64_t i) { return p[i]; }

// fixed-order block reduction of one double per thread (256 threads); result valid in thread 0
__device__ __forceinline__ double block_sum(double v, double* red) {
    red[threadIdx.x] = v;
    __syncthreads();
    for (int s = TB / 2; s > 0; s >>= 1) {
        if ((int)threadIdx.x < s) red[threadIdx.x] += red[threadIdx.x + s];
        __syncthreads();
    }
    const double r = red[0];
    __syncthreads();
    return r;
}
}  // namespace

// u[t, i] = bf16(h[t, i] r_t gamma_i), r_t = (mean_i h[t, i]^2 + eps)^(-1/2); one block per token.
template <typename TIn>
__global__ __launch_bounds__(256) void rmsnorm_kernel(const TIn* __restrict__ h, int64_t T, int64_t d,
                                                      const float* __restrict__ gamma, double eps,
                                                      uint16_t* __restrict__ u) {
    __shared__ double red[TB];
    for (int64_t t = blockIdx.x; t < T; t += gridDim.x) {
        const TIn* row = h + t * d;
        double ss = 0.0;
        for (int64_t i = threadIdx.x; i < d; i += TB) {
            const double x = (double)ld_act(row, i);
            ss += x * x;
        }
        const double r = 1.0 / sqrt(block_sum(ss, red) / (double)d + eps);
        for (int64_t i = threadIdx.x; i < d; i += TB)
            u[t * d + i] = f2bf((float)((double)ld_act(row, i) * r * (double)gamma[i]));
    }
}

hipError_t rmsnorm_bf16(const uint16_t* h, int64_t T, int64_t d, const float* gamma, double eps, uint16_t* u,
                        hipStream_t st) {
    if (T <= 0) return hipSuccess;
    hipLaunchKernelGGL(rmsnorm_kernel<uint16_t>, dim3((unsigned)(T < 65536 ? T : 65536)), dim3(TB), 0, st, h, T, d,
                       gamma, eps, u);
    return hipGetLastError();
}
hipError_t rmsnorm_f32(const float* h, int64_t T, int64_t d, const float* gamma, double eps, uint16_t* u,
                       hipStream_t st) {
    if (T <= 0) return hipSuccess;
    hipLaunchKernelGGL(rmsnorm_kernel<float>, dim3((unsigned)(T < 65536 ? T : 65536)), dim3(TB), 0, st, h, T, d,
                       gamma, eps, u);
    return hipGetLastError();
}

// z = bf16(silu(a) b), silu(a) = a / (1 + e^-a), in float64 from the float32 a and b.
__device__ __forceinline__ uint16_t swiglu_elem(float av, float bv) {
    const double x = (double)av;
    return f2bf((float)(x / (1.0 + exp(-x)) * (double)bv));
}
__global__ void swiglu_fwd_kernel(const float* __restrict__ a, const float* __restrict__ b, uint16_t* __restrict__ z,
                                  int64_t count) {
    for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < count; e += (int64_t)gridDim.x * blockDim.x)
        z[e] = swiglu_elem(a[e], b[e]);
}
// four consecutive elements per thread (count a multiple of 4, 16-byte aligned inputs, 8-byte aligned output)
__global__ void swiglu_fwd4_kernel(const float* __restrict__ a, const float* __restrict__ b, uint16_t* __restrict__ z,
                                   int64_t quads) {
    for (int64_t q = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; q < quads; q += (int64_t)gridDim.x * blockDim.x) {
        const f32x4 xa = *reinterpret_cast<const f32x4*>(a + 4 * q);
        const f32x4 xb = *reinterpret_cast<const f32x4*>(b + 4 * q);
        u16x4 o;
#pragma unroll
        for (int u = 0; u < 4; ++u) o[u] = swiglu_elem(xa[u], xb[u]);
        *reinterpret_cast<u16x4*>(z + 4 * q) = o;
    }
}
hipError_t swiglu_fwd(const float* a, const float* b, uint16_t* z, int64_t count, hipStream_t st) {
    if (count <= 0) return hipSuccess;
    if (count % 4 == 0 && ((uintptr_t)a & 15u) == 0 && ((uintptr_t)b & 15u) == 0 && ((uintptr_t)z & 7u) == 0) {
        hipLaunchKernelGGL(swiglu_fwd4_kernel, dim3(grid_for(count / 4)), dim3(TB), 0, st, a, b, z, count / 4);
    } else {
        hipLaunchKernelGGL(swiglu_fwd_kernel, dim3(grid_for(count)), dim3(TB), 0, st, a, b, z, count);
    }
    return hipGetLastError();
}

// y = h + out (float32; out bf16), dy = y - ystar when dy != NULL.
template <typename TIn>
__global__ void residual_out_kernel(const TIn* __restrict__ h, const uint16_t* __restrict__ out,
                                    const float* __restrict__ ystar, float* __restrict__ y, float* __restrict__ dy,
                                    int64_t count) {
    for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < count; e += (int64_t)gridDim.x * blockDim.x) {
        const float v = ld_act(h, e) + bf2f(out[e]);
        if (y) y[e] = v;
        if (dy) dy[e] = v - ystar[e];
    }
}
hipError_t residual_out_bf16(const uint16_t* h, const uint16_t* out, const float* ystar, float* y, float* dy,
                             int64_t count, hipStream_t st) {
    if (count <= 0) return hipSuccess;
    hipLaunchKernelGGL(residual_out_kernel<uint16_t>, dim3(grid_for(count)), dim3(TB), 0, st, h, out, ystar, y, dy,
                       count);
    return hipGetLastError();
}
hipError_t residual_out_f32(const float* h, const uint16_t* out, const float* ystar, float* y, float* dy,
                            int64_t count, hipStream_t st) {
    if (count <= 0) return hipSuccess;
    hipLaunchKernelGGL(residual_out_kernel<float>, dim3(grid_for(count)), dim3(TB), 0, st, h, out, ystar, y, dy,
                       count);
    return hipGetLastError();
}

// out = s * x, and hi/lo = split(out) when hi != NULL.
__global__ void scale_split_kernel(const float* __restrict__ x, float s, float* __restrict__ out,
                                   uint16_t* __restrict__ hi, uint16_t* __restrict__ lo, int64_t count) {
    for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < count; e += (int64_t)gridDim.x * blockDim.x) {
        const float v = s * x[e];
        if (out) out[e] = v;
        if (hi) split_bf16(v, hi[e], lo[e]);
    }
}
hipError_t scale_split(const float* x, float s, float* out, uint16_t* hi, uint16_t* lo, int64_t count,
                       hipStream_t st) {
    if (count <= 0) return hipSuccess;
    hipLaunchKernelGGL(scale_split_kernel, dim3(grid_for(count)), dim3(TB), 0, st, x, s, out, hi, lo, count);
    return hipGetLastError();
}

// partials[b] = scale * (fixed-order sum over the block's grid-stride share of x y), float64.
constexpr int DOT32_BLOCKS = 1024;
__global__ __launch_bounds__(256) void dot_f32_kernel(const float* __restrict__ x, const float* __restrict__ y,
                                                      int64_t count, double scale, double* __restrict__ partials) {
    __shared__ double red[TB];
    double acc = 0.0;
    for (int64_t e = (int64_t)blockIdx.x * TB + threadIdx.x; e < count; e += (int64_t)DOT32_BLOCKS * TB)
        acc += (double)x[e] * (double)y[e];
    const double s = block_sum(acc, red);
    if (threadIdx.x == 0) partials[blockIdx.x] = scale * s;
}
hipError_t dot_f32(const float* x, const float* y, int64_t count, double scale, double* partials, hipStream_t st) {
    hipLaunchKernelGGL(dot_f32_kernel, dim3(DOT32_BLOCKS), dim3(TB), 0, st, x, y, count, scale, partials);
    return hipGetLastError();
}
int64_t dot_f32_partials() { return DOT32_BLOCKS; }

// SwiGLU backward to one of its inputs from dz [T, f]:
//   gate (which 0): v = dz b sigma(a) (1 + a (1 - sigma(a)));   up (which 1): v = dz a sigma(a)
// written as a bf16 hi/lo pair, transposed ([f][ldo], column t) when transposed != 0 (the
// operand of the weight gradient v^T u), else row-major [T][f] (the operand of v W).
// The transposed form goes through a 64 x 64 LDS tile.
__global__ __launch_bounds__(256) void swiglu_bwd_kernel(const float* __restrict__ dz, const float* __restrict__ a,
                                                         const float* __restrict__ b, int which, int64_t T, int64_t f,
                                                         int transposed, uint16_t* __restrict__ hi,
                                                         uint16_t* __restrict__ lo, int64_t ldo, int64_t tiles_f) {
    __shared__ float tile[64][65];
    const int64_t tt = blockIdx.x / tiles_f, tf = blockIdx.x % tiles_f;
    const int64_t t0 = tt * 64, f0 = tf * 64;
    const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
    for (int rr = ty; rr < 64; rr += 4) {
        const int64_t t = t0 + rr, i = f0 + tx;
        float v = 0.f;
        if (t < T && i < f) {
            const int64_t e = t * f + i;
            const double x = (double)a[e];
            const double sg = 1.0 / (1.0 + exp(-x));
            const double w = which == 0 ? (double)b[e] * sg * (1.0 + x * (1.0 - sg)) : x * sg;
            v = (float)((double)dz[e] * w);
        }
        if (!transposed) {
            if (t < T && i < f) split_bf16(v, hi[t * ldo + i], lo[t * ldo + i]);
        } else {
            tile[rr][tx] = v;
        }
    }
    if (!transposed) return;
    __syncthreads();
    for (int cc = ty; cc < 64; cc += 4) {
        const int64_t i = f0 + cc, t = t0 + tx;
        if (t < T && i < f) split_bf16(tile[tx][cc], hi[i * ldo + t], lo[i * ldo + t]);
    }
}
// Both row-major SwiGLU backward outputs of one dz in one pass (the gate's to hi0/lo0, the up
// projection's to hi1/lo1), four consecutive columns per thread when rows allow 16-byte loads;
// per element the arithmetic of swiglu_bwd_kernel, so both outputs are bitwise the same.
__device__ __forceinline__ void swiglu_bwd_pair_elem(float d, float av, float bv, uint16_t& h0, uint16_t& l0,
                                                     uint16_t& h1, uint16_t& l1) {
    const double x = (double)av;
    const double sg = 1.0 / (1.0 + exp(-x));
    const double w0 = (double)bv * sg * (1.0 + x * (1.0 - sg));
    const double w1 = x * sg;
    split_bf16((float)((double)d * w0), h0, l0);
    split_bf16((float)((double)d * w1), h1, l1);
}
__global__ __launch_bounds__(256) void swiglu_bwd_pair_kernel(const float* __restrict__ dz, const float* __restrict__ a,
                                                              const float* __restrict__ b, int64_t T, int64_t f,
                                                              uint16_t* __restrict__ hi0, uint16_t* __restrict__ lo0,
                                                              uint16_t* __restrict__ hi1, uint16_t* __restrict__ lo1,
                                                              int64_t ldo, int vec) {
    const int64_t fq = vec ? f / 4 : f;
    const int64_t n = T * fq;
    for (int64_t q = (int64_t)blockIdx.x * TB + threadIdx.x; q < n; q += (int64_t)gridDim.x * TB) {
        const int64_t t = q / fq, c = q - t * fq;
        if (vec) {
            const int64_t e = t * f + 4 * c, o = t * ldo + 4 * c;
            const f32x4 xd = *reinterpret_cast<const f32x4*>(dz + e);
            const f32x4 xa = *reinterpret_cast<const f32x4*>(a + e);
            const f32x4 xb = *reinterpret_cast<const f32x4*>(b + e);
            u16x4 h0, l0, h1, l1;
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                uint16_t a0, a1, b0, b1;
                swiglu_bwd_pair_elem(xd[u], xa[u], xb[u], a0, a1, b0, b1);
                h0[u] = a0;
                l0[u] = a1;
                h1[u] = b0;
                l1[u] = b1;
            }
            *reinterpret_cast<u16x4*>(hi0 + o) = h0;
            *reinterpret_cast<u16x4*>(lo0 + o) = l0;
            *reinterpret_cast<u16x4*>(hi1 + o) = h1;
            *reinterpret_cast<u16x4*>(lo1 + o) = l1;
        } else {
            const int64_t e = t * f + c, o = t * ldo + c;
            swiglu_bwd_pair_elem(dz[e], a[e], b[e], hi0[o], lo0[o], hi1[o], lo1[o]);
        }
    }
}
hipError_t swiglu_bwd_pair(const float* dz, const float* a, const float* b, int64_t T, int64_t f, uint16_t* hi0,
                           uint16_t* lo0, uint16_t* hi1, uint16_t* lo1, int64_t ldo, hipStream_t st) {
    if (T <= 0 || f <= 0) return hipSuccess;
    auto a16 = [](const void* p) { return ((uintptr_t)p & 15u) == 0; };
    auto a8 = [](const void* p) { return ((uintptr_t)p & 7u) == 0; };
    const int vec = f % 4 == 0 && ldo % 4 == 0 && a16(dz) && a16(a) && a16(b) && a8(hi0) && a8(lo0) && a8(hi1) && a8(lo1);
    const int64_t n = T * (vec ? f / 4 : f);
    hipLaunchKernelGGL(swiglu_bwd_pair_kernel, dim3(grid_for(n)), dim3(TB), 0, st, dz, a, b, T, f, hi0, lo0, hi1, lo1,
                       ldo, vec);
    return hipGetLastError();
}

hipError_t swiglu_bwd(const float* dz, const float* a, const float* b, int which, int64_t T, int64_t f,
                      int transposed, uint16_t* hi, uint16_t* lo, int64_t ldo, hipStream_t st) {
    if (T <= 0 || f <= 0) return hipSuccess;
    const int64_t tiles_t = (T + 63) / 64, tiles_f = (f + 63) / 64;
    hipLaunchKernelGGL(swiglu_bwd_kernel, dim3((unsigned)(tiles_t * tiles_f)), dim3(TB), 0, st, dz, a, b, which, T, f,
                       transposed, hi, lo, ldo, tiles_f);
    return hipGetLastError();
}

// hi/lo[c * ldo + r] = split(in[r * ldi + c]) for r < rows, c < cols (float32 in, transposed out).
__global__ __launch_bounds__(256) void transpose_split_f32_kernel(const float* __restrict__ in, int64_t ldi,
                                                                  uint16_t* __restrict__ hi, uint16_t* __restrict__ lo,
                                                                  int64_t ldo, int64_t rows, int64_t cols,
                                                                  int64_t tiles_c) {
    __shared__ float tile[64][65];
    const int64_t tr = blockIdx.x / tiles_c, tc = blockIdx.x % tiles_c;
    const int64_t r0 = tr * 64, c0 = tc * 64;
    const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
    for (int rr = ty; rr < 64; rr += 4) {
        const int64_t r = r0 + rr, c = c0 + tx;
        tile[rr][tx] = (r < rows && c < cols) ? in[r * ldi + c] : 0.f;
    }
    __syncthreads();
    for (int cc = ty; cc < 64; cc += 4) {
        const int64_t c = c0 + cc, r = r0 + tx;
        if (r < rows && c < cols) split_bf16(tile[tx][cc], hi[c * ldo + r], lo[c * ldo + r]);
    }
}
hipError_t transpose_split_f32(const float* in, int64_t ldi, uint16_t* hi, uint16_t* lo, int64_t ldo, int64_t rows,
                               int64_t cols, hipStream_t st) {
    if (rows <= 0 || cols <= 0) return hipSuccess;
    const int64_t tr = (rows + 63) / 64, tc = (cols + 63) / 64;
    hipLaunchKernelGGL(transpose_split_f32_kernel, dim3((unsigned)(tr * tc)), dim3(TB), 0, st, in, ldi, hi, lo, ldo,
                       rows, cols, tc);
    return hipGetLastError();
}

// The next block's input gradient blended into the current one, per token:
//   dh = g2 + r (gamma du) - r^3 h mean_i(h gamma du),  r = (mean_i h^2 + eps)^(-1/2)   (RMSNorm backward)
//   g  = alpha g + (1 - alpha) dh
// with h the next block's input (this block's output y), in float64; one block per token.
__global__ __launch_bounds__(256) void rmsnorm_bwd_blend_kernel(const float* __restrict__ h,
                                                                const float* __restrict__ g2,
                                                                const float* __restrict__ du,
                                                                const float* __restrict__ gamma, double eps,
                                                                double alpha, int64_t T, int64_t d,
                                                                float* __restrict__ g) {
    __shared__ double red[TB];
    for (int64_t t = blockIdx.x; t < T; t += gridDim.x) {
        const float* hr = h + t * d;
        const float* dr = du + t * d;
        double ss = 0.0, hd = 0.0;
        for (int64_t i = threadIdx.x; i < d; i += TB) {
            const double x = (double)hr[i];
            ss += x * x;
            hd += x * (double)gamma[i] * (double)dr[i];
        }
        const double r = 1.0 / sqrt(block_sum(ss, red) / (double)d + eps);
        const double mhd = block_sum(hd, red) / (double)d;
        for (int64_t i = threadIdx.x; i < d; i += TB) {
            const int64_t e = t * d + i;
            const double dh = (double)g2[e] + r * (double)gamma[i] * (double)dr[i] - r * r * r * (double)hr[i] * mhd;
            g[e] = (float)((alpha != 0.0 ? alpha * (double)g[e] : 0.0) + (1.0 - alpha) * dh);
        }
    }
}
hipError_t rmsnorm_bwd_blend(const float* h, const float* g2, const float* du, const float* gamma, double eps,
                             double alpha, int64_t T, int64_t d, float* g, hipStream_t st) {
    if (T <= 0) return hipSuccess;
    hipLaunchKernelGGL(rmsnorm_bwd_blend_kernel, dim3((unsigned)(T < 65536 ? T : 65536)), dim3(TB), 0, st, h, g2, du,
                       gamma, eps, alpha, T, d, g);
    return hipGetLastError();
}

}  // namespace realq
