// Memory-bound helper kernels: fills, bf16 transposes and splits, deterministic
// reductions and the fused split-K reduction + Adam update (Appendix D.1 constants
// arrive as arguments).  Every kernel here is HBM-bound; loops are grid-strided
// with coalesced rows.
#include "common.h"
#include "kernels.h"

namespace realq {

namespace {
constexpr int TB = 256;
inline unsigned grid_for(int64_t count, int per_thread = 1) {
    int64_t b = (count + (int64_t)TB * per_thread - 1) / ((int64_t)TB * per_thread);
    if (b < 1) b = 1;
    if (b > 65536) b = 65536;
    return (unsigned)b;
}
}  // namespace

template <class T>
__global__ void fill_kernel(T* p, T v, int64_t count) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < count; i += (int64_t)gridDim.x * blockDim.x)
        p[i] = v;
}

hipError_t fill_f32(float* p, float v, int64_t count, hipStream_t st) {
    if (count <= 0) return hipSuccess;
    hipLaunchKernelGGL(fill_kernel<float>, dim3(grid_for(count, 4)), dim3(TB), 0, st, p, v, count);
    return hipGetLastError();
}
hipError_t fill_f64(double* p, double v, int64_t count, hipStream_t st) {
    if (count <= 0) return hipSuccess;
    hipLaunchKernelGGL(fill_kernel<double>, dim3(grid_for(count, 4)), dim3(TB), 0, st, p, v, count);
    return hipGetLastError();
}
hipError_t fill_u16(uint16_t* p, uint16_t v, int64_t count, hipStream_t st) {
    if (count <= 0) return hipSuccess;
    hipLaunchKernelGGL(fill_kernel<uint16_t>, dim3(grid_for(count, 4)), dim3(TB), 0, st, p, v, count);
    return hipGetLastError();
}

// ---------------------------------------------------------------- tiled transposes (64 x 64 tiles via LDS)
// MODE 0: plain copy of bit patterns; MODE 1: value s[r] * x, written as a hi/lo bf16 pair and,
// when o3 != NULL, a third bf16 term of what hi + lo leaves (hi + lo + o3 holds all 24 bits of
// the float32 product).
template <int MODE>
__global__ __launch_bounds__(256) void transpose_kernel(const uint16_t* __restrict__ in, int64_t ldi,
                                                        const float* __restrict__ s, uint16_t* __restrict__ o1,
                                                        uint16_t* __restrict__ o2, uint16_t* __restrict__ o3,
                                                        int64_t ldo, int64_t rows, int64_t cols, int64_t tiles_c) {
    __shared__ float tile[64][65];
    const int64_t tr = blockIdx.x / tiles_c, tc = blockIdx.x % tiles_c;
    const int64_t r0 = tr * 64, c0 = tc * 64;
    const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;  // 4 rows of 64 threads
    for (int rr = ty; rr < 64; rr += 4) {
        int64_t r = r0 + rr, c = c0 + tx;
        float v = 0.f;
        if (r < rows && c < cols) {
            v = bf2f(in[r * ldi + c]);
            if (MODE == 1 && s) v *= s[r];
        }
        tile[rr][tx] = v;
    }
    __syncthreads();
    for (int cc = ty; cc < 64; cc += 4) {
        int64_t c = c0 + cc, r = r0 + tx;
        if (r < rows && c < cols) {
            float v = tile[tx][cc];
            if (MODE == 0) {
                o1[c * ldo + r] = f2bf(v);  // exact: v is a bf16 value
            } else {
                uint16_t hi, lo;
                split_bf16(v, hi, lo);
                o1[c * ldo + r] = hi;
                o2[c * ldo + r] = lo;
                // v - hi and then - lo are exact in float32 (each term keeps v's leading bits)
                if (o3) o3[c * ldo + r] = f2bf((v - bf2f(hi)) - bf2f(lo));
            }
        }
    }
}

hipError_t transpose_u16(const uint16_t* in, int64_t ldi, uint16_t* out, int64_t ldo, int64_t rows, int64_t cols,
                         hipStream_t st) {
    if (rows <= 0 || cols <= 0) return hipSuccess;
    int64_t tr = (rows + 63) / 64, tc = (cols + 63) / 64;
    hipLaunchKernelGGL(transpose_kernel<0>, dim3((unsigned)(tr * tc)), dim3(256), 0, st, in, ldi, nullptr, out,
                       nullptr, nullptr, ldo, rows, cols, tc);
    return hipGetLastError();
}

hipError_t transpose_scale_split(const uint16_t* in, int64_t ldi, const float* s, uint16_t* hi, uint16_t* lo,
                                 uint16_t* lo2, int64_t ldo, int64_t rows, int64_t cols, hipStream_t st) {
    if (rows <= 0 || cols <= 0) return hipSuccess;
    int64_t tr = (rows + 63) / 64, tc = (cols + 63) / 64;
    hipLaunchKernelGGL(transpose_kernel<1>, dim3((unsigned)(tr * tc)), dim3(256), 0, st, in, ldi, s, hi, lo, lo2,
                       ldo, rows, cols, tc);
    return hipGetLastError();
}

// Input perturbation of one token chunk, transposed: delta = Xhat - X (rows = tokens), and
// the hi/lo bf16 pairs of s[r] * delta and of delta, written as [cols][rows].
__global__ __launch_bounds__(256) void transpose_delta_kernel(const uint16_t* __restrict__ Xh,
                                                              const uint16_t* __restrict__ X, int64_t ldi,
                                                              const float* __restrict__ s, uint16_t* __restrict__ sdh,
                                                              uint16_t* __restrict__ sdl, uint16_t* __restrict__ dh,
                                                              uint16_t* __restrict__ dl, int64_t ldo, int64_t rows,
                                                              int64_t cols, int64_t tiles_c) {
    __shared__ float td[64][65];
    __shared__ float ts[64];
    const int64_t tr = blockIdx.x / tiles_c, tc = blockIdx.x % tiles_c;
    const int64_t r0 = tr * 64, c0 = tc * 64;
    const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
    for (int rr = ty; rr < 64; rr += 4) {
        const int64_t r = r0 + rr, c = c0 + tx;
        float v = 0.f;
        if (r < rows && c < cols) v = bf2f(Xh[r * ldi + c]) - bf2f(X[r * ldi + c]);
        td[rr][tx] = v;
    }
    if (threadIdx.x < 64) {
        const int64_t r = r0 + threadIdx.x;
        ts[threadIdx.x] = (s && r < rows) ? s[r] : 1.f;
    }
    __syncthreads();
    for (int cc = ty; cc < 64; cc += 4) {
        const int64_t c = c0 + cc, r = r0 + tx;
        if (r < rows && c < cols) {
            const float d = td[tx][cc];
            uint16_t hi, lo;
            split_bf16(d * ts[tx], hi, lo);
            sdh[c * ldo + r] = hi;
            sdl[c * ldo + r] = lo;
            split_bf16(d, hi, lo);
            dh[c * ldo + r] = hi;
            dl[c * ldo + r] = lo;
        }
    }
}

hipError_t transpose_delta_split(const uint16_t* Xh, const uint16_t* X, int64_t ldi, const float* s, uint16_t* sdh,
                                 uint16_t* sdl, uint16_t* dh, uint16_t* dl, int64_t ldo, int64_t rows, int64_t cols,
                                 hipStream_t st) {
    if (rows <= 0 || cols <= 0) return hipSuccess;
    const int64_t tr = (rows + 63) / 64, tc = (cols + 63) / 64;
    hipLaunchKernelGGL(transpose_delta_kernel, dim3((unsigned)(tr * tc)), dim3(256), 0, st, Xh, X, ldi, s, sdh, sdl,
                       dh, dl, ldo, rows, cols, tc);
    return hipGetLastError();
}

// hi/lo bf16 pair of float(in[i])
__global__ void split_f64_kernel(const double* __restrict__ in, uint16_t* __restrict__ hi, uint16_t* __restrict__ lo,
                                 int64_t count) {
    for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < count; e += (int64_t)gridDim.x * blockDim.x) {
        uint16_t h, l;
        split_bf16((float)in[e], h, l);
        hi[e] = h;
        lo[e] = l;
    }
}

hipError_t split_f64(const double* in, uint16_t* hi, uint16_t* lo, int64_t count, hipStream_t st) {
    if (count <= 0) return hipSuccess;
    hipLaunchKernelGGL(split_f64_kernel, dim3(grid_for(count, 4)), dim3(TB), 0, st, in, hi, lo, count);
    return hipGetLastError();
}

__device__ __forceinline__ void split3(float x, uint16_t& h, uint16_t& l, uint16_t& l2) {
    h = f2bf(x);
    const float r1 = x - bf2f(h);
    l = f2bf(r1);
    l2 = f2bf(r1 - bf2f(l));
}

__global__ void split3_f64_kernel(const double* __restrict__ in, uint16_t* __restrict__ hi, uint16_t* __restrict__ lo,
                                  uint16_t* __restrict__ lo2, int64_t count) {
    for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < count; e += (int64_t)gridDim.x * blockDim.x)
        split3((float)in[e], hi[e], lo[e], lo2[e]);
}

hipError_t split3_f64(const double* in, uint16_t* hi, uint16_t* lo, uint16_t* lo2, int64_t count, hipStream_t st) {
    if (count <= 0) return hipSuccess;
    hipLaunchKernelGGL(split3_f64_kernel, dim3(grid_for(count, 4)), dim3(TB), 0, st, in, hi, lo, lo2, count);
    return hipGetLastError();
}

__global__ void split3_f32_kernel(const float* __restrict__ A, int64_t lda, uint16_t* __restrict__ hi,
                                  uint16_t* __restrict__ lo, uint16_t* __restrict__ lo2, int64_t ld, int64_t cols,
                                  int64_t total) {
    for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < total; e += (int64_t)gridDim.x * blockDim.x) {
        const int64_t i = e / cols, j = e % cols;
        const int64_t o = i * ld + j;
        split3(A[i * lda + j], hi[o], lo[o], lo2[o]);
    }
}

hipError_t split3_f32(const float* A, int64_t lda, uint16_t* hi, uint16_t* lo, uint16_t* lo2, int64_t ld,
                      int64_t rows, int64_t cols, hipStream_t st) {
    const int64_t total = rows * cols;
    if (total <= 0) return hipSuccess;
    hipLaunchKernelGGL(split3_f32_kernel, dim3(grid_for(total, 4)), dim3(TB), 0, st, A, lda, hi, lo, lo2, ld, cols,
                       total);
    return hipGetLastError();
}

// flag |= 1 when any of the count bf16 values is nonzero (either sign of zero counts as zero)
__global__ void any_nonzero_u16_kernel(const uint16_t* __restrict__ p, int64_t count, int* __restrict__ flag) {
    uint32_t any = 0;
    for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < count; e += (int64_t)gridDim.x * blockDim.x)
        any |= p[e] & 0x7FFFu;
    if (any) atomicOr(flag, 1);
}

hipError_t any_nonzero_u16(const uint16_t* p, int64_t count, int* flag, hipStream_t st) {
    if (count <= 0) return hipSuccess;
    hipLaunchKernelGGL(any_nonzero_u16_kernel, dim3(grid_for(count, 8)), dim3(TB), 0, st, p, count, flag);
    return hipGetLastError();
}

// G[i][j] = C0[i][c1 + j] + P[i][c1 + j]   (m x w, C0 and P with row stride ld)
__global__ void gram_grad_kernel(const float* __restrict__ C0, const float* __restrict__ P, int64_t ld, int64_t c1,
                                 int64_t w, int64_t total, float* __restrict__ G) {
    for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < total; e += (int64_t)gridDim.x * blockDim.x) {
        const int64_t i = e / w, j = c1 + e % w;
        G[e] = C0[i * ld + j] + P[i * ld + j];
    }
}

hipError_t gram_grad(const float* C0, const float* P, int64_t ld, int64_t c1, int64_t m, int64_t w, float* G,
                     hipStream_t st) {
    const int64_t total = m * w;
    if (total <= 0) return hipSuccess;
    hipLaunchKernelGGL(gram_grad_kernel, dim3(grid_for(total, 4)), dim3(TB), 0, st, C0, P, ld, c1, w, total, G);
    return hipGetLastError();
}

// out = A - double(B) (float64 minus float32, elementwise)
__global__ void sub_f64_f32_kernel(const double* __restrict__ A, const float* __restrict__ B, double* __restrict__ out,
                                   int64_t count) {
    for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < count; e += (int64_t)gridDim.x * blockDim.x)
        out[e] = A[e] - (double)B[e];
}

hipError_t sub_f64_f32(const double* A, const float* B, double* out, int64_t count, hipStream_t st) {
    if (count <= 0) return hipSuccess;
    hipLaunchKernelGGL(sub_f64_f32_kernel, dim3(grid_for(count, 4)), dim3(TB), 0, st, A, B, out, count);
    return hipGetLastError();
}

// Deterministic dot product of two float64 arrays: each of DOT_BLOCKS blocks sums a fixed
// strided subset in a fixed order and reduces it in a fixed tree; partials[b] receives it.
constexpr int DOT_BLOCKS = 1024;
__global__ __launch_bounds__(256) void dot_f64_kernel(const double* __restrict__ X, const double* __restrict__ Y,
                                                      int64_t count, double* __restrict__ partials) {
    __shared__ double red[256];
    double acc = 0.0;
    for (int64_t e = blockIdx.x * 256 + threadIdx.x; e < count; e += (int64_t)DOT_BLOCKS * 256) acc += X[e] * Y[e];
    red[threadIdx.x] = acc;
    __syncthreads();
    for (int st = 128; st > 0; st >>= 1) {
        if (threadIdx.x < st) red[threadIdx.x] += red[threadIdx.x + st];
        __syncthreads();
    }
    if (threadIdx.x == 0) partials[blockIdx.x] = red[0];
}

// Gram form of a BGD step: sum over all weights of (2 C0 + P) (W - W0), same fixed-order
// partials as dot_f64.
__global__ __launch_bounds__(256) void dot_gram_kernel(const float* __restrict__ C0, const float* __restrict__ P,
                                                       const double* __restrict__ W, const float* __restrict__ W0,
                                                       int64_t count, double* __restrict__ partials) {
    __shared__ double red[256];
    double acc = 0.0;
    for (int64_t e = blockIdx.x * 256 + threadIdx.x; e < count; e += (int64_t)DOT_BLOCKS * 256)
        acc += (2.0 * (double)C0[e] + (double)P[e]) * (W[e] - (double)W0[e]);
    red[threadIdx.x] = acc;
    __syncthreads();
    for (int st = 128; st > 0; st >>= 1) {
        if (threadIdx.x < st) red[threadIdx.x] += red[threadIdx.x + st];
        __syncthreads();
    }
    if (threadIdx.x == 0) partials[blockIdx.x] = red[0];
}

hipError_t dot_gram(const float* C0, const float* P, const double* W, const float* W0, int64_t count,
                    double* partials, hipStream_t st) {
    hipLaunchKernelGGL(dot_gram_kernel, dim3(DOT_BLOCKS), dim3(256), 0, st, C0, P, W, W0, count, partials);
    return hipGetLastError();
}

hipError_t dot_f64(const double* X, const double* Y, int64_t count, double* partials, hipStream_t st) {
    hipLaunchKernelGGL(dot_f64_kernel, dim3(DOT_BLOCKS), dim3(256), 0, st, X, Y, count, partials);
    return hipGetLastError();
}
int64_t dot_f64_partials() { return DOT_BLOCKS; }

__global__ __launch_bounds__(256) void transpose_f32_kernel(const float* __restrict__ in, int64_t ldi,
                                                            float* __restrict__ out, int64_t ldo, int64_t rows,
                                                            int64_t cols, int64_t tiles_c) {
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
        if (r < rows && c < cols) out[c * ldo + r] = tile[tx][cc];
    }
}

hipError_t transpose_f32(const float* in, int64_t ldi, float* out, int64_t ldo, int64_t rows, int64_t cols,
                         hipStream_t st) {
    if (rows <= 0 || cols <= 0) return hipSuccess;
    const int64_t tr = (rows + 63) / 64, tc = (cols + 63) / 64;
    hipLaunchKernelGGL(transpose_f32_kernel, dim3((unsigned)(tr * tc)), dim3(256), 0, st, in, ldi, out, ldo, rows,
                       cols, tc);
    return hipGetLastError();
}

// ---------------------------------------------------------------- splits
__global__ void split_diff_f32_kernel(const float* __restrict__ A, int64_t lda, const float* __restrict__ Bm,
                                      int64_t ldb, uint16_t* __restrict__ hi, uint16_t* __restrict__ lo, int64_t ld,
                                      int64_t rows, int64_t cols) {
    const int64_t total = rows * cols;
    for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < total; e += (int64_t)gridDim.x * blockDim.x) {
        int64_t i = e / cols, j = e % cols;
        float v = A[i * lda + j];
        if (Bm) v -= Bm[i * ldb + j];
        uint16_t h, l;
        split_bf16(v, h, l);
        hi[i * ld + j] = h;
        lo[i * ld + j] = l;
    }
}

__global__ void split_diff_f64_kernel(const double* __restrict__ A, int64_t lda, const float* __restrict__ Bm,
                                      int64_t ldb, uint16_t* __restrict__ hi, uint16_t* __restrict__ lo, int64_t ld,
                                      int64_t rows, int64_t cols) {
    const int64_t total = rows * cols;
    for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < total; e += (int64_t)gridDim.x * blockDim.x) {
        const int64_t i = e / cols, j = e % cols;
        const float v = (float)(A[i * lda + j] - (double)Bm[i * ldb + j]);
        uint16_t h, l;
        split_bf16(v, h, l);
        hi[i * ld + j] = h;
        lo[i * ld + j] = l;
    }
}

hipError_t split_diff_f64(const double* A, int64_t lda, const float* Bm, int64_t ldb, uint16_t* hi, uint16_t* lo,
                          int64_t ld, int64_t rows, int64_t cols, hipStream_t st) {
    const int64_t total = rows * cols;
    if (total <= 0) return hipSuccess;
    hipLaunchKernelGGL(split_diff_f64_kernel, dim3(grid_for(total, 4)), dim3(TB), 0, st, A, lda, Bm, ldb, hi, lo, ld,
                       rows, cols);
    return hipGetLastError();
}

__global__ void widen_kernel(const float* __restrict__ in, double* __restrict__ out, int64_t count) {
    for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < count; e += (int64_t)gridDim.x * blockDim.x)
        out[e] = (double)in[e];
}

__global__ void narrow_kernel(const double* __restrict__ in, float* __restrict__ out, int64_t count) {
    for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < count; e += (int64_t)gridDim.x * blockDim.x)
        out[e] = (float)in[e];
}

hipError_t widen_f32(const float* in, double* out, int64_t count, hipStream_t st) {
    if (count <= 0) return hipSuccess;
    hipLaunchKernelGGL(widen_kernel, dim3(grid_for(count, 4)), dim3(TB), 0, st, in, out, count);
    return hipGetLastError();
}

hipError_t narrow_f64(const double* in, float* out, int64_t count, hipStream_t st) {
    if (count <= 0) return hipSuccess;
    hipLaunchKernelGGL(narrow_kernel, dim3(grid_for(count, 4)), dim3(TB), 0, st, in, out, count);
    return hipGetLastError();
}

hipError_t split_diff_f32(const float* A, int64_t lda, const float* Bm, int64_t ldb, uint16_t* hi, uint16_t* lo,
                          int64_t ld, int64_t rows, int64_t cols, hipStream_t st) {
    if (rows <= 0 || cols <= 0) return hipSuccess;
    hipLaunchKernelGGL(split_diff_f32_kernel, dim3(grid_for(rows * cols, 4)), dim3(TB), 0, st, A, lda, Bm, ldb, hi, lo,
                       ld, rows, cols);
    return hipGetLastError();
}

// Blended metric of Eq. slide_window as a bf16 pair: x = alpha (M or I)[i][k] + (1 - alpha) P[i][k]
// (P may be NULL), hi = bf16(x), lo = bf16(x - hi); m x m, row-major.
__global__ void blend_split_kernel(const float* __restrict__ M, const float* __restrict__ P, float alpha, int64_t m,
                                   uint16_t* __restrict__ hi, uint16_t* __restrict__ lo) {
    const int64_t total = m * m;
    for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < total; e += (int64_t)gridDim.x * blockDim.x) {
        const int64_t i = e / m, k = e % m;
        float v = alpha * (M ? M[e] : (i == k ? 1.f : 0.f));
        if (P) v += (1.f - alpha) * P[e];
        uint16_t h, l;
        split_bf16(v, h, l);
        hi[e] = h;
        lo[e] = l;
    }
}

hipError_t blend_split(const float* M, const float* P, float alpha, int64_t m, uint16_t* hi, uint16_t* lo,
                       hipStream_t st) {
    if (m <= 0) return hipSuccess;
    hipLaunchKernelGGL(blend_split_kernel, dim3(grid_for(m * m, 4)), dim3(TB), 0, st, M, P, alpha, m, hi, lo);
    return hipGetLastError();
}

__global__ void split_diff_bf16_kernel(const uint16_t* __restrict__ a, const uint16_t* __restrict__ b,
                                       uint16_t* __restrict__ hi, uint16_t* __restrict__ lo, int64_t count) {
    for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < count; e += (int64_t)gridDim.x * blockDim.x) {
        float v = bf2f(a[e]) - bf2f(b[e]);  // exact in float32 for bf16 inputs of similar magnitude
        uint16_t h, l;
        split_bf16(v, h, l);
        hi[e] = h;
        lo[e] = l;
    }
}

hipError_t split_diff_bf16(const uint16_t* a, const uint16_t* b, uint16_t* hi, uint16_t* lo, int64_t count,
                           hipStream_t st) {
    if (count <= 0) return hipSuccess;
    hipLaunchKernelGGL(split_diff_bf16_kernel, dim3(grid_for(count, 4)), dim3(TB), 0, st, a, b, hi, lo, count);
    return hipGetLastError();
}

// ---------------------------------------------------------------- deterministic reduction
__global__ __launch_bounds__(256) void reduce_partials_kernel(const double* __restrict__ p, int64_t count,
                                                              double scale, double* out) {
    __shared__ double red[256];
    double acc = 0.0;
    for (int64_t i = threadIdx.x; i < count; i += 256) acc += p[i];
    red[threadIdx.x] = acc;
    __syncthreads();
    for (int s = 128; s > 0; s >>= 1) {
        if (threadIdx.x < s) red[threadIdx.x] += red[threadIdx.x + s];
        __syncthreads();
    }
    if (threadIdx.x == 0) *out = red[0] * scale;
}

hipError_t reduce_partials(const double* partials, int64_t count, double scale, double* out, hipStream_t st) {
    hipLaunchKernelGGL(reduce_partials_kernel, dim3(1), dim3(256), 0, st, partials, count, scale, out);
    return hipGetLastError();
}

// ---------------------------------------------------------------- split-K reduction + Adam
// Bias-corrected Adam in the Kingma-Ba form: m = b1 m + (1-b1) g, v = b2 v + (1-b2) g^2,
// w -= lr * (m * bc1) / (sqrt(v * bc2) + eps).  The moments and the step are float32; the
// step is added to the float64 working weight.
__device__ __forceinline__ void adam_elem(const AdamArgs& a, int64_t i, int64_t j, float g) {
    const int64_t idx = i * a.n + j;
    float mv = a.beta1 * a.mA[idx] + (1.f - a.beta1) * g;
    float vv = a.beta2 * a.vA[idx] + (1.f - a.beta2) * g * g;
    a.mA[idx] = mv;
    a.vA[idx] = vv;
    float mh = mv * a.bc1;
    float vh = vv * a.bc2;
    const float step = a.lr * mh / (sqrtf(vh) + a.eps);
    const double w = a.W[idx] - (double)step;
    a.W[idx] = w;
    if (a.Dacc) {
        const float d = (a.inc_reset ? 0.f : a.Dacc[idx]) - step;
        a.Dacc[idx] = d;
        a.Dinc[idx] = f2bf(d);
    }
    if (!a.Dhi) return;
    uint16_t h, l;
    split_bf16((float)(w - (double)a.W0[idx]), h, l);
    a.Dhi[idx] = h;
    a.Dlo[idx] = l;
}

__global__ void adam_kernel(AdamArgs a) {
    const int64_t w = a.n - a.c1;
    const int64_t total = a.m * w;
    const int64_t zstride = a.m * w;
    for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < total; e += (int64_t)gridDim.x * blockDim.x) {
        float g = 0.f;
        for (int64_t z = 0; z < a.splits; ++z) g += a.Gp[z * zstride + e];
        if (a.g0_mode == 2) g += a.G0[e];
        else if (a.g0_mode == 1) a.G0[e] = g;
        g *= a.gscale;
        int64_t i = e / w, j = a.c1 + e % w;
        adam_elem(a, i, j, g);
    }
}

hipError_t adam_update(const AdamArgs& a, hipStream_t st) {
    const int64_t total = a.m * (a.n - a.c1);
    if (total <= 0) return hipSuccess;
    hipLaunchKernelGGL(adam_kernel, dim3(grid_for(total, 4)), dim3(TB), 0, st, a);
    return hipGetLastError();
}

// The cross term <G0, Dinc> in fixed-order per-block float64 sums, then one block adds it to L0
// and the partial sums of s_t acc^2.
constexpr int INC_DOT_BLOCKS = 512;
__global__ __launch_bounds__(256) void inc_dot_kernel(const float* __restrict__ G0, const uint16_t* __restrict__ Dinc,
                                                      int64_t ldd, int64_t m, int64_t w, double* __restrict__ dots) {
    __shared__ double red[256];
    double acc = 0.0;
    for (int64_t i = blockIdx.x; i < m; i += INC_DOT_BLOCKS) {  // rows, coalesced along each
        const float* g = G0 + i * w;
        const uint16_t* d = Dinc + i * ldd;
        for (int64_t j = threadIdx.x; j < w; j += 256) acc += (double)g[j] * (double)bf2f(d[j]);
    }
    red[threadIdx.x] = acc;
    __syncthreads();
    for (int k = 128; k > 0; k >>= 1) {
        if (threadIdx.x < k) red[threadIdx.x] += red[threadIdx.x + k];
        __syncthreads();
    }
    if (threadIdx.x == 0) dots[blockIdx.x] = red[0];
}

__global__ __launch_bounds__(256) void inc_loss_kernel(const double* __restrict__ L0, const double* __restrict__ dots,
                                                       const double* __restrict__ parts, int64_t nparts, double T,
                                                       double* __restrict__ out) {
    __shared__ double rd[256], rp[256];
    double d = 0.0, p = 0.0;
    for (int64_t k = threadIdx.x; k < INC_DOT_BLOCKS; k += 256) d += dots[k];
    for (int64_t k = threadIdx.x; k < nparts; k += 256) p += parts[k];
    rd[threadIdx.x] = d;
    rp[threadIdx.x] = p;
    __syncthreads();
    for (int k = 128; k > 0; k >>= 1) {
        if (threadIdx.x < k) {
            rd[threadIdx.x] += rd[threadIdx.x + k];
            rp[threadIdx.x] += rp[threadIdx.x + k];
        }
        __syncthreads();
    }
    if (threadIdx.x == 0) *out = *L0 + rd[0] / T + 0.5 / T * rp[0];
}

int64_t inc_loss_partials() { return INC_DOT_BLOCKS; }

hipError_t inc_loss(const double* L0, const float* G0, const uint16_t* Dinc, int64_t ldd, int64_t m, int64_t w,
                    const double* parts, int64_t nparts, double T, double* dots, double* out, hipStream_t st) {
    hipLaunchKernelGGL(inc_dot_kernel, dim3(INC_DOT_BLOCKS), dim3(256), 0, st, G0, Dinc, ldd, m, w, dots);
    hipLaunchKernelGGL(inc_loss_kernel, dim3(1), dim3(256), 0, st, L0, dots, parts, nparts, T, out);
    return hipGetLastError();
}

__global__ void adam_dense_kernel(AdamArgs a, const float* __restrict__ G) {
    const int64_t w = a.n - a.c1;
    const int64_t total = a.m * w;
    for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < total; e += (int64_t)gridDim.x * blockDim.x) {
        int64_t i = e / w, j = a.c1 + e % w;
        adam_elem(a, i, j, G[e]);
    }
}

hipError_t adam_update_dense(const AdamArgs& a, const float* G, hipStream_t st) {
    const int64_t total = a.m * (a.n - a.c1);
    if (total <= 0) return hipSuccess;
    hipLaunchKernelGGL(adam_dense_kernel, dim3(grid_for(total, 4)), dim3(TB), 0, st, a, G);
    return hipGetLastError();
}

__global__ void reduce_splits_kernel(const float* __restrict__ Gp, int64_t splits, int64_t total, float gscale,
                                     float* __restrict__ G, int accumulate) {
    for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < total; e += (int64_t)gridDim.x * blockDim.x) {
        float g = 0.f;
        for (int64_t z = 0; z < splits; ++z) g += Gp[z * total + e];
        g *= gscale;
        G[e] = accumulate ? G[e] + g : g;
    }
}

hipError_t reduce_splits(const float* Gp, int64_t splits, int64_t m, int64_t w, float gscale, float* G,
                         bool accumulate, hipStream_t st) {
    const int64_t total = m * w;
    if (total <= 0) return hipSuccess;
    hipLaunchKernelGGL(reduce_splits_kernel, dim3(grid_for(total, 4)), dim3(TB), 0, st, Gp, splits, total, gscale, G,
                       (int)accumulate);
    return hipGetLastError();
}

}  // namespace realq
