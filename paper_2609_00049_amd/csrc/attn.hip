// Attention half of the block-output surrogate (Sec. 4.2-4.4 with a full decoder block):
// rotary position embedding and causal softmax attention with grouped key/value heads, forward
// and backward.  Sequences of L consecutive tokens; head h reads key/value head h / (H / Hkv).
// Scores, softmax and the value sums run in float64 (one block per query row, or per key row for
// the key/value gradients) so that the bf16 roundings of the block fall where exact arithmetic
// puts them; the probabilities and score gradients are kept as float32 [S][H][L][L] with zeros
// above the diagonal.
#include "common.h"
#include "kernels.h"

namespace realq {

namespace {
constexpr int TB = 256;
__device__ __forceinline__ double block_reduce(double v, double* red, bool is_max) {
    red[threadIdx.x] = v;
    __syncthreads();
    for (int s = TB / 2; s > 0; s >>= 1) {
        if ((int)threadIdx.x < s)
            red[threadIdx.x] = is_max ? fmax(red[threadIdx.x], red[threadIdx.x + s]) : red[threadIdx.x] + red[threadIdx.x + s];
        __syncthreads();
    }
    const double r = red[0];
    __syncthreads();
    return r;
}
}  // namespace

// Rotary embedding over pairs (i, i + hd/2) of each head, angle (t mod L) base^(-2i/hd):
//   forward (bf16 in and out):  (x1 c - x2 s, x2 c + x1 s)
//   inverse (float32 in and out): (x1 c + x2 s, x2 c - x1 s)
template <bool FWD, typename TI, typename TO>
__global__ void rope_kernel(const TI* __restrict__ in, TO* __restrict__ out, int64_t T, int64_t n, int64_t hd,
                            int64_t L, double base) {
    const int64_t half = hd / 2, total = T * n * half;
    for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < total; e += (int64_t)gridDim.x * blockDim.x) {
        const int64_t t = e / (n * half), r = e % (n * half), h = r / half, i = r % half;
        const double ang = (double)(t % L) * pow(base, -2.0 * (double)i / (double)hd);
        double s, c;
        sincos(ang, &s, &c);
        const int64_t p = t * n * hd + h * hd + i;
        double x1, x2;
        if constexpr (FWD) {
            x1 = (double)bf2f(in[p]);
            x2 = (double)bf2f(in[p + half]);
            out[p] = f2bf((float)(x1 * c - x2 * s));
            out[p + half] = f2bf((float)(x2 * c + x1 * s));
        } else {
            x1 = (double)in[p];
            x2 = (double)in[p + half];
            out[p] = (float)(x1 * c + x2 * s);
            out[p + half] = (float)(x2 * c - x1 * s);
        }
    }
}

static unsigned grid_of(int64_t count) {
    int64_t b = (count + TB * 4 - 1) / (TB * 4);
    return (unsigned)(b < 1 ? 1 : (b > 65536 ? 65536 : b));
}

hipError_t rope_fwd(const uint16_t* in, uint16_t* out, int64_t T, int64_t n, int64_t hd, int64_t L, double base,
                    hipStream_t st) {
    if (T <= 0) return hipSuccess;
    hipLaunchKernelGGL((rope_kernel<true, uint16_t, uint16_t>), dim3(grid_of(T * n * hd / 2)), dim3(TB), 0, st, in,
                       out, T, n, hd, L, base);
    return hipGetLastError();
}
hipError_t rope_inv(const float* in, float* out, int64_t T, int64_t n, int64_t hd, int64_t L, double base,
                    hipStream_t st) {
    if (T <= 0) return hipSuccess;
    hipLaunchKernelGGL((rope_kernel<false, float, float>), dim3(grid_of(T * n * hd / 2)), dim3(TB), 0, st, in, out,
                       T, n, hd, L, base);
    return hipGetLastError();
}

// P[s][h][i][j] = softmax over j <= i of qr_i . kr_j / sqrt(hd) (zeros for j > i); one block per
// (s, h, i).  qr [T][H hd], kr [T][Hkv hd] bf16.
__global__ __launch_bounds__(256) void attn_probs_kernel(const uint16_t* __restrict__ qr,
                                                         const uint16_t* __restrict__ kr, int64_t H, int64_t Hkv,
                                                         int64_t hd, int64_t L, float* __restrict__ P) {
    extern __shared__ double sh[];  // [hd] query row, then [L] scores
    __shared__ double red[TB];
    double* qs = sh;
    double* sc = sh + hd;
    const int64_t row = blockIdx.x;  // (s * H + h) * L + i
    const int64_t i = row % L, sh_ = row / L, h = sh_ % H, s = sh_ / H;
    const int64_t g = h / (H / Hkv);
    const int64_t tq = s * L + i;
    for (int64_t c = threadIdx.x; c < hd; c += TB) qs[c] = (double)bf2f(qr[tq * H * hd + h * hd + c]);
    __syncthreads();
    const double scale = 1.0 / sqrt((double)hd);
    double mx = -INFINITY;
    for (int64_t j = threadIdx.x; j <= i; j += TB) {
        const uint16_t* kj = kr + (s * L + j) * Hkv * hd + g * hd;
        double acc = 0.0;
        for (int64_t c = 0; c < hd; ++c) acc += qs[c] * (double)bf2f(kj[c]);
        sc[j] = acc * scale;
        mx = fmax(mx, sc[j]);
    }
    mx = block_reduce(mx, red, true);
    double sum = 0.0;
    for (int64_t j = threadIdx.x; j <= i; j += TB) {
        const double e = exp(sc[j] - mx);
        sc[j] = e;
        sum += e;
    }
    sum = block_reduce(sum, red, false);
    float* prow = P + row * L;
    for (int64_t j = threadIdx.x; j < L; j += TB) prow[j] = j <= i ? (float)(sc[j] / sum) : 0.f;
}

// O[t][h hd + c] = bf16(sum_{j <= i} P[s][h][i][j] v[s L + j][g hd + c]); one block per (s, h, i).
__global__ __launch_bounds__(256) void attn_out_kernel(const float* __restrict__ P, const uint16_t* __restrict__ v,
                                                       int64_t H, int64_t Hkv, int64_t hd, int64_t L,
                                                       uint16_t* __restrict__ O) {
    const int64_t row = blockIdx.x;
    const int64_t i = row % L, sh_ = row / L, h = sh_ % H, s = sh_ / H;
    const int64_t g = h / (H / Hkv);
    const float* prow = P + row * L;
    for (int64_t c = threadIdx.x; c < hd; c += TB) {
        double acc = 0.0;
        for (int64_t j = 0; j <= i; ++j) acc += (double)prow[j] * (double)bf2f(v[(s * L + j) * Hkv * hd + g * hd + c]);
        O[(s * L + i) * H * hd + h * hd + c] = f2bf((float)acc);
    }
}

hipError_t attn_fwd(const uint16_t* qr, const uint16_t* kr, const uint16_t* v, int64_t T, int64_t H, int64_t Hkv,
                    int64_t hd, int64_t L, float* P, uint16_t* O, hipStream_t st) {
    if (T <= 0) return hipSuccess;
    const int64_t rows = (T / L) * H * L;
    const size_t shm = (size_t)(hd + L) * sizeof(double);
    hipLaunchKernelGGL(attn_probs_kernel, dim3((unsigned)rows), dim3(TB), shm, st, qr, kr, H, Hkv, hd, L, P);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(attn_out_kernel, dim3((unsigned)rows), dim3(TB), 0, st, P, v, H, Hkv, hd, L, O);
    return hipGetLastError();
}

// dS[s][h][i][j] = P_ij (dP_ij - sum_j' P_ij' dP_ij'), dP_ij = dO_i . v_j (j <= i; zeros above).
__global__ __launch_bounds__(256) void attn_ds_kernel(const float* __restrict__ P, const float* __restrict__ dO,
                                                      const uint16_t* __restrict__ v, int64_t H, int64_t Hkv,
                                                      int64_t hd, int64_t L, float* __restrict__ dS) {
    extern __shared__ double sh[];  // [hd] dO row, then [L] dP
    __shared__ double red[TB];
    double* dos = sh;
    double* dp = sh + hd;
    const int64_t row = blockIdx.x;
    const int64_t i = row % L, sh_ = row / L, h = sh_ % H, s = sh_ / H;
    const int64_t g = h / (H / Hkv);
    for (int64_t c = threadIdx.x; c < hd; c += TB) dos[c] = (double)dO[(s * L + i) * H * hd + h * hd + c];
    __syncthreads();
    const float* prow = P + row * L;
    double dsum = 0.0;
    for (int64_t j = threadIdx.x; j <= i; j += TB) {
        const uint16_t* vj = v + (s * L + j) * Hkv * hd + g * hd;
        double acc = 0.0;
        for (int64_t c = 0; c < hd; ++c) acc += dos[c] * (double)bf2f(vj[c]);
        dp[j] = acc;
        dsum += (double)prow[j] * acc;
    }
    dsum = block_reduce(dsum, red, false);
    float* drow = dS + row * L;
    for (int64_t j = threadIdx.x; j < L; j += TB) drow[j] = j <= i ? (float)((double)prow[j] * (dp[j] - dsum)) : 0.f;
}

// dqr[t][h hd + c] = sum_{j <= i} dS_ij kr[s L + j][g hd + c] / sqrt(hd); one block per (s, h, i).
__global__ __launch_bounds__(256) void attn_dq_kernel(const float* __restrict__ dS, const uint16_t* __restrict__ kr,
                                                      int64_t H, int64_t Hkv, int64_t hd, int64_t L,
                                                      float* __restrict__ dq) {
    const int64_t row = blockIdx.x;
    const int64_t i = row % L, sh_ = row / L, h = sh_ % H, s = sh_ / H;
    const int64_t g = h / (H / Hkv);
    const float* drow = dS + row * L;
    const double scale = 1.0 / sqrt((double)hd);
    for (int64_t c = threadIdx.x; c < hd; c += TB) {
        double acc = 0.0;
        for (int64_t j = 0; j <= i; ++j) acc += (double)drow[j] * (double)bf2f(kr[(s * L + j) * Hkv * hd + g * hd + c]);
        dq[(s * L + i) * H * hd + h * hd + c] = (float)(acc * scale);
    }
}

// For key/value row j of head g (one block per (s, g, j)), summed over the query heads of g:
//   dkr[j][c] = sum_h sum_{i >= j} dS[h][i][j] qr[i][h hd + c] / sqrt(hd)
//   dv[j][c]  = sum_h sum_{i >= j} P[h][i][j]  dO[i][h hd + c]
__global__ __launch_bounds__(256) void attn_dkv_kernel(const float* __restrict__ P, const float* __restrict__ dS,
                                                       const uint16_t* __restrict__ qr, const float* __restrict__ dO,
                                                       int64_t H, int64_t Hkv, int64_t hd, int64_t L,
                                                       float* __restrict__ dk, float* __restrict__ dv) {
    const int64_t row = blockIdx.x;  // (s * Hkv + g) * L + j
    const int64_t j = row % L, sg = row / L, g = sg % Hkv, s = sg / Hkv;
    const int64_t rep = H / Hkv;
    const double scale = 1.0 / sqrt((double)hd);
    for (int64_t c = threadIdx.x; c < hd; c += TB) {
        double ak = 0.0, av = 0.0;
        for (int64_t hh = 0; hh < rep; ++hh) {
            const int64_t h = g * rep + hh;
            const int64_t base = ((s * H + h) * L) * L + j;  // element [s][h][i][j] = base + i L
            for (int64_t i = j; i < L; ++i) {
                const int64_t t = s * L + i;
                ak += (double)dS[base + i * L] * (double)bf2f(qr[t * H * hd + h * hd + c]);
                av += (double)P[base + i * L] * (double)dO[t * H * hd + h * hd + c];
            }
        }
        dk[(s * L + j) * Hkv * hd + g * hd + c] = (float)(ak * scale);
        dv[(s * L + j) * Hkv * hd + g * hd + c] = (float)av;
    }
}

hipError_t attn_bwd(const float* P, const float* dO, const uint16_t* qr, const uint16_t* kr, const uint16_t* v,
                    int64_t T, int64_t H, int64_t Hkv, int64_t hd, int64_t L, float* dS, float* dq, float* dk,
                    float* dv, hipStream_t st) {
    if (T <= 0) return hipSuccess;
    const int64_t S = T / L;
    const int64_t rows = S * H * L;
    const size_t shm = (size_t)(hd + L) * sizeof(double);
    hipLaunchKernelGGL(attn_ds_kernel, dim3((unsigned)rows), dim3(TB), shm, st, P, dO, v, H, Hkv, hd, L, dS);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(attn_dq_kernel, dim3((unsigned)rows), dim3(TB), 0, st, dS, kr, H, Hkv, hd, L, dq);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(attn_dkv_kernel, dim3((unsigned)(S * Hkv * L)), dim3(TB), 0, st, P, dS, qr, dO, H, Hkv, hd, L,
                       dk, dv);
    return hipGetLastError();
}

}  // namespace realq
