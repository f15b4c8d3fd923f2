// Attention half of the block-output surrogate (Sec. 4.2-4.4 with a full decoder block):
// rotary position embedding and causal softmax attention with grouped key/value heads, forward
// and backward.  Sequences of L consecutive tokens; head h reads key/value head h / (H / Hkv).
//
// The contractions run on v_mfma_f32_32x32x16_bf16, one 32 x 32 output tile per wave:
//   scores  S = qr kr^T / sqrt(hd)       bf16 operands, exact products, float32 sums
//   output  O = P v                      P carried as three bf16 terms (all 24 bits)
//   dP = dO v^T                          dO in three bf16 terms (dP - D cancels)
//   dQ = dS kr, dK = dS^T qr, dV = P^T dO   float32 operands as bf16 hi/lo
// The softmax and the row term D_i = sum_j P_ij dP_ij = dO_i . O_i run in float64.  P is kept as
// float32 [S][H][L][L] (zeros above the diagonal within the diagonal tile; tiles above it are not
// written); the backward writes dS, dS^T
// and P^T as bf16 hi/lo pairs for the tiles on or below the diagonal, so every MFMA operand is a
// 16-byte load of 8 consecutive contraction indices.
#include "common.h"
#include "kernels.h"

namespace realq {

namespace {
constexpr int TB = 256;
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

// ---------------------------------------------------------------- MFMA attention
//
// Fragments of v_mfma_f32_32x32x16_bf16 (C = A B^T over one 16-wide k step): a lane supplies 8
// consecutive k (offset 8 (lane / 32)) of row (lane % 32) of A and of B; acc[e] is C[r][c] with
// r = 8 (e / 4) + 4 (lane / 32) + e % 4 and c = lane % 32.
namespace {
constexpr int AT = 32;
constexpr int TSTR = AT + 8;  // bf16 per row of a staged 32 x 32 tile (80 bytes: 16-byte aligned rows)

__device__ __forceinline__ bf16x8 ld8(const uint16_t* p) { return *reinterpret_cast<const bf16x8*>(p); }

__device__ __forceinline__ void split8x3(const float* p, bf16x8& hi, bf16x8& lo, bf16x8& lo2) {
    const f32x4 x0 = *reinterpret_cast<const f32x4*>(p);
    const f32x4 x1 = *reinterpret_cast<const f32x4*>(p + 4);
    u16x8 h, l, l2;
#pragma unroll
    for (int u = 0; u < 8; ++u) {
        const float x = u < 4 ? x0[u] : x1[u - 4];
        h[u] = f2bf(x);
        const float r = x - bf2f(h[u]);
        l[u] = f2bf(r);
        l2[u] = f2bf(r - bf2f(l[u]));
    }
    hi = __builtin_bit_cast(bf16x8, h);
    lo = __builtin_bit_cast(bf16x8, l);
    lo2 = __builtin_bit_cast(bf16x8, l2);
}

__device__ __forceinline__ f32x16 mfma(bf16x8 a, bf16x8 b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ f32x16 zero16() {
    f32x16 z;
#pragma unroll
    for (int e = 0; e < 16; ++e) z[e] = 0.f;
    return z;
}

__device__ __forceinline__ int acc_row(int e, int lane) { return 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3); }

__device__ double block_sum(double v, double* red) {
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
__device__ double block_max(double v, double* red) {
    red[threadIdx.x] = v;
    __syncthreads();
    for (int s = TB / 2; s > 0; s >>= 1) {
        if ((int)threadIdx.x < s) red[threadIdx.x] = fmax(red[threadIdx.x], red[threadIdx.x + s]);
        __syncthreads();
    }
    const double r = red[0];
    __syncthreads();
    return r;
}
}  // namespace

// Raw scaled scores of the causal tiles: grid (S H nt, ceil(nt / 4)), 4 waves, wave w of block y
// takes key tile jt = 4 y + w of query tile it (tiles above the diagonal are skipped).
__global__ __launch_bounds__(256) void attn_scores_kernel(const uint16_t* __restrict__ qr,
                                                          const uint16_t* __restrict__ kr, int64_t H, int64_t Hkv,
                                                          int64_t hd, int64_t L, float* __restrict__ P) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int64_t nt = L / AT;
    const int64_t it = blockIdx.x % nt, sh = blockIdx.x / nt, h = sh % H, s = sh / H;
    const int64_t jt = (int64_t)blockIdx.y * 4 + wave;
    if (jt > it) return;
    const int64_t g = h / (H / Hkv);
    const uint16_t* a = qr + (s * L + it * AT + (lane & 31)) * (H * hd) + h * hd + 8 * (lane >> 5);
    const uint16_t* b = kr + (s * L + jt * AT + (lane & 31)) * (Hkv * hd) + g * hd + 8 * (lane >> 5);
    f32x16 acc = zero16();
    for (int64_t k0 = 0; k0 < hd; k0 += 16) acc = mfma(ld8(a + k0), ld8(b + k0), acc);
    const float scale = (float)(1.0 / sqrt((double)hd));
    float* out = P + (sh * L + it * AT) * L + jt * AT + (lane & 31);
#pragma unroll
    for (int e = 0; e < 16; ++e) out[(int64_t)acc_row(e, lane) * L] = acc[e] * scale;
}

// Row softmax over j <= i in float64, zeros after i up to the end of the diagonal tile (entries
// of tiles above the diagonal are never read).  One block per row.
__global__ __launch_bounds__(256) void attn_softmax_kernel(int64_t L, float* __restrict__ P) {
    __shared__ double red[TB];
    const int64_t row = blockIdx.x, i = row % L;
    const int64_t jend = (i / AT + 1) * AT;
    float* p = P + row * L;
    double mx = -INFINITY;
    for (int64_t j = threadIdx.x; j <= i; j += TB) mx = fmax(mx, (double)p[j]);
    mx = block_max(mx, red);
    double sum = 0.0;
    for (int64_t j = threadIdx.x; j <= i; j += TB) sum += exp((double)p[j] - mx);
    sum = block_sum(sum, red);
    for (int64_t j = threadIdx.x; j < jend; j += TB) p[j] = j <= i ? (float)(exp((double)p[j] - mx) / sum) : 0.f;
}

// O = P v: grid (S H nt, ceil(hd / 32 / 4)), wave w of block y takes value-column tile 4 y + w.
// P rows as three bf16 terms, vt = v^T [Hkv hd][T].  Writes O32 (float32) and O (bf16).
__global__ __launch_bounds__(256) void attn_pv_kernel(const float* __restrict__ P, const uint16_t* __restrict__ vt,
                                                      int64_t T, int64_t H, int64_t Hkv, int64_t hd, int64_t L,
                                                      float* __restrict__ O32, uint16_t* __restrict__ O) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int64_t nt = L / AT;
    const int64_t it = blockIdx.x % nt, sh = blockIdx.x / nt, h = sh % H, s = sh / H;
    const int64_t ct = (int64_t)blockIdx.y * 4 + wave;
    if (ct >= hd / AT) return;
    const int64_t g = h / (H / Hkv);
    const float* a = P + (sh * L + it * AT + (lane & 31)) * L + 8 * (lane >> 5);
    const uint16_t* b = vt + (g * hd + ct * AT + (lane & 31)) * T + s * L + 8 * (lane >> 5);
    f32x16 acc = zero16();
    const int64_t jend = (it + 1) * AT;
    for (int64_t j0 = 0; j0 < jend; j0 += 32) {  // jend is a multiple of 32: two steps per trip
        bf16x8 ah, al, al2, bh, bl, bl2;
        split8x3(a + j0, ah, al, al2);
        split8x3(a + j0 + 16, bh, bl, bl2);
        const bf16x8 v0 = ld8(b + j0), v1 = ld8(b + j0 + 16);
        acc = mfma(ah, v0, acc);
        acc = mfma(al, v0, acc);
        acc = mfma(al2, v0, acc);
        acc = mfma(bh, v1, acc);
        acc = mfma(bl, v1, acc);
        acc = mfma(bl2, v1, acc);
    }
    const int64_t col = h * hd + ct * AT + (lane & 31);
#pragma unroll
    for (int e = 0; e < 16; ++e) {
        const int64_t t = s * L + it * AT + acc_row(e, lane);
        O32[t * H * hd + col] = acc[e];
        O[t * H * hd + col] = f2bf(acc[e]);
    }
}

hipError_t attn_fwd(const uint16_t* qr, const uint16_t* kr, const uint16_t* v, int64_t T, int64_t H, int64_t Hkv,
                    int64_t hd, int64_t L, float* P, float* O32, uint16_t* O, uint16_t* vt, hipStream_t st) {
    if (T <= 0) return hipSuccess;
    const int64_t S = T / L, nt = L / AT;
    hipError_t e = transpose_u16(v, Hkv * hd, vt, T, T, Hkv * hd, st);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(attn_scores_kernel, dim3((unsigned)(S * H * nt), (unsigned)((nt + 3) / 4)), dim3(256), 0, st,
                       qr, kr, H, Hkv, hd, L, P);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(attn_softmax_kernel, dim3((unsigned)(S * H * L)), dim3(TB), 0, st, L, P);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(attn_pv_kernel, dim3((unsigned)(S * H * nt), (unsigned)((hd / AT + 3) / 4)), dim3(256), 0, st,
                       P, vt, T, H, Hkv, hd, L, O32, O);
    return hipGetLastError();
}

// D[t][h] = sum_c dO[t][h hd + c] O32[t][h hd + c] (float64); one thread per (t, h).
__global__ void attn_rowdot_kernel(const float* __restrict__ dO, const float* __restrict__ O32, int64_t TH,
                                   int64_t hd, double* __restrict__ D) {
    for (int64_t r = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; r < TH; r += (int64_t)gridDim.x * blockDim.x) {
        const float* a = dO + r * hd;
        const float* b = O32 + r * hd;
        double acc = 0.0;
        for (int64_t c = 0; c < hd; ++c) acc += (double)a[c] * (double)b[c];
        D[r] = acc;
    }
}

// dS = P o (dP - D), dP = dO v^T (dO in three bf16 terms), for the causal tiles (same grid as the scores);
// writes dS [i][j], dS^T and P^T [j][i] as bf16 hi/lo.
__global__ __launch_bounds__(256) void attn_ds_kernel(const float* __restrict__ P, const float* __restrict__ dO,
                                                      const uint16_t* __restrict__ v, const double* __restrict__ D,
                                                      int64_t H, int64_t Hkv, int64_t hd, int64_t L,
                                                      uint16_t* __restrict__ dSh, uint16_t* __restrict__ dSl,
                                                      uint16_t* __restrict__ dSth, uint16_t* __restrict__ dStl,
                                                      uint16_t* __restrict__ Pth, uint16_t* __restrict__ Ptl) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int64_t nt = L / AT;
    const int64_t it = blockIdx.x % nt, sh = blockIdx.x / nt, h = sh % H, s = sh / H;
    const int64_t jt = (int64_t)blockIdx.y * 4 + wave;
    if (jt > it) return;
    const int64_t g = h / (H / Hkv);
    const float* a = dO + (s * L + it * AT + (lane & 31)) * (H * hd) + h * hd + 8 * (lane >> 5);
    const uint16_t* b = v + (s * L + jt * AT + (lane & 31)) * (Hkv * hd) + g * hd + 8 * (lane >> 5);
    f32x16 acc = zero16();
    for (int64_t k0 = 0; k0 < hd; k0 += 16) {  // dO in three terms: dP - D cancels
        bf16x8 ah, al, al2;
        split8x3(a + k0, ah, al, al2);
        const bf16x8 bv = ld8(b + k0);
        acc = mfma(ah, bv, acc);
        acc = mfma(al, bv, acc);
        acc = mfma(al2, bv, acc);
    }
    // The six bf16 tiles go out through a per-wave LDS tile (transposed there for dS^T and P^T), so
    // every row segment is written as 16-byte stores: lane l then owns 8 consecutive entries of
    // row l / 4 (and of row 16 + l / 4).
    __shared__ __attribute__((aligned(16))) uint16_t stage[4][AT][TSTR];
    uint16_t(*tb)[TSTR] = stage[wave];
    uint16_t vh[16], vl[16], qh[16], ql[16];
#pragma unroll
    for (int e = 0; e < 16; ++e) {
        const int64_t i = it * AT + acc_row(e, lane);
        const float p = P[(sh * L + i) * L + jt * AT + (lane & 31)];
        const float ds = (float)((double)p * ((double)acc[e] - D[(s * L + i) * H + h]));
        split_bf16(ds, vh[e], vl[e]);
        split_bf16(p, qh[e], ql[e]);
    }
    const int r = lane >> 2, c8 = (lane & 3) * 8;
    auto flush = [&](const uint16_t (&v)[16], bool transposed, uint16_t* dst, int64_t row0, int64_t col0) {
#pragma unroll
        for (int e = 0; e < 16; ++e) {
            const int a = acc_row(e, lane), b = lane & 31;
            if (transposed) tb[b][a] = v[e];
            else tb[a][b] = v[e];
        }
        __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
#pragma unroll
        for (int half = 0; half < 2; ++half) {
            const int rr = r + 16 * half;
            *reinterpret_cast<u16x8*>(dst + (sh * L + row0 + rr) * L + col0 + c8) =
                *reinterpret_cast<const u16x8*>(&tb[rr][c8]);
        }
        __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
    };
    flush(vh, false, dSh, it * AT, jt * AT);
    flush(vl, false, dSl, it * AT, jt * AT);
    flush(vh, true, dSth, jt * AT, it * AT);
    flush(vl, true, dStl, jt * AT, it * AT);
    flush(qh, true, Pth, jt * AT, it * AT);
    flush(ql, true, Ptl, jt * AT, it * AT);
}

// dqr = dS kr / sqrt(hd): grid (S H nt, ceil(hd / 32 / 4)); kt = kr^T [Hkv hd][T].
__global__ __launch_bounds__(256) void attn_dq_kernel(const uint16_t* __restrict__ dSh, const uint16_t* __restrict__ dSl,
                                                      const uint16_t* __restrict__ kt, int64_t T, int64_t H,
                                                      int64_t Hkv, int64_t hd, int64_t L, float* __restrict__ dq) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int64_t nt = L / AT;
    const int64_t it = blockIdx.x % nt, sh = blockIdx.x / nt, h = sh % H, s = sh / H;
    const int64_t ct = (int64_t)blockIdx.y * 4 + wave;
    if (ct >= hd / AT) return;
    const int64_t g = h / (H / Hkv);
    const int64_t arow = (sh * L + it * AT + (lane & 31)) * L + 8 * (lane >> 5);
    const uint16_t* b = kt + (g * hd + ct * AT + (lane & 31)) * T + s * L + 8 * (lane >> 5);
    f32x16 acc = zero16();
    const int64_t jend = (it + 1) * AT;
    for (int64_t j0 = 0; j0 < jend; j0 += 32) {  // two steps per trip
        const bf16x8 b0 = ld8(b + j0), b1 = ld8(b + j0 + 16);
        const bf16x8 h0 = ld8(dSh + arow + j0), l0 = ld8(dSl + arow + j0);
        const bf16x8 h1 = ld8(dSh + arow + j0 + 16), l1 = ld8(dSl + arow + j0 + 16);
        acc = mfma(h0, b0, acc);
        acc = mfma(l0, b0, acc);
        acc = mfma(h1, b1, acc);
        acc = mfma(l1, b1, acc);
    }
    const float scale = (float)(1.0 / sqrt((double)hd));
    const int64_t col = h * hd + ct * AT + (lane & 31);
#pragma unroll
    for (int e = 0; e < 16; ++e) dq[(s * L + it * AT + acc_row(e, lane)) * H * hd + col] = acc[e] * scale;
}

// dkr = sum_h dS^T qr / sqrt(hd), dv = sum_h P^T dO over the query heads of key/value head g:
// grid (S Hkv nt, ceil(hd / 32 / 4)); qt = qr^T [H hd][T], dOt = dO^T as hi/lo [H hd][T].
__global__ __launch_bounds__(256) void attn_dkv_kernel(const uint16_t* __restrict__ dSth,
                                                       const uint16_t* __restrict__ dStl,
                                                       const uint16_t* __restrict__ Pth, const uint16_t* __restrict__ Ptl,
                                                       const uint16_t* __restrict__ qt,
                                                       const uint16_t* __restrict__ dOth,
                                                       const uint16_t* __restrict__ dOtl, int64_t T, int64_t H,
                                                       int64_t Hkv, int64_t hd, int64_t L, float* __restrict__ dk,
                                                       float* __restrict__ dv) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int64_t nt = L / AT;
    const int64_t jt = blockIdx.x % nt, sg = blockIdx.x / nt, g = sg % Hkv, s = sg / Hkv;
    const int64_t ct = (int64_t)blockIdx.y * 4 + wave;
    if (ct >= hd / AT) return;
    const int64_t rep = H / Hkv;
    f32x16 ak = zero16(), av = zero16();
    for (int64_t hh = 0; hh < rep; ++hh) {
        const int64_t h = g * rep + hh, sh = s * H + h;
        const int64_t arow = (sh * L + jt * AT + (lane & 31)) * L + 8 * (lane >> 5);
        const int64_t brow = (h * hd + ct * AT + (lane & 31)) * T + s * L + 8 * (lane >> 5);
        for (int64_t i0 = jt * AT; i0 < L; i0 += 32) {  // L - jt 32 is a multiple of 32: two steps per trip
            bf16x8 q[2], sh_[2], sl[2], ph[2], pl[2], doh[2], dol[2];
#pragma unroll
            for (int u = 0; u < 2; ++u) {
                const int64_t k = i0 + 16 * u;
                q[u] = ld8(qt + brow + k);
                sh_[u] = ld8(dSth + arow + k);
                sl[u] = ld8(dStl + arow + k);
                ph[u] = ld8(Pth + arow + k);
                pl[u] = ld8(Ptl + arow + k);
                doh[u] = ld8(dOth + brow + k);
                dol[u] = ld8(dOtl + brow + k);
            }
#pragma unroll
            for (int u = 0; u < 2; ++u) {
                ak = mfma(sh_[u], q[u], ak);
                ak = mfma(sl[u], q[u], ak);
                av = mfma(ph[u], doh[u], av);
                av = mfma(pl[u], doh[u], av);
                av = mfma(ph[u], dol[u], av);
            }
        }
    }
    const float scale = (float)(1.0 / sqrt((double)hd));
    const int64_t col = g * hd + ct * AT + (lane & 31);
#pragma unroll
    for (int e = 0; e < 16; ++e) {
        const int64_t t = s * L + jt * AT + acc_row(e, lane);
        dk[t * Hkv * hd + col] = ak[e] * scale;
        dv[t * Hkv * hd + col] = av[e];
    }
}

hipError_t attn_bwd(const float* P, const float* O32, const float* dO, const uint16_t* qr, const uint16_t* kr,
                    const uint16_t* v, int64_t T, int64_t H, int64_t Hkv, int64_t hd, int64_t L, const AttnScratch& w,
                    float* dq, float* dk, float* dv, hipStream_t st) {
    if (T <= 0) return hipSuccess;
    const int64_t S = T / L, nt = L / AT;
    hipError_t e;
    hipLaunchKernelGGL(attn_rowdot_kernel, dim3(grid_of(T * H)), dim3(TB), 0, st, dO, O32, T * H, hd, w.D);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if ((e = transpose_u16(kr, Hkv * hd, w.kt, T, T, Hkv * hd, st)) != hipSuccess) return e;
    if ((e = transpose_u16(qr, H * hd, w.qt, T, T, H * hd, st)) != hipSuccess) return e;
    if ((e = transpose_split_f32(dO, H * hd, w.dOth, w.dOtl, T, T, H * hd, st)) != hipSuccess) return e;
    hipLaunchKernelGGL(attn_ds_kernel, dim3((unsigned)(S * H * nt), (unsigned)((nt + 3) / 4)), dim3(256), 0, st, P, dO,
                       v, w.D, H, Hkv, hd, L, w.dSh, w.dSl, w.dSth, w.dStl, w.Pth, w.Ptl);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    const unsigned cy = (unsigned)((hd / AT + 3) / 4);
    hipLaunchKernelGGL(attn_dq_kernel, dim3((unsigned)(S * H * nt), cy), dim3(256), 0, st, w.dSh, w.dSl, w.kt, T, H,
                       Hkv, hd, L, dq);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(attn_dkv_kernel, dim3((unsigned)(S * Hkv * nt), cy), dim3(256), 0, st, w.dSth, w.dStl, w.Pth,
                       w.Ptl, w.qt, w.dOth, w.dOtl, T, H, Hkv, hd, L, dk, dv);
    return hipGetLastError();
}

}  // namespace realq
