// Attention half of the block-output surrogate (Sec. 4.2-4.4 with a full decoder block):
// rotary position embedding and causal softmax attention with grouped key/value heads, forward
// and backward.  Sequences of L consecutive tokens; head h reads key/value head h / (H / Hkv).
//
// The contractions run on v_mfma_f32_32x32x16_bf16, one 32 x 32 output tile per wave:
//   scores  S = qr kr^T / sqrt(hd)       bf16 operands, exact products, float32 sums
//   output  O = P v                      P carried as three bf16 terms (all 24 bits)
//   dP = dO v^T                          dO in three bf16 terms (dP - D cancels)
//   dQ = dS kr, dK = dS^T qr, dV = P^T dO   float32 operands as bf16 hi/lo
// The softmax (each query row's max and sum in a first pass over its key tiles, the forward keeping
// only the row log-sum-exp; each exponential itself in float32) and the row term
// D_i = sum_j P_ij dP_ij = dO_i . O_i run in float64.  The backward
// recomputes P from the log-sum-exp and writes dS, dS^T and P^T as bf16 hi/lo pairs for the tiles
// on or below the diagonal, so every MFMA operand is a 16-byte load of 8 consecutive contraction
// indices.
#include "common.h"
#include "kernels.h"

namespace realq {

namespace {
constexpr int TB = 256;
}  // namespace

// Rotary embedding over pairs (i, i + hd/2) of each head, angle (t mod L) base^(-2i/hd):
//   forward (bf16 in and out):  (x1 c - x2 s, x2 c + x1 s)
//   inverse (float32 in and out): (x1 c + x2 s, x2 c - x1 s)
// cs [L][hd/2][2]: cos and sin of the angle of each position and pair (float64), computed once by
// rope_table_kernel rather than per element.
__global__ void rope_table_kernel(double* __restrict__ cs, int64_t L, int64_t hd, double base) {
    const int64_t half = hd / 2, total = L * half;
    for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < total; e += (int64_t)gridDim.x * blockDim.x) {
        const int64_t pos = e / half, i = e % half;
        const double ang = (double)pos * pow(base, -2.0 * (double)i / (double)hd);
        double s, c;
        sincos(ang, &s, &c);
        cs[2 * e] = c;
        cs[2 * e + 1] = s;
    }
}

template <bool FWD, typename TI, typename TO>
__global__ void rope_kernel(const TI* __restrict__ in, TO* __restrict__ out, const double* __restrict__ cs, int64_t T,
                            int64_t n, int64_t hd, int64_t L) {
    const int64_t half = hd / 2, total = T * n * half;
    for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < total; e += (int64_t)gridDim.x * blockDim.x) {
        const int64_t t = e / (n * half), r = e % (n * half), h = r / half, i = r % half;
        const double2 sc = *reinterpret_cast<const double2*>(cs + 2 * ((t % L) * half + i));
        const double c = sc.x, s = sc.y;
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

hipError_t rope_table(double* cs, int64_t L, int64_t hd, double base, hipStream_t st) {
    hipLaunchKernelGGL(rope_table_kernel, dim3(grid_of(L * hd / 2)), dim3(TB), 0, st, cs, L, hd, base);
    return hipGetLastError();
}
hipError_t rope_fwd(const uint16_t* in, uint16_t* out, const double* cs, int64_t T, int64_t n, int64_t hd, int64_t L,
                    hipStream_t st) {
    if (T <= 0) return hipSuccess;
    hipLaunchKernelGGL((rope_kernel<true, uint16_t, uint16_t>), dim3(grid_of(T * n * hd / 2)), dim3(TB), 0, st, in,
                       out, cs, T, n, hd, L);
    return hipGetLastError();
}
hipError_t rope_inv(const float* in, float* out, const double* cs, int64_t T, int64_t n, int64_t hd, int64_t L,
                    hipStream_t st) {
    if (T <= 0) return hipSuccess;
    hipLaunchKernelGGL((rope_kernel<false, float, float>), dim3(grid_of(T * n * hd / 2)), dim3(TB), 0, st, in, out,
                       cs, T, n, hd, L);
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
typedef uint16_t u16x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
constexpr int TSTR32 = AT + 4;  // uint32 per row of a staged 32 x 32 tile of hi | lo pairs (144 bytes)

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

__device__ __forceinline__ void split8x3(const float (&x8)[8], bf16x8& hi, bf16x8& lo, bf16x8& lo2) {
    u16x8 h, l, l2;
#pragma unroll
    for (int u = 0; u < 8; ++u) {
        const float x = x8[u];
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

}  // namespace

// Fused forward for one 32-row query tile per wave, in two passes over the key tiles up to the
// diagonal.  Pass 1: scores on MFMA and each row's max and sum of exponentials (lane 2r + h owns
// half h of row r; max and sum in float64, each exponent in float64 and its exponential in
// float32).  Pass 2: the scores again, P = exp(s - max) / sum as three bf16 terms, P v on MFMA.
// Writes O32 = P v, O = bf16(O32) and the row log-sum-exp LSE = max + log(sum) (float64 [T][H]),
// from which the backward recomputes P.  Value columns go in groups of up to CG 32-column tiles
// (one group for head_dim <= 128).  grid (S H ceil(nt / 4)), 4 waves; wave w of block x takes
// query tile nt - 1 - (4 (x mod nq) + w), so the longest rows start first.
constexpr int CG = 4;
__global__ __launch_bounds__(256) void attn_fwd_kernel(const uint16_t* __restrict__ qr,
                                                       const uint16_t* __restrict__ kr,
                                                       const uint16_t* __restrict__ vt, int64_t T, int64_t H,
                                                       int64_t Hkv, int64_t hd, int64_t L, float* __restrict__ O32,
                                                       uint16_t* __restrict__ O, double* __restrict__ LSE) {
    __shared__ float sS[4][AT][AT + 1];
    __shared__ __attribute__((aligned(16))) uint16_t sP[4][3][AT][TSTR];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int64_t nt = L / AT, nq = (nt + 3) / 4;
    const int64_t sh = blockIdx.x / nq, h = sh % H, s = sh / H;
    const int64_t it = nt - 1 - (4 * (int64_t)(blockIdx.x % nq) + wave);
    if (it < 0) return;
    const int64_t g = h / (H / Hkv);
    const int nk = (int)(hd / 16), nct = (int)(hd / AT);
    const double scale = 1.0 / sqrt((double)hd);
    float(*Sw)[AT + 1] = sS[wave];
    uint16_t(*Pw)[AT][TSTR] = sP[wave];
    const int rr = lane >> 1, hh = lane & 1, c32 = lane & 31, k8 = 8 * (lane >> 5);
    const uint16_t* qa = qr + (s * L + it * AT + c32) * (H * hd) + h * hd + k8;
    const uint16_t* kb0 = kr + (s * L + c32) * (Hkv * hd) + g * hd + k8;
    const int64_t kstep = AT * Hkv * hd;  // one key tile further
    // scores of key tile jt into this wave's LDS tile (entries above the diagonal: -inf)
    auto scores = [&](int64_t jt) {
        const uint16_t* kb = kb0 + jt * kstep;
        f32x16 acc = zero16();
        for (int kk = 0; kk < nk; ++kk) acc = mfma(ld8(qa + 16 * kk), ld8(kb + 16 * kk), acc);
        const bool diag = jt == it;
#pragma unroll
        for (int e = 0; e < 16; ++e) {
            const int r = acc_row(e, lane);
            Sw[r][c32] = (diag && c32 > r) ? -INFINITY : acc[e];
        }
        __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
    };
    // pass 1: the row max and sum
    double m_row = -INFINITY, l_row = 0.0;
    for (int64_t jt = 0; jt <= it; ++jt) {
        scores(jt);
        float smax = -INFINITY;  // scaling by a positive constant keeps the order
#pragma unroll
        for (int k = 0; k < 16; ++k) smax = fmaxf(smax, Sw[rr][16 * hh + k]);
        smax = fmaxf(smax, __shfl_xor(smax, 1));
        const double m_new = fmax(m_row, (double)smax * scale);
        double sum = 0.0;
#pragma unroll
        for (int k = 0; k < 16; ++k) sum += (double)expf((float)((double)Sw[rr][16 * hh + k] * scale - m_new));
        sum += __shfl_xor(sum, 1);
        l_row = l_row * exp(m_row - m_new) + sum;
        m_row = m_new;
        __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
    }
    if (hh == 0) LSE[(s * L + it * AT + rr) * H + h] = m_row + log(l_row);
    const double inv_l = 1.0 / l_row;
    // pass 2: P v per group of value-column tiles
    for (int c0 = 0; c0 < nct; c0 += CG) {
        f32x16 oacc[CG];
        const uint16_t* vb[CG];
#pragma unroll
        for (int ct = 0; ct < CG; ++ct) {
            oacc[ct] = zero16();
            vb[ct] = vt + (g * hd + (int64_t)(c0 + ct) * AT + c32) * T + s * L + k8;
        }
        for (int64_t jt = 0; jt <= it; ++jt) {
            scores(jt);
#pragma unroll
            for (int k = 0; k < 16; ++k) {
                const float pf =
                    (float)((double)expf((float)((double)Sw[rr][16 * hh + k] * scale - m_row)) * inv_l);
                const uint16_t ph = f2bf(pf);
                const float r1 = pf - bf2f(ph);
                const uint16_t pl = f2bf(r1);
                Pw[0][rr][16 * hh + k] = ph;
                Pw[1][rr][16 * hh + k] = pl;
                Pw[2][rr][16 * hh + k] = f2bf(r1 - bf2f(pl));
            }
            __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
#pragma unroll
            for (int k2 = 0; k2 < 2; ++k2) {
                const int col = 16 * k2 + k8;
                const bf16x8 ah = ld8(&Pw[0][c32][col]);
                const bf16x8 al = ld8(&Pw[1][c32][col]);
                const bf16x8 al2 = ld8(&Pw[2][c32][col]);
#pragma unroll
                for (int ct = 0; ct < CG; ++ct) {
                    if (c0 + ct >= nct) continue;
                    const bf16x8 bv = ld8(vb[ct] + jt * AT + 16 * k2);
                    oacc[ct] = mfma(ah, bv, oacc[ct]);
                    oacc[ct] = mfma(al, bv, oacc[ct]);
                    oacc[ct] = mfma(al2, bv, oacc[ct]);
                }
            }
            __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
        }
#pragma unroll
        for (int ct = 0; ct < CG; ++ct) {
            if (c0 + ct >= nct) continue;
            const int64_t col = h * hd + (int64_t)(c0 + ct) * AT + c32;
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                const int64_t t = s * L + it * AT + acc_row(e, lane);
                O32[t * H * hd + col] = oacc[ct][e];
                O[t * H * hd + col] = f2bf(oacc[ct][e]);
            }
        }
    }
}

// The same forward with the key and value tiles staged in LDS and shared by the block's four query
// tiles (one per wave, the waves of a block take consecutive query tiles of one head): every key
// tile is loaded once per block with direct-to-LDS 16-byte loads into one of two buffers, the next
// tile's loads overlapping the current tile's work, and each wave keeps its query fragments in
// registers.  Per lane the arithmetic (MFMA order, the float64 statistics, the three-term P) is that
// of attn_fwd_kernel, so the outputs are bitwise the same.  LDS rows are XOR-swizzled by 16-byte
// chunk so the fragment reads (one chunk of 16 or 32 consecutive rows) are free of bank conflicts:
//   key tile   [32 keys][HD] bf16, chunk c of key row r at position c ^ (r mod HD/8)
//   value tile [HD cols][32 keys] bf16 (from v^T), chunk c of row r at c ^ ((r/2 ^ r/8) mod 4)
namespace {
__device__ __forceinline__ void attn_dma16(const void* sbase, uint32_t voff, uint32_t lds) {
    asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(voff), "s"(sbase), "s"(lds)
                 : "memory", "m0");
}
template <int N>
__device__ __forceinline__ void attn_wait_vm() {
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}
__device__ __forceinline__ int vswz(int r) { return ((r >> 1) ^ (r >> 3)) & 3; }
}  // namespace

template <int HD>
__global__ __launch_bounds__(256) void attn_fwd_lds_kernel(const uint16_t* __restrict__ qr,
                                                           const uint16_t* __restrict__ kr,
                                                           const uint16_t* __restrict__ vt, int64_t T, int64_t H,
                                                           int64_t Hkv, int64_t L, float* __restrict__ O32,
                                                           uint16_t* __restrict__ O, double* __restrict__ LSE) {
    constexpr int NK = HD / 16, NCT = HD / AT;
    constexpr int KCH = HD / 8;                // 16-byte chunks per key row
    constexpr int KBYTES = AT * HD * 2, VBYTES = HD * AT * 2;
    constexpr int KDMA = KBYTES / 1024 / 4, VDMA = VBYTES / 1024 / 4;  // 1 KB loads per wave and tile
    static_assert(KDMA >= 1 && VDMA >= 1 && NCT <= CG, "head width");
    __shared__ float sS[4][AT][AT + 1];
    __shared__ __attribute__((aligned(16))) uint16_t sP[4][3][AT][TSTR];
    __shared__ __attribute__((aligned(16))) uint16_t sKV[2][(KBYTES + VBYTES) / 2];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int wv = __builtin_amdgcn_readfirstlane(wave);
    const int64_t nt = L / AT, nq = (nt + 3) / 4;
    const int64_t sh = blockIdx.x / nq, h = sh % H, s = sh / H;
    const int64_t qb = blockIdx.x % nq;
    const int64_t itmax = nt - 1 - 4 * qb;          // the block's longest row of key tiles
    const int64_t it = itmax - wave;                 // this wave's query tile (may be < 0)
    const int64_t g = h / (H / Hkv);
    const double scale = 1.0 / sqrt((double)HD);
    float(*Sw)[AT + 1] = sS[wave];
    uint16_t(*Pw)[AT][TSTR] = sP[wave];
    const int rr = lane >> 1, hh = lane & 1, c32 = lane & 31, k8 = 8 * (lane >> 5);
    const int64_t ldk = Hkv * HD;                    // key row stride (elements)
    const uint16_t* kbase = kr + (s * L) * ldk + g * HD;
    const uint16_t* vbase = vt + (g * HD) * T + s * L;
    const uint32_t lds0 = (uint32_t)(uintptr_t)&sKV[0][0];
    constexpr uint32_t BUFB = KBYTES + VBYTES;
    // this wave's share of key tile jt (and with V, its value tile) into buffer b
    auto load_tile = [&](int64_t jt, int b, bool with_v) {
        const uint32_t kd = lds0 + (uint32_t)b * BUFB;
        const char* kb = reinterpret_cast<const char*>(kbase + jt * AT * ldk);
#pragma unroll
        for (int q = 0; q < KDMA; ++q) {
            const int qi = wv * KDMA + q;                    // 1 KB piece of the tile
            const int row = qi * (1024 / (HD * 2)) + lane / KCH, pos = lane % KCH;
            const int c = pos ^ (row % KCH);
            attn_dma16(kb, (uint32_t)((row * ldk + c * 8) * 2), kd + (uint32_t)qi * 1024);
        }
        if (with_v) {
            const char* vb = reinterpret_cast<const char*>(vbase + jt * AT);
#pragma unroll
            for (int q = 0; q < VDMA; ++q) {
                const int qi = wv * VDMA + q;
                const int row = qi * 16 + (lane >> 2), pos = lane & 3;
                const int c = pos ^ vswz(row);
                attn_dma16(vb, (uint32_t)((row * T + c * 8) * 2), kd + KBYTES + (uint32_t)qi * 1024);
            }
        }
    };
    const bool active0 = it >= 0;
    // query fragments of this wave's tile, kept for both passes
    bf16x8 qf[NK];
    if (active0) {
        const uint16_t* qa = qr + (s * L + it * AT + c32) * (H * HD) + h * HD + k8;
#pragma unroll
        for (int kk = 0; kk < NK; ++kk) qf[kk] = ld8(qa + 16 * kk);
    }
    auto scores = [&](int b, int64_t jt) {
        const uint16_t* kt = &sKV[b][0];
        f32x16 acc = zero16();
#pragma unroll
        for (int kk = 0; kk < NK; ++kk) {
            const int c = 2 * kk + (lane >> 5);
            const bf16x8 bk = ld8(kt + c32 * HD + ((c ^ (c32 % KCH)) * 8));
            acc = mfma(qf[kk], bk, acc);
        }
        const bool diag = jt == it;
#pragma unroll
        for (int e = 0; e < 16; ++e) {
            const int r = acc_row(e, lane);
            Sw[r][c32] = (diag && c32 > r) ? -INFINITY : acc[e];
        }
        __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
    };
    // pass 1: the row max and sum
    double m_row = -INFINITY, l_row = 0.0;
    load_tile(0, 0, false);
    for (int64_t jt = 0; jt <= itmax; ++jt) {
        attn_wait_vm<0>();                 // this wave's share of tile jt has landed
        __syncthreads();                   // every share landed; tile jt-1's buffer is free
        if (jt + 1 <= itmax) load_tile(jt + 1, (int)((jt + 1) & 1), false);
        if (jt <= it) {
            scores((int)(jt & 1), jt);
            float smax = -INFINITY;  // scaling by a positive constant keeps the order
#pragma unroll
            for (int k = 0; k < 16; ++k) smax = fmaxf(smax, Sw[rr][16 * hh + k]);
            smax = fmaxf(smax, __shfl_xor(smax, 1));
            const double m_new = fmax(m_row, (double)smax * scale);
            double sum = 0.0;
#pragma unroll
            for (int k = 0; k < 16; ++k) sum += (double)expf((float)((double)Sw[rr][16 * hh + k] * scale - m_new));
            sum += __shfl_xor(sum, 1);
            l_row = l_row * exp(m_row - m_new) + sum;
            m_row = m_new;
            __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
        }
    }
    if (active0 && hh == 0) LSE[(s * L + it * AT + rr) * H + h] = m_row + log(l_row);
    const double inv_l = 1.0 / l_row;
    // pass 2: P v over the value-column tiles
    f32x16 oacc[NCT];
#pragma unroll
    for (int ct = 0; ct < NCT; ++ct) oacc[ct] = zero16();
    attn_wait_vm<0>();
    __syncthreads();                       // pass 1's reads of both buffers are done
    load_tile(0, 0, true);
    for (int64_t jt = 0; jt <= itmax; ++jt) {
        attn_wait_vm<0>();
        __syncthreads();
        if (jt + 1 <= itmax) load_tile(jt + 1, (int)((jt + 1) & 1), true);
        if (jt <= it) {
            const int b = (int)(jt & 1);
            scores(b, jt);
#pragma unroll
            for (int k = 0; k < 16; ++k) {
                const float pf =
                    (float)((double)expf((float)((double)Sw[rr][16 * hh + k] * scale - m_row)) * inv_l);
                const uint16_t ph = f2bf(pf);
                const float r1 = pf - bf2f(ph);
                const uint16_t pl = f2bf(r1);
                Pw[0][rr][16 * hh + k] = ph;
                Pw[1][rr][16 * hh + k] = pl;
                Pw[2][rr][16 * hh + k] = f2bf(r1 - bf2f(pl));
            }
            __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
            const uint16_t* vtile = &sKV[b][KBYTES / 2];
#pragma unroll
            for (int k2 = 0; k2 < 2; ++k2) {
                const int col = 16 * k2 + k8;
                const bf16x8 ah = ld8(&Pw[0][c32][col]);
                const bf16x8 al = ld8(&Pw[1][c32][col]);
                const bf16x8 al2 = ld8(&Pw[2][c32][col]);
                const int c = 2 * k2 + (lane >> 5);
#pragma unroll
                for (int ct = 0; ct < NCT; ++ct) {
                    const int row = ct * AT + c32;
                    const bf16x8 bv = ld8(vtile + row * AT + ((c ^ vswz(row)) * 8));
                    oacc[ct] = mfma(ah, bv, oacc[ct]);
                    oacc[ct] = mfma(al, bv, oacc[ct]);
                    oacc[ct] = mfma(al2, bv, oacc[ct]);
                }
            }
            __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
        }
    }
    if (!active0) return;
#pragma unroll
    for (int ct = 0; ct < NCT; ++ct) {
        const int64_t col = h * HD + (int64_t)ct * AT + c32;
#pragma unroll
        for (int e = 0; e < 16; ++e) {
            const int64_t t = s * L + it * AT + acc_row(e, lane);
            O32[t * H * HD + col] = oacc[ct][e];
            O[t * H * HD + col] = f2bf(oacc[ct][e]);
        }
    }
}

hipError_t attn_fwd(const uint16_t* qr, const uint16_t* kr, const uint16_t* v, int64_t T, int64_t H, int64_t Hkv,
                    int64_t hd, int64_t L, double* LSE, float* O32, uint16_t* O, uint16_t* vt, hipStream_t st) {
    if (T <= 0) return hipSuccess;
    const int64_t S = T / L, nt = L / AT;
    hipError_t e = transpose_u16(v, Hkv * hd, vt, T, T, Hkv * hd, st);
    if (e != hipSuccess) return e;
    const dim3 grid((unsigned)(S * H * ((nt + 3) / 4)));
    // the LDS-staged kernel where the 32-bit load offsets of a tile fit (rows of v^T are T long)
    const bool lds_ok = (int64_t)hd * T * 2 < (int64_t(1) << 31) && (((uintptr_t)kr | (uintptr_t)vt) & 15) == 0 &&
                        (Hkv * hd) % 8 == 0 && T % 8 == 0;
    if (lds_ok && hd == 128)
        hipLaunchKernelGGL((attn_fwd_lds_kernel<128>), grid, dim3(256), 0, st, qr, kr, vt, T, H, Hkv, L, O32, O, LSE);
    else if (lds_ok && hd == 64)
        hipLaunchKernelGGL((attn_fwd_lds_kernel<64>), grid, dim3(256), 0, st, qr, kr, vt, T, H, Hkv, L, O32, O, LSE);
    else
        hipLaunchKernelGGL(attn_fwd_kernel, grid, dim3(256), 0, st, qr, kr, vt, T, H, Hkv, hd, L, O32, O, LSE);
    return hipGetLastError();
}

// D[t][h] = sum_c dO[t][h hd + c] O32[t][h hd + c] (float64, summed in order of c); a block takes 32
// rows: the 256 threads stage both row sets through LDS with coalesced 16-byte loads, then one
// thread per row sums it.  hd a multiple of 32, at most 256.
constexpr int RD_ROWS = 32;
__global__ __launch_bounds__(256) void attn_rowdot_kernel(const float* __restrict__ dO, const float* __restrict__ O32,
                                                          int64_t TH, int64_t hd, double* __restrict__ D) {
    __shared__ float sa[RD_ROWS * (256 + 1)];
    __shared__ float sb[RD_ROWS * (256 + 1)];
    const int64_t r0 = (int64_t)blockIdx.x * RD_ROWS;
    const int64_t rows = TH - r0 < RD_ROWS ? TH - r0 : RD_ROWS;
    const int64_t st = hd + 1;
    const int64_t n4 = rows * hd / 4;
    for (int64_t q = threadIdx.x; q < n4; q += 256) {
        const int64_t rr = (q * 4) / hd, c = (q * 4) % hd;
        const float4 a = *reinterpret_cast<const float4*>(dO + (r0 + rr) * hd + c);
        const float4 b = *reinterpret_cast<const float4*>(O32 + (r0 + rr) * hd + c);
        float* pa = sa + rr * st + c;
        float* pb = sb + rr * st + c;
        pa[0] = a.x; pa[1] = a.y; pa[2] = a.z; pa[3] = a.w;
        pb[0] = b.x; pb[1] = b.y; pb[2] = b.z; pb[3] = b.w;
    }
    __syncthreads();
    if (threadIdx.x < rows) {
        const float* a = sa + threadIdx.x * st;
        const float* b = sb + threadIdx.x * st;
        double acc = 0.0;
        for (int64_t c = 0; c < hd; ++c) acc += (double)a[c] * (double)b[c];
        D[r0 + threadIdx.x] = acc;
    }
}

// dS = P o (dP - D) for the causal tiles, P_ij = exp(qr_i . kr_j / sqrt(hd) - LSE_i) recomputed from
// the forward's row log-sum-exp (the same MFMA sums as the forward), dP = dO v^T (dO in three bf16
// terms); grid (S H nt, ceil(nt / 4)), wave w of block y takes key tile 4 y + w of query tile it.
// Writes dS [i][j], dS^T and P^T [j][i] as bf16 hi/lo.
__global__ __launch_bounds__(256) void attn_ds_kernel(const uint16_t* __restrict__ qr, const uint16_t* __restrict__ kr,
                                                      const double* __restrict__ LSE, const float* __restrict__ dO,
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
    const uint16_t* qa = qr + (s * L + it * AT + (lane & 31)) * (H * hd) + h * hd + 8 * (lane >> 5);
    const uint16_t* kb = kr + (s * L + jt * AT + (lane & 31)) * (Hkv * hd) + g * hd + 8 * (lane >> 5);
    f32x16 acc = zero16(), sc = zero16();
    for (int64_t k0 = 0; k0 < hd; k0 += 16) {  // dO in three terms: dP - D cancels
        bf16x8 ah, al, al2;
        split8x3(a + k0, ah, al, al2);
        const bf16x8 bv = ld8(b + k0);
        acc = mfma(ah, bv, acc);
        acc = mfma(al, bv, acc);
        acc = mfma(al2, bv, acc);
        sc = mfma(ld8(qa + k0), ld8(kb + k0), sc);
    }
    const double scale = 1.0 / sqrt((double)hd);
    // The six bf16 tiles go out through a per-wave LDS tile (transposed there for dS^T and P^T), so
    // every row segment is written as 16-byte stores: lane l then owns 8 consecutive entries of
    // row l / 4 (and of row 16 + l / 4).
    __shared__ __attribute__((aligned(16))) uint16_t stage[4][AT][TSTR];
    uint16_t(*tb)[TSTR] = stage[wave];
    uint16_t vh[16], vl[16], qh[16], ql[16];
#pragma unroll
    for (int e = 0; e < 16; ++e) {
        const int64_t i = it * AT + acc_row(e, lane), j = jt * AT + (lane & 31);
        const float p = j <= i ? expf((float)((double)sc[e] * scale - LSE[(s * L + i) * H + h])) : 0.f;
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

// attn_ds_kernel with the work of a query tile in one wave (used when the grid has at least 512
// blocks: with 300 registers a wave has its SIMD to itself): the four waves of a block take
// consecutive query tiles of one head (as the forward's), keep their query fragments, LSE and D in
// LDS and their dO rows in registers (split into three terms per key tile), and walk the
// key tiles on or below their diagonal while the block streams each key tile and value tile into
// two LDS buffers (rows XOR-swizzled as in the forward).  Per element the arithmetic is that of
// attn_ds_kernel, so the six outputs are bitwise the same.
template <int HD>
__global__ __launch_bounds__(256) void attn_ds_lds_kernel(const uint16_t* __restrict__ qr,
                                                          const uint16_t* __restrict__ kr,
                                                          const double* __restrict__ LSE,
                                                          const float* __restrict__ dO,
                                                          const uint16_t* __restrict__ v,
                                                          const double* __restrict__ D, int64_t H, int64_t Hkv,
                                                          int64_t L, uint16_t* __restrict__ dSh,
                                                          uint16_t* __restrict__ dSl, uint16_t* __restrict__ dSth,
                                                          uint16_t* __restrict__ dStl, uint16_t* __restrict__ Pth,
                                                          uint16_t* __restrict__ Ptl) {
    constexpr int NK = HD / 16;
    constexpr int KCH = HD / 8;
    constexpr int TBYTES = AT * HD * 2;                  // one key (or value) tile
    constexpr int TDMA = TBYTES / 1024 / 4;              // 1 KB loads per wave and tile
    static_assert(TDMA >= 1, "head width");
    __shared__ __attribute__((aligned(16))) uint16_t sKV[2][TBYTES];   // [buf][key tile | value tile]
    __shared__ __attribute__((aligned(16))) uint16_t sQ[4][AT * HD];    // each wave's query rows (swizzled)
    __shared__ __attribute__((aligned(16))) uint32_t stage[4][AT][TSTR32];
    __shared__ double sLD[4][2][AT];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int wv = __builtin_amdgcn_readfirstlane(wave);
    const int64_t nt = L / AT, nq = (nt + 3) / 4;
    const int64_t sh = blockIdx.x / nq, h = sh % H, s = sh / H;
    const int64_t qb = blockIdx.x % nq;
    const int64_t itmax = nt - 1 - 4 * qb;
    const int64_t it = itmax - wave;
    const bool active = it >= 0;
    const int64_t g = h / (H / Hkv);
    const int64_t ldk = Hkv * HD;
    const int c32 = lane & 31, k8 = 8 * (lane >> 5);
    const uint16_t* kbase = kr + (s * L) * ldk + g * HD;
    const uint16_t* vbase = v + (s * L) * ldk + g * HD;
    const uint32_t lds0 = (uint32_t)(uintptr_t)&sKV[0][0];
    auto load_tile = [&](int64_t jt, int b) {
        const uint32_t dst = lds0 + (uint32_t)b * (2 * TBYTES);
        const char* kb = reinterpret_cast<const char*>(kbase + jt * AT * ldk);
        const char* vb = reinterpret_cast<const char*>(vbase + jt * AT * ldk);
#pragma unroll
        for (int q = 0; q < TDMA; ++q) {
            const int qi = wv * TDMA + q;
            const int row = qi * (1024 / (HD * 2)) + lane / KCH, pos = lane % KCH;
            const uint32_t off = (uint32_t)((row * ldk + (pos ^ (row % KCH)) * 8) * 2);
            attn_dma16(kb, off, dst + (uint32_t)qi * 1024);
            attn_dma16(vb, off, dst + TBYTES + (uint32_t)qi * 1024);
        }
    };
    // this wave's rows: query fragments (LDS), dO (registers, split once into its three bf16
    // terms: the same for every key tile), LSE and D (LDS)
    uint16_t* const qw = sQ[wave];
    bf16x8 dOh[NK], dOl[NK], dOl2[NK];
#pragma unroll
    for (int kk = 0; kk < NK; ++kk) dOh[kk] = dOl[kk] = dOl2[kk] = bf16x8{};
    if (active) {
        const uint16_t* qa = qr + (s * L + it * AT + c32) * (H * HD) + h * HD + k8;
        const float* a = dO + (s * L + it * AT + c32) * (H * HD) + h * HD + k8;
#pragma unroll
        for (int kk = 0; kk < NK; ++kk) {
            const int c = 2 * kk + (lane >> 5);
            *reinterpret_cast<u16x8*>(qw + c32 * HD + (c ^ (c32 % KCH)) * 8) =
                *reinterpret_cast<const u16x8*>(qa + 16 * kk);
            split8x3(a + 16 * kk, dOh[kk], dOl[kk], dOl2[kk]);
        }
        if (lane < AT) {
            sLD[wave][0][lane] = LSE[(s * L + it * AT + lane) * H + h];
            sLD[wave][1][lane] = D[(s * L + it * AT + lane) * H + h];
        }
    }
    const double scale = 1.0 / sqrt((double)HD);
    uint32_t(*tb)[TSTR32] = stage[wave];
    const int r = lane >> 2, c8 = (lane & 3) * 8;
    // values packed as hi | lo << 16, staged whole and split into the hi and lo arrays on the way out
    auto flush = [&](const uint32_t (&val)[16], bool transposed, uint16_t* dst_hi, uint16_t* dst_lo, int64_t row0,
                     int64_t col0) {
#pragma unroll
        for (int e = 0; e < 16; ++e) {
            const int a = acc_row(e, lane), b = lane & 31;
            if (transposed) tb[b][a] = val[e];
            else tb[a][b] = val[e];
        }
        __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
#pragma unroll
        for (int half = 0; half < 2; ++half) {
            const int rr = r + 16 * half;
            const u32x4 v0 = *reinterpret_cast<const u32x4*>(&tb[rr][c8]);
            const u32x4 v1 = *reinterpret_cast<const u32x4*>(&tb[rr][c8 + 4]);
            u16x8 h, l;
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                h[u] = (uint16_t)(v0[u] & 0xffffu);
                l[u] = (uint16_t)(v0[u] >> 16);
                h[u + 4] = (uint16_t)(v1[u] & 0xffffu);
                l[u + 4] = (uint16_t)(v1[u] >> 16);
            }
            const int64_t o = (sh * L + row0 + rr) * L + col0 + c8;
            *reinterpret_cast<u16x8*>(dst_hi + o) = h;
            *reinterpret_cast<u16x8*>(dst_lo + o) = l;
        }
        __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
    };
    load_tile(0, 0);
    for (int64_t jt = 0; jt <= itmax; ++jt) {
        // this wave's loads of tile jt have landed; the 12 stores of the previous tile, issued after
        // those loads, may still be in flight
        if (jt >= 1 && jt - 1 <= it) attn_wait_vm<12>();
        else attn_wait_vm<0>();
        __syncthreads();
        if (jt + 1 <= itmax) load_tile(jt + 1, (int)((jt + 1) & 1));
        if (jt > it) continue;
        const uint16_t* kt = &sKV[jt & 1][0];
        const uint16_t* vt_ = kt + TBYTES / 2;
        f32x16 acc = zero16(), sc = zero16();
#pragma unroll
        for (int kk = 0; kk < NK; ++kk) {  // dO in three terms: dP - D cancels
            const int c = 2 * kk + (lane >> 5);
            const int off = c32 * HD + ((c ^ (c32 % KCH)) * 8);
            const bf16x8 bv = ld8(vt_ + off);
            acc = mfma(dOh[kk], bv, acc);
            acc = mfma(dOl[kk], bv, acc);
            acc = mfma(dOl2[kk], bv, acc);
            sc = mfma(ld8(qw + off), ld8(kt + off), sc);
        }
        uint32_t dsv[16], pv2[16];
#pragma unroll
        for (int e = 0; e < 16; ++e) {
            const int ir = acc_row(e, lane);
            const int64_t i = it * AT + ir, j = jt * AT + c32;
            const float pv = j <= i ? expf((float)((double)sc[e] * scale - sLD[wave][0][ir])) : 0.f;
            const float ds = (float)((double)pv * ((double)acc[e] - sLD[wave][1][ir]));
            uint16_t a0, a1, b0, b1;
            split_bf16(ds, a0, a1);
            split_bf16(pv, b0, b1);
            dsv[e] = (uint32_t)a0 | ((uint32_t)a1 << 16);
            pv2[e] = (uint32_t)b0 | ((uint32_t)b1 << 16);
        }
        flush(dsv, false, dSh, dSl, it * AT, jt * AT);
        flush(dsv, true, dSth, dStl, jt * AT, it * AT);
        flush(pv2, true, Pth, Ptl, jt * AT, it * AT);
    }
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

// attn_dq_kernel with the four waves of a block on four consecutive query tiles of one head (the
// longest first), each computing every value-column tile: the k^T tile of a key tile (the head's
// HD rows over its 32 tokens) is loaded once per block, one step ahead into registers, and stored
// to one of two LDS buffers (rows swizzled as the forward's value tile); each wave's dS hi/lo
// fragments are loaded one step ahead.  Every accumulator takes its products in the old order,
// so dq is bitwise the same.  grid (S H ceil(nt / 4)).
template <int HD>
__global__ __launch_bounds__(256) void attn_dq_lds_kernel(const uint16_t* __restrict__ dSh,
                                                          const uint16_t* __restrict__ dSl,
                                                          const uint16_t* __restrict__ kt, int64_t T, int64_t H,
                                                          int64_t Hkv, int64_t L, float* __restrict__ dq) {
    constexpr int NCT = HD / AT;
    constexpr int BT = HD * AT;
    constexpr int BCH = HD * 4 / 256;                 // 16-byte chunks per thread and step
    static_assert(HD * 4 % 256 == 0, "head width");
    __shared__ __attribute__((aligned(16))) uint16_t sB[2][BT];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int64_t nt = L / AT, nq = (nt + 3) / 4;
    const int64_t sh = blockIdx.x / nq, h = sh % H, s = sh / H;
    const int64_t qb = blockIdx.x % nq;
    const int64_t itmax = nt - 1 - 4 * qb;
    const int64_t it = itmax - wave;
    const int64_t g = h / (H / Hkv);
    const int c32 = lane & 31, k8 = 8 * (lane >> 5);
    u16x8 breg[BCH];
    auto load_B = [&](int64_t jt) {
#pragma unroll
        for (int q = 0; q < BCH; ++q) {
            const int id = threadIdx.x + 256 * q;
            const int row = id >> 2, c = id & 3;
            breg[q] = *reinterpret_cast<const u16x8*>(kt + (g * HD + row) * T + s * L + jt * AT + c * 8);
        }
    };
    auto store_B = [&](int b) {
#pragma unroll
        for (int q = 0; q < BCH; ++q) {
            const int id = threadIdx.x + 256 * q;
            const int row = id >> 2, c = id & 3;
            *reinterpret_cast<u16x8*>(&sB[b][row * AT + ((c ^ vswz(row)) * 8)]) = breg[q];
        }
    };
    struct AF {
        bf16x8 h[2], l[2];
    };
    const int64_t arow = (sh * L + it * AT + c32) * L + k8;
    auto load_A = [&](int64_t jt, AF& f) {
#pragma unroll
        for (int u = 0; u < 2; ++u) {
            f.h[u] = ld8(dSh + arow + jt * AT + 16 * u);
            f.l[u] = ld8(dSl + arow + jt * AT + 16 * u);
        }
    };
    f32x16 acc[NCT];
#pragma unroll
    for (int ct = 0; ct < NCT; ++ct) acc[ct] = zero16();
    AF acur, anxt;
    if (it >= 0) load_A(0, acur);
    load_B(0);
    store_B(0);
    __syncthreads();
    for (int64_t jt = 0; jt <= itmax; ++jt) {
        const bool more = jt + 1 <= itmax;
        if (more && jt + 1 <= it) load_A(jt + 1, anxt);
        if (more) load_B(jt + 1);
        if (jt <= it) {
            const uint16_t* bt = sB[jt & 1];
#pragma unroll
            for (int u = 0; u < 2; ++u) {
                const int c = 2 * u + (lane >> 5);
#pragma unroll
                for (int ct = 0; ct < NCT; ++ct) {
                    const int row = ct * AT + c32;
                    const bf16x8 b = ld8(bt + row * AT + ((c ^ vswz(row)) * 8));
                    acc[ct] = mfma(acur.h[u], b, acc[ct]);
                    acc[ct] = mfma(acur.l[u], b, acc[ct]);
                }
            }
        }
        if (more) store_B((int)((jt + 1) & 1));
        __syncthreads();
        acur = anxt;
    }
    if (it < 0) return;
    const float scale = (float)(1.0 / sqrt((double)HD));
#pragma unroll
    for (int ct = 0; ct < NCT; ++ct) {
        const int64_t col = h * HD + ct * AT + c32;
#pragma unroll
        for (int e = 0; e < 16; ++e) dq[(s * L + it * AT + acc_row(e, lane)) * H * HD + col] = acc[ct][e] * scale;
    }
}

// Query tiles per chunk of the dK/dV sums: each (key tile, chunk) pair is one wave, so no wave
// walks more than CH query tiles per head.
constexpr int CH = 8;
int64_t attn_dkv_chunks(int64_t L) { return (L / AT + CH - 1) / CH; }

// Partial dkr = sum_h dS^T qr / sqrt(hd) and dv = sum_h P^T dO over the query heads of key/value
// head g and the query tiles of chunk z (tiles [z CH, z CH + CH) on or past the key tile):
// grid (S Hkv nt, ceil(hd / 32 / 4), nch); qt = qr^T [H hd][T], dOt = dO^T as hi/lo [H hd][T].
// Writes part[z][0][T][Hkv hd] (dk) and part[z][1][T][Hkv hd] (dv); chunks wholly before the key
// tile write nothing (the reduction skips them).
__global__ __launch_bounds__(256) void attn_dkv_kernel(const uint16_t* __restrict__ dSth,
                                                       const uint16_t* __restrict__ dStl,
                                                       const uint16_t* __restrict__ Pth, const uint16_t* __restrict__ Ptl,
                                                       const uint16_t* __restrict__ qt,
                                                       const uint16_t* __restrict__ dOth,
                                                       const uint16_t* __restrict__ dOtl, int64_t T, int64_t H,
                                                       int64_t Hkv, int64_t hd, int64_t L, float* __restrict__ part) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int64_t nt = L / AT;
    const int64_t jt = blockIdx.x % nt, sg = blockIdx.x / nt, g = sg % Hkv, s = sg / Hkv;
    const int64_t ct = (int64_t)blockIdx.y * 4 + wave;
    const int64_t z = blockIdx.z;
    if (ct >= hd / AT || (z + 1) * CH <= jt) return;
    const int64_t ibeg = (jt > z * CH ? jt : z * CH) * AT, iend = ((z + 1) * CH < nt ? (z + 1) * CH : nt) * AT;
    const int64_t rep = H / Hkv;
    f32x16 ak = zero16(), av = zero16();
    for (int64_t hh = 0; hh < rep; ++hh) {
        const int64_t h = g * rep + hh, sh = s * H + h;
        const int64_t arow = (sh * L + jt * AT + (lane & 31)) * L + 8 * (lane >> 5);
        const int64_t brow = (h * hd + ct * AT + (lane & 31)) * T + s * L + 8 * (lane >> 5);
        for (int64_t i0 = ibeg; i0 < iend; i0 += 32) {  // whole tiles: two steps per trip
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
    const int64_t col = g * hd + ct * AT + (lane & 31), TK = T * Hkv * hd;
    float* pk = part + 2 * z * TK;
#pragma unroll
    for (int e = 0; e < 16; ++e) {
        const int64_t t = s * L + jt * AT + acc_row(e, lane);
        pk[t * Hkv * hd + col] = ak[e] * scale;
        pk[TK + t * Hkv * hd + col] = av[e];
    }
}

// attn_dkv_kernel with the four waves of a block on four consecutive key tiles of one key/value
// head, each computing all HD/32 value-column tiles: the B operands of a step (head h of the
// group, query tile it: the 32 tokens of q^T and of dO^T hi/lo over the head's HD rows, 24 KB for
// HD = 128) are loaded once per block, one step ahead into registers, and stored to one of two LDS
// buffers (rows swizzled as the forward's value tile); each wave's dS^T / P^T fragments of the
// step are loaded one step ahead into registers, before the block's loads of the following step,
// so no wait for them waits for those.  Steps run over the group's heads, then the chunk's query
// tiles, as in attn_dkv_kernel, and every accumulator takes its products in the same order: the
// partial sums are bitwise the same.  grid (S Hkv ceil(nt / 4), nch).
template <int HD>
__global__ __launch_bounds__(256) void attn_dkv_lds_kernel(const uint16_t* __restrict__ dSth,
                                                           const uint16_t* __restrict__ dStl,
                                                           const uint16_t* __restrict__ Pth,
                                                           const uint16_t* __restrict__ Ptl,
                                                           const uint16_t* __restrict__ qt,
                                                           const uint16_t* __restrict__ dOth,
                                                           const uint16_t* __restrict__ dOtl, int64_t T, int64_t H,
                                                           int64_t Hkv, int64_t L, float* __restrict__ part) {
    constexpr int NCT = HD / AT;
    constexpr int BT = HD * AT;                       // bf16 per B tile
    constexpr int BCH = 3 * HD * 4 / 256;             // 16-byte chunks per thread and step
    static_assert(3 * HD * 4 % 256 == 0, "head width");
    __shared__ __attribute__((aligned(16))) uint16_t sB[2][3][BT];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int64_t nt = L / AT, ng = (nt + 3) / 4;
    const int64_t jg = blockIdx.x % ng, sg = blockIdx.x / ng, g = sg % Hkv, s = sg / Hkv;
    const int64_t z = blockIdx.y;
    const int64_t jt = 4 * jg + wave;
    const int64_t i0 = (4 * jg > z * CH ? 4 * jg : z * CH), i1 = ((z + 1) * CH < nt ? (z + 1) * CH : nt);
    if (i0 >= i1) return;                             // the whole chunk lies before the group's key tiles
    const bool wave_on = jt < nt && (z + 1) * CH > jt;  // this wave's key tile has terms in the chunk
    const int64_t rep = H / Hkv;
    const int64_t nsteps = rep * (i1 - i0);
    const int c32 = lane & 31, k8 = 8 * (lane >> 5);
    const uint16_t* Bsrc[3] = {qt, dOth, dOtl};
    // step x: head hh = x / (i1 - i0), query tile it = i0 + x % (i1 - i0)
    auto step_of = [&](int64_t x, int64_t& h, int64_t& it) {
        h = g * rep + x / (i1 - i0);
        it = i0 + x % (i1 - i0);
    };
    u16x8 breg[BCH];
    auto load_B = [&](int64_t x) {
        int64_t h, it;
        step_of(x, h, it);
#pragma unroll
        for (int q = 0; q < BCH; ++q) {
            const int id = threadIdx.x + 256 * q;
            const int a = id / (HD * 4), row = (id % (HD * 4)) >> 2, c = id & 3;
            breg[q] = *reinterpret_cast<const u16x8*>(Bsrc[a] + (h * HD + row) * T + s * L + it * AT + c * 8);
        }
    };
    auto store_B = [&](int b) {
#pragma unroll
        for (int q = 0; q < BCH; ++q) {
            const int id = threadIdx.x + 256 * q;
            const int a = id / (HD * 4), row = (id % (HD * 4)) >> 2, c = id & 3;
            *reinterpret_cast<u16x8*>(&sB[b][a][row * AT + ((c ^ vswz(row)) * 8)]) = breg[q];
        }
    };
    struct AF {
        bf16x8 sh[2], sl[2], ph[2], pl[2];
    };
    auto load_A = [&](int64_t x, AF& f) {
        int64_t h, it;
        step_of(x, h, it);
        const int64_t sh = s * H + h;
        const int64_t arow = (sh * L + jt * AT + c32) * L + it * AT + k8;
#pragma unroll
        for (int u = 0; u < 2; ++u) {
            f.sh[u] = ld8(dSth + arow + 16 * u);
            f.sl[u] = ld8(dStl + arow + 16 * u);
            f.ph[u] = ld8(Pth + arow + 16 * u);
            f.pl[u] = ld8(Ptl + arow + 16 * u);
        }
    };
    auto active = [&](int64_t x) {
        int64_t h, it;
        step_of(x, h, it);
        return wave_on && it >= jt;
    };
    f32x16 ak[NCT], av[NCT];
#pragma unroll
    for (int ct = 0; ct < NCT; ++ct) {
        ak[ct] = zero16();
        av[ct] = zero16();
    }
    AF acur, anxt;
    if (active(0)) load_A(0, acur);
    load_B(0);
    store_B(0);
    __syncthreads();
    for (int64_t x = 0; x < nsteps; ++x) {
        const bool more = x + 1 < nsteps;
        if (more && active(x + 1)) load_A(x + 1, anxt);
        if (more) load_B(x + 1);
        if (active(x)) {
            const uint16_t* bq = sB[x & 1][0];
            const uint16_t* bh = sB[x & 1][1];
            const uint16_t* bl = sB[x & 1][2];
#pragma unroll
            for (int u = 0; u < 2; ++u) {
                const int c = 2 * u + (lane >> 5);
#pragma unroll
                for (int ct = 0; ct < NCT; ++ct) {
                    const int row = ct * AT + c32;
                    const int off = row * AT + ((c ^ vswz(row)) * 8);
                    const bf16x8 q = ld8(bq + off), doh = ld8(bh + off), dol = ld8(bl + off);
                    ak[ct] = mfma(acur.sh[u], q, ak[ct]);
                    ak[ct] = mfma(acur.sl[u], q, ak[ct]);
                    av[ct] = mfma(acur.ph[u], doh, av[ct]);
                    av[ct] = mfma(acur.pl[u], doh, av[ct]);
                    av[ct] = mfma(acur.ph[u], dol, av[ct]);
                }
            }
        }
        if (more) store_B((int)((x + 1) & 1));
        __syncthreads();
        acur = anxt;
    }
    if (!wave_on) return;
    const float scale = (float)(1.0 / sqrt((double)HD));
    const int64_t TK = T * Hkv * HD;
    float* pk = part + 2 * z * TK;
#pragma unroll
    for (int ct = 0; ct < NCT; ++ct) {
        const int64_t col = g * HD + ct * AT + c32;
#pragma unroll
        for (int e = 0; e < 16; ++e) {
            const int64_t t = s * L + jt * AT + acc_row(e, lane);
            pk[t * Hkv * HD + col] = ak[ct][e] * scale;
            pk[TK + t * Hkv * HD + col] = av[ct][e];
        }
    }
}

// dk, dv [T][Hkv hd] = sum over the chunks z of token t's key tile and after (z ascending: a fixed
// order) of the partial sums.
__global__ void attn_dkv_reduce_kernel(const float* __restrict__ part, int64_t T, int64_t K, int64_t L,
                                       int64_t nch, float* __restrict__ dk, float* __restrict__ dv) {
    const int64_t TK = T * K;
    for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < TK; e += (int64_t)gridDim.x * blockDim.x) {
        const int64_t jt = ((e / K) % L) / AT;
        float a = 0.f, b = 0.f;
        for (int64_t z = jt / CH; z < nch; ++z) {
            a += part[2 * z * TK + e];
            b += part[(2 * z + 1) * TK + e];
        }
        dk[e] = a;
        dv[e] = b;
    }
}

hipError_t attn_bwd(const double* LSE, const float* O32, const float* dO, const uint16_t* qr, const uint16_t* kr,
                    const uint16_t* v, int64_t T, int64_t H, int64_t Hkv, int64_t hd, int64_t L, const AttnScratch& w,
                    float* dq, float* dk, float* dv, hipStream_t st) {
    if (T <= 0) return hipSuccess;
    const int64_t S = T / L, nt = L / AT;
    hipError_t e;
    hipLaunchKernelGGL(attn_rowdot_kernel, dim3((unsigned)((T * H + RD_ROWS - 1) / RD_ROWS)), dim3(256), 0, st, dO, O32,
                       T * H, hd, w.D);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if ((e = transpose_u16(kr, Hkv * hd, w.kt, T, T, Hkv * hd, st)) != hipSuccess) return e;
    if ((e = transpose_u16(qr, H * hd, w.qt, T, T, H * hd, st)) != hipSuccess) return e;
    if ((e = transpose_split_f32(dO, H * hd, w.dOth, w.dOtl, T, T, H * hd, st)) != hipSuccess) return e;
    // the query-tile-per-wave kernel needs enough blocks to fill the chip (one wave per SIMD)
    const bool lds_ok = (((uintptr_t)kr | (uintptr_t)v) & 15) == 0 && (Hkv * hd) % 8 == 0 &&
                        (int64_t)AT * Hkv * hd * 2 < (int64_t(1) << 31) && S * H * ((nt + 3) / 4) >= 512;
    const dim3 gq((unsigned)(S * H * ((nt + 3) / 4)));
    if (lds_ok && hd == 128)
        hipLaunchKernelGGL((attn_ds_lds_kernel<128>), gq, dim3(256), 0, st, qr, kr, LSE, dO, v, w.D, H, Hkv, L, w.dSh,
                           w.dSl, w.dSth, w.dStl, w.Pth, w.Ptl);
    else if (lds_ok && hd == 64)
        hipLaunchKernelGGL((attn_ds_lds_kernel<64>), gq, dim3(256), 0, st, qr, kr, LSE, dO, v, w.D, H, Hkv, L, w.dSh,
                           w.dSl, w.dSth, w.dStl, w.Pth, w.Ptl);
    else
        hipLaunchKernelGGL(attn_ds_kernel, dim3((unsigned)(S * H * nt), (unsigned)((nt + 3) / 4)), dim3(256), 0, st, qr,
                           kr, LSE, dO, v, w.D, H, Hkv, hd, L, w.dSh, w.dSl, w.dSth, w.dStl, w.Pth, w.Ptl);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    const unsigned cy = (unsigned)((hd / AT + 3) / 4);
    const bool dq_lds = T % 8 == 0 && (hd == 128 || hd == 64) && S * H * ((nt + 3) / 4) >= 64;
    if (dq_lds && hd == 128)
        hipLaunchKernelGGL((attn_dq_lds_kernel<128>), dim3((unsigned)(S * H * ((nt + 3) / 4))), dim3(256), 0, st, w.dSh,
                           w.dSl, w.kt, T, H, Hkv, L, dq);
    else if (dq_lds)
        hipLaunchKernelGGL((attn_dq_lds_kernel<64>), dim3((unsigned)(S * H * ((nt + 3) / 4))), dim3(256), 0, st, w.dSh,
                           w.dSl, w.kt, T, H, Hkv, L, dq);
    else
        hipLaunchKernelGGL(attn_dq_kernel, dim3((unsigned)(S * H * nt), cy), dim3(256), 0, st, w.dSh, w.dSl, w.kt, T, H,
                           Hkv, hd, L, dq);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    const int64_t nch = attn_dkv_chunks(L);
    const bool dkv_lds = T % 8 == 0 && (hd == 128 || hd == 64) && S * Hkv * ((nt + 3) / 4) * nch >= 64;
    if (dkv_lds && hd == 128)
        hipLaunchKernelGGL((attn_dkv_lds_kernel<128>), dim3((unsigned)(S * Hkv * ((nt + 3) / 4)), (unsigned)nch),
                           dim3(256), 0, st, w.dSth, w.dStl, w.Pth, w.Ptl, w.qt, w.dOth, w.dOtl, T, H, Hkv, L, w.part);
    else if (dkv_lds)
        hipLaunchKernelGGL((attn_dkv_lds_kernel<64>), dim3((unsigned)(S * Hkv * ((nt + 3) / 4)), (unsigned)nch),
                           dim3(256), 0, st, w.dSth, w.dStl, w.Pth, w.Ptl, w.qt, w.dOth, w.dOtl, T, H, Hkv, L, w.part);
    else
        hipLaunchKernelGGL(attn_dkv_kernel, dim3((unsigned)(S * Hkv * nt), cy, (unsigned)nch), dim3(256), 0, st,
                           w.dSth, w.dStl, w.Pth, w.Ptl, w.qt, w.dOth, w.dOtl, T, H, Hkv, hd, L, w.part);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(attn_dkv_reduce_kernel, dim3(grid_of(T * Hkv * hd)), dim3(TB), 0, st, w.part, T, Hkv * hd, L, nch,
                       dk, dv);
    return hipGetLastError();
}

}  // namespace realq
