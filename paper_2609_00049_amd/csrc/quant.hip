// Quantization of one column block (Alg. 1 inner loop; Sec. 3.2 Eq. gptq_update).
//
// One wave64 owns one weight row at a time; lane l holds block columns l and l+64
// in registers.  Per row:
//   1. dead columns of the block are zeroed;
//   2. when a quantization group starts (a group may span the whole row), its
//      (scale, zero) pair is searched in
//      float64: lanes split the shrink factors p_k = 1 - k/100 (lane l takes k = l and
//      k = l + 64), every lane scores all zero points of its k over the group's
//      values (broadcast with readlane); one wave reduction finds the least error,
//      errors up to least * (1 + 2^-40) + 2^-60 * sum x^2 form one tie, and a second
//      reduction picks the least (k, |z - z_nat|, z) among them, with
//      z_nat = rint(-lo maxq / (hi - lo)); the symmetric quantizer takes the range
//      [-max|x|, max|x|] and only the zero point (maxq + 1) / 2;
//   3. columns are quantized in order with the scale as stored (float32):
//      q = clamp(rint(w/s) + z, 0, maxq) decided in float64, w_hat = s (q - z) (exact in
//      float64, so the float32 output is the float32 dequantization of the stored
//      parameters), and the error
//      e = (w - w_hat) / U_jj is propagated to the block's later columns with row j of
//      the inverse factor U (held in LDS);
//
// Every float64 step that decides an integer (rint of x / s, the candidate errors, the
// natural zero) uses correctly rounded IEEE operations without fused multiply-adds, so
// that an exact tie of the underlying arithmetic is seen as a tie here too.
//   4. w_hat, codes, the block error E and the bf16 split of w_hat - W0 are written.
// The working weights are float64 (one row in registers, two values per lane): every
// later column takes up to 127 compensation updates here and more from the trailing
// update, Block-GD and later blocks, and a float32 running value would drift by
// about 1e-8, enough to move a few codes per module across a rounding boundary.
//
// obs_update_kernel then applies the trailing update W[:, c1:] -= E_b U[b, c1:]
// (Sec. 3.2) in float64 and refreshes the bf16 split of W - W0 for those columns.
#include "common.h"
#include "kernels.h"

namespace realq {

namespace {
constexpr int QB = 128;          // maximum block width
constexpr int WAVES = 4;
constexpr int ROWS_PER_WAVE = 4;
constexpr int ROWS_PER_WG = WAVES * ROWS_PER_WAVE;

__device__ __forceinline__ double bcast(double v, int lane) {
    const int lo = __builtin_amdgcn_readlane(__double2loint(v), lane);
    const int hi = __builtin_amdgcn_readlane(__double2hiint(v), lane);
    return __hiloint2double(hi, lo);
}

constexpr double TIE_RTOL = 0x1p-40;  // search errors within TIE_RTOL * least + TIE_ATOL * sum x^2
constexpr double TIE_ATOL = 0x1p-60;  // are one tie

struct Best {
    int k, dist, z;
};

__device__ __forceinline__ bool better(const Best& a, const Best& b) {
    if (a.k != b.k) return a.k < b.k;
    if (a.dist != b.dist) return a.dist < b.dist;
    return a.z < b.z;
}

// Per-lane state of the search for one group.
struct Search {
    double lo, hi, ss;
    double s[2];
    int kk[2];
    bool valid[2];
    double err[2][16];
};

}  // namespace

template <int MAXQ>
__device__ __forceinline__ void search_accumulate(Search& S, double x) {
#pragma clang fp contract(off)
#pragma unroll
    for (int a = 0; a < 2; ++a) {
        if (!S.valid[a]) continue;
        const double r = rint(x / S.s[a]);
#pragma unroll
        for (int z = 0; z <= MAXQ; ++z) {
            // q - z with q = clamp(r + z, 0, maxq) equals clamp(r, -z, maxq - z)
            const double c = fmin(fmax(r, (double)(-z)), (double)(MAXQ - z));
            const double d = x - S.s[a] * c;
            S.err[a][z] = fma(d, d, S.err[a][z]);
        }
    }
}

template <int MAXQ>
__device__ __forceinline__ void search_begin(Search& S, double lo, double hi, double ss, int grid, int lane,
                                             bool sym) {
#pragma clang fp contract(off)
    lo = fmin(0.0, lo);
    hi = fmax(0.0, hi);
    if (sym) {
        const double amax = fmax(-lo, hi);
        lo = -amax;
        hi = amax;
    }
    if (lo == hi) {
        lo = -1.0;
        hi = 1.0;
    }
    S.lo = lo;
    S.hi = hi;
    S.ss = ss;
#pragma unroll
    for (int a = 0; a < 2; ++a) {
        const int k = lane + 64 * a;
        S.kk[a] = k;
        S.valid[a] = k < grid;
        const double p = 1.0 - (double)k / 100.0;
        S.s[a] = (p * (hi - lo)) / (double)MAXQ;
#pragma unroll
        for (int z = 0; z <= MAXQ; ++z) S.err[a][z] = 0.0;
    }
}

// Reduce the per-lane candidates to the winner; returns (scale, zero) in all lanes.
template <int MAXQ>
__device__ __forceinline__ void search_finish(const Search& S, double& scale, int& zero, bool sym) {
#pragma clang fp contract(off)
    constexpr int ZSYM = (MAXQ + 1) / 2;
    double emin = INFINITY;
#pragma unroll
    for (int a = 0; a < 2; ++a) {
        if (!S.valid[a]) continue;
#pragma unroll
        for (int z = 0; z <= MAXQ; ++z)
            if (!sym || z == ZSYM) emin = fmin(emin, S.err[a][z]);
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) emin = fmin(emin, __shfl_xor(emin, off));
    const double thr = emin * (1.0 + TIE_RTOL) + TIE_ATOL * S.ss;
    // the shrink factor cancels from -p_k lo / s_k: one natural zero for every k
    const int znat = (int)fmin(fmax(rint((-S.lo * (double)MAXQ) / (S.hi - S.lo)), 0.0), (double)MAXQ);
    Best best{1 << 30, 1 << 30, 1 << 30};
#pragma unroll
    for (int a = 0; a < 2; ++a) {
        if (!S.valid[a]) continue;
#pragma unroll
        for (int z = 0; z <= MAXQ; ++z) {
            if (sym && z != ZSYM) continue;
            const Best c{S.kk[a], abs(z - znat), z};
            if (S.err[a][z] <= thr && better(c, best)) best = c;
        }
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
        Best o;
        o.k = __shfl_xor(best.k, off);
        o.dist = __shfl_xor(best.dist, off);
        o.z = __shfl_xor(best.z, off);
        if (better(o, best)) best = o;
    }
    const double p = 1.0 - (double)best.k / 100.0;
    scale = (p * (S.hi - S.lo)) / (double)MAXQ;
    zero = best.z;
}

template <int MAXQ>
__global__ __launch_bounds__(256) void quantize_block_kernel(QuantArgs q) {
    __shared__ float sU[QB * QB];
    const int64_t bs = q.bs, c0 = q.c0, n = q.n;
    // stage U[c0:c0+bs, c0:c0+bs]
    for (int e = threadIdx.x; e < bs * bs; e += blockDim.x) {
        int a = e / bs, b = e % bs;
        sU[a * QB + b] = q.U[(c0 + a) * n + c0 + b];
    }
    __syncthreads();

    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int64_t group = q.group;
    for (int rr = 0; rr < ROWS_PER_WAVE; ++rr) {
        const int64_t i = (int64_t)blockIdx.x * ROWS_PER_WG + wave * ROWS_PER_WAVE + rr;
        if (i >= q.m) break;  // uniform within the wave; no block-level barrier below
        double* Wrow = q.W + i * n;
        const bool in0 = lane < bs, in1 = lane + 64 < bs;
        double w0 = in0 ? Wrow[c0 + lane] : 0.0;
        double w1 = in1 ? Wrow[c0 + 64 + lane] : 0.0;
        if (q.dead) {
            if (in0 && q.dead[c0 + lane]) w0 = 0.0;
            if (in1 && q.dead[c0 + 64 + lane]) w1 = 0.0;
        }
        double scale = 1.0;
        double zf = 0.0;
        if (c0 % group != 0) {  // group started in an earlier block: reuse its parameters
            const int64_t g = c0 / group;
            scale = (double)q.scales[i * q.ngroups + g];
            zf = (double)q.zeros[i * q.ngroups + g];
        }
        double e0 = 0.0, e1 = 0.0;
        uint8_t code0 = 0, code1 = 0;
        for (int64_t j = 0; j < bs; ++j) {
            const int64_t col = c0 + j;
            if (col % group == 0) {
                // ---- (scale, zero) search over the group's current values
                const int64_t glen = min(group, n - col);
                Search S;
                double lo = INFINITY, hi = -INFINITY, ss = 0.0;
                if (j + glen <= bs) {
                    // whole group inside the block: values in registers
                    for (int64_t e = 0; e < glen; ++e) {
                        const int64_t jj = j + e;
                        const double x = bcast(jj < 64 ? w0 : w1, (int)(jj & 63));
                        lo = fmin(lo, x);
                        hi = fmax(hi, x);
                        ss = fma(x, x, ss);
                    }
                    search_begin<MAXQ>(S, lo, hi, ss, q.grid, lane, q.sym != 0);
                    for (int64_t e = 0; e < glen; ++e) {
                        const int64_t jj = j + e;
                        search_accumulate<MAXQ>(S, bcast(jj < 64 ? w0 : w1, (int)(jj & 63)));
                    }
                } else {
                    // group extends past the block (only at j == 0): read the untouched row
                    for (int64_t e0c = 0; e0c < glen; e0c += 64) {
                        const int64_t cc = col + e0c + lane;
                        double v = 0.0;
                        if (e0c + lane < glen) {
                            v = Wrow[cc];
                            if (q.dead && q.dead[cc]) v = 0.0;
                        }
                        const int cnt = (int)min((int64_t)64, glen - e0c);
                        for (int e = 0; e < cnt; ++e) {
                            const double x = bcast(v, e);
                            lo = fmin(lo, x);
                            hi = fmax(hi, x);
                            ss = fma(x, x, ss);
                        }
                    }
                    search_begin<MAXQ>(S, lo, hi, ss, q.grid, lane, q.sym != 0);
                    for (int64_t e0c = 0; e0c < glen; e0c += 64) {
                        const int64_t cc = col + e0c + lane;
                        double v = 0.0;
                        if (e0c + lane < glen) {
                            v = Wrow[cc];
                            if (q.dead && q.dead[cc]) v = 0.0;
                        }
                        const int cnt = (int)min((int64_t)64, glen - e0c);
                        for (int e = 0; e < cnt; ++e) search_accumulate<MAXQ>(S, bcast(v, e));
                    }
                }
                int zi;
                search_finish<MAXQ>(S, scale, zi, q.sym != 0);
                scale = (double)(float)scale;  // the stored float32 scale is the one used
                zf = (double)zi;
                if (lane == 0) {
                    q.scales[i * q.ngroups + col / group] = (float)scale;
                    q.zeros[i * q.ngroups + col / group] = (uint8_t)zi;
                }
            }
            // ---- quantize column j and compensate the block's later columns
            const double wj = bcast(j < 64 ? w0 : w1, (int)(j & 63));
            const double qv = fmin(fmax(rint(wj / scale) + zf, 0.0), (double)MAXQ);
            const double wq = scale * (qv - zf);
            const double err = (wj - wq) / (double)sU[j * QB + j];
            if (j < 64) {
                if (lane == j) {
                    w0 = wq;
                    e0 = err;
                    code0 = (uint8_t)qv;
                }
            } else if (lane == j - 64) {
                w1 = wq;
                e1 = err;
                code1 = (uint8_t)qv;
            }
            if (lane > j && in0) w0 = fma(-err, (double)sU[j * QB + lane], w0);
            if (lane + 64 > j && in1) w1 = fma(-err, (double)sU[j * QB + lane + 64], w1);
        }
        // ---- write back
        if (in0) {
            const int64_t c = c0 + lane;
            Wrow[c] = w0;
            q.codes[i * n + c] = code0;
            q.E[i * bs + lane] = e0;
            if (q.Dhi) {
                uint16_t h, l;
                split_bf16((float)(w0 - (double)q.W0[i * n + c]), h, l);
                q.Dhi[i * n + c] = h;
                q.Dlo[i * n + c] = l;
            }
        }
        if (in1) {
            const int64_t c = c0 + 64 + lane;
            Wrow[c] = w1;
            q.codes[i * n + c] = code1;
            q.E[i * bs + 64 + lane] = e1;
            if (q.Dhi) {
                uint16_t h, l;
                split_bf16((float)(w1 - (double)q.W0[i * n + c]), h, l);
                q.Dhi[i * n + c] = h;
                q.Dlo[i * n + c] = l;
            }
        }
    }
}

hipError_t quantize_block(const QuantArgs& q, hipStream_t st) {
    if (q.m <= 0 || q.bs <= 0) return hipSuccess;
    const unsigned grid = (unsigned)((q.m + ROWS_PER_WG - 1) / ROWS_PER_WG);
    switch (q.bits) {
#define RQ_CASE(b)                                                                                 \
    case b:                                                                                        \
        hipLaunchKernelGGL(quantize_block_kernel<(1 << b) - 1>, dim3(grid), dim3(256), 0, st, q); \
        break;
        RQ_CASE(2)
        RQ_CASE(3)
        RQ_CASE(4)
#undef RQ_CASE
        default:
            return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

// ---------------------------------------------------------------- trailing update, float64
namespace {
constexpr int OTM = 64, OTN = 64, OTK = 16;
}

__global__ __launch_bounds__(256) void obs_update_kernel(ObsArgs a, int64_t tiles_n) {
    __shared__ double sE[OTK][OTM + 1];
    __shared__ double sU2[OTK][OTN + 1];
    const int64_t tm = blockIdx.x / tiles_n, tn = blockIdx.x % tiles_n;
    const int64_t m0 = tm * OTM, n0 = tn * OTN;
    const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;  // 16 x 16 threads, 4x4 outputs each
    double acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = 0.0;
    for (int64_t k0 = 0; k0 < a.K; k0 += OTK) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int e = threadIdx.x + r * 256;
            const int row = e / OTK, kk = e % OTK;
            const int64_t gi = m0 + row, gk = k0 + kk;
            sE[kk][row] = (gi < a.M && gk < a.K) ? a.E[gi * a.lde + gk] : 0.0;
        }
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int e = threadIdx.x + r * 256;
            const int kk = e / OTN, col = e % OTN;
            const int64_t gk = k0 + kk, gj = n0 + col;
            sU2[kk][col] = (gk < a.K && gj < a.N) ? (double)a.U[gk * a.ldu + gj] : 0.0;
        }
        __syncthreads();
#pragma unroll
        for (int kk = 0; kk < OTK; ++kk) {
            double ev[4], uv[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) ev[i] = sE[kk][ty * 4 + i];
#pragma unroll
            for (int j = 0; j < 4; ++j) uv[j] = sU2[kk][tx + 16 * j];
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) acc[i][j] = fma(ev[i], uv[j], acc[i][j]);
        }
        __syncthreads();
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int64_t gi = m0 + ty * 4 + i;
        if (gi >= a.M) continue;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int64_t gj = n0 + tx + 16 * j;
            if (gj >= a.N) continue;
            double* w = a.W + gi * a.ldw + gj;
            const double v = *w - acc[i][j];
            *w = v;
            if (a.Dhi) {
                uint16_t h, l;
                split_bf16((float)(v - (double)a.W0[gi * a.ldw0 + gj]), h, l);
                a.Dhi[gi * a.ldd + gj] = h;
                a.Dlo[gi * a.ldd + gj] = l;
            }
        }
    }
}

hipError_t obs_update(const ObsArgs& a, hipStream_t st) {
    if (a.M <= 0 || a.N <= 0 || a.K <= 0) return hipSuccess;
    const int64_t tiles_m = (a.M + OTM - 1) / OTM, tiles_n = (a.N + OTN - 1) / OTN;
    hipLaunchKernelGGL(obs_update_kernel, dim3((unsigned)(tiles_m * tiles_n)), dim3(256), 0, st, a, tiles_n);
    return hipGetLastError();
}

}  // namespace realq
