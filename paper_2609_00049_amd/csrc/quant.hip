// Quantization of one column block (Alg. 1 inner loop; Sec. 3.2 Eq. gptq_update).
//
// One wave64 owns one weight row at a time; lane l holds block columns l and l+64
// in registers.  Per row:
//   1. dead columns of the block are zeroed;
//   2. when a quantization group starts, its (scale, zero) pair is searched in
//      float64: lanes split the shrink factors p_k = 1 - k/100 (lane l takes k = l and
//      k = l + 64), every lane scores all zero points of its k over the group's
//      values (broadcast with readlane), and a wave reduction picks the
//      lexicographic minimum of (err, k, |z - z_nat(k)|, z);
//   3. columns are quantized in order, q = clamp(rint(w/s) + z, 0, maxq),
//      w_hat = s (q - z), and the error e = (w - w_hat) / U_jj is propagated to the
//      block's later columns with row j of the inverse factor U (held in LDS);
//   4. w_hat, codes, the block error E and the bf16 split of w_hat - W0 are written.
#include "common.h"
#include "kernels.h"

namespace realq {

namespace {
constexpr int QB = 128;          // maximum block width
constexpr int WAVES = 4;
constexpr int ROWS_PER_WAVE = 4;
constexpr int ROWS_PER_WG = WAVES * ROWS_PER_WAVE;

__device__ __forceinline__ float bcast(float v, int lane) {
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), lane));
}

struct Best {
    double err;
    int k, dist, z;
};

__device__ __forceinline__ bool better(const Best& a, const Best& b) {
    if (a.err != b.err) return a.err < b.err;
    if (a.k != b.k) return a.k < b.k;
    if (a.dist != b.dist) return a.dist < b.dist;
    return a.z < b.z;
}

// Per-lane state of the search for one group.
struct Search {
    double lo, hi;
    double s[2], inv[2];
    int kk[2];
    bool valid[2];
    double err[2][16];
};

}  // namespace

template <int MAXQ>
__device__ __forceinline__ void search_accumulate(Search& S, double x) {
#pragma unroll
    for (int a = 0; a < 2; ++a) {
        if (!S.valid[a]) continue;
        const double r = rint(x * S.inv[a]);
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
__device__ __forceinline__ void search_begin(Search& S, double lo, double hi, int grid, int lane) {
    lo = fmin(0.0, lo);
    hi = fmax(0.0, hi);
    if (lo == hi) {
        lo = -1.0;
        hi = 1.0;
    }
    S.lo = lo;
    S.hi = hi;
#pragma unroll
    for (int a = 0; a < 2; ++a) {
        const int k = lane + 64 * a;
        S.kk[a] = k;
        S.valid[a] = k < grid;
        const double p = 1.0 - (double)k / 100.0;
        S.s[a] = (p * (hi - lo)) / (double)MAXQ;
        S.inv[a] = 1.0 / S.s[a];
#pragma unroll
        for (int z = 0; z <= MAXQ; ++z) S.err[a][z] = 0.0;
    }
}

// Reduce the per-lane candidates to the winner; returns (scale, zero) in all lanes.
template <int MAXQ>
__device__ __forceinline__ void search_finish(const Search& S, double& scale, int& zero) {
    Best best{INFINITY, 1 << 30, 1 << 30, 1 << 30};
#pragma unroll
    for (int a = 0; a < 2; ++a) {
        if (!S.valid[a]) continue;
        const double p = 1.0 - (double)S.kk[a] / 100.0;
        double zn = rint(-(p * S.lo) / S.s[a]);
        zn = fmin(fmax(zn, 0.0), (double)MAXQ);
        const int znat = (int)zn;
#pragma unroll
        for (int z = 0; z <= MAXQ; ++z) {
            Best c{S.err[a][z], S.kk[a], abs(z - znat), z};
            if (better(c, best)) best = c;
        }
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
        Best o;
        o.err = __shfl_xor(best.err, off);
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
        float* Wrow = q.W + i * n;
        const bool in0 = lane < bs, in1 = lane + 64 < bs;
        float w0 = in0 ? Wrow[c0 + lane] : 0.f;
        float w1 = in1 ? Wrow[c0 + 64 + lane] : 0.f;
        if (q.dead) {
            if (in0 && q.dead[c0 + lane]) w0 = 0.f;
            if (in1 && q.dead[c0 + 64 + lane]) w1 = 0.f;
        }
        float scale = 1.f;
        float zf = 0.f;
        if (c0 % group != 0) {  // group started in an earlier block: reuse its parameters
            const int64_t g = c0 / group;
            scale = q.scales[i * q.ngroups + g];
            zf = (float)q.zeros[i * q.ngroups + g];
        }
        float e0 = 0.f, e1 = 0.f;
        uint8_t code0 = 0, code1 = 0;
        for (int64_t j = 0; j < bs; ++j) {
            const int64_t col = c0 + j;
            if (col % group == 0) {
                // ---- (scale, zero) search over the group's current values
                const int64_t glen = min(group, n - col);
                Search S;
                double lo = INFINITY, hi = -INFINITY;
                if (j + glen <= bs) {
                    // whole group inside the block: values in registers
                    for (int64_t e = 0; e < glen; ++e) {
                        const int64_t jj = j + e;
                        const float x = bcast(jj < 64 ? w0 : w1, (int)(jj & 63));
                        lo = fmin(lo, (double)x);
                        hi = fmax(hi, (double)x);
                    }
                    search_begin<MAXQ>(S, lo, hi, q.grid, lane);
                    for (int64_t e = 0; e < glen; ++e) {
                        const int64_t jj = j + e;
                        const float x = bcast(jj < 64 ? w0 : w1, (int)(jj & 63));
                        search_accumulate<MAXQ>(S, (double)x);
                    }
                } else {
                    // group extends past the block (only at j == 0): read the untouched row
                    for (int64_t e0c = 0; e0c < glen; e0c += 64) {
                        const int64_t cc = col + e0c + lane;
                        float v = 0.f;
                        if (e0c + lane < glen) {
                            v = Wrow[cc];
                            if (q.dead && q.dead[cc]) v = 0.f;
                        }
                        const int cnt = (int)min((int64_t)64, glen - e0c);
                        for (int e = 0; e < cnt; ++e) {
                            const float x = bcast(v, e);
                            lo = fmin(lo, (double)x);
                            hi = fmax(hi, (double)x);
                        }
                    }
                    search_begin<MAXQ>(S, lo, hi, q.grid, lane);
                    for (int64_t e0c = 0; e0c < glen; e0c += 64) {
                        const int64_t cc = col + e0c + lane;
                        float v = 0.f;
                        if (e0c + lane < glen) {
                            v = Wrow[cc];
                            if (q.dead && q.dead[cc]) v = 0.f;
                        }
                        const int cnt = (int)min((int64_t)64, glen - e0c);
                        for (int e = 0; e < cnt; ++e) search_accumulate<MAXQ>(S, (double)bcast(v, e));
                    }
                }
                double sd;
                int zi;
                search_finish<MAXQ>(S, sd, zi);
                scale = (float)sd;
                zf = (float)zi;
                if (lane == 0) {
                    q.scales[i * q.ngroups + col / group] = scale;
                    q.zeros[i * q.ngroups + col / group] = (uint8_t)zi;
                }
            }
            // ---- quantize column j and compensate the block's later columns
            const float wj = bcast(j < 64 ? w0 : w1, (int)(j & 63));
            const float qv = fminf(fmaxf(rintf(wj / scale) + zf, 0.f), (float)MAXQ);
            const float wq = scale * (qv - zf);
            const float err = (wj - wq) / sU[j * QB + j];
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
            if (lane > j && in0) w0 = fmaf(-err, sU[j * QB + lane], w0);
            if (lane + 64 > j && in1) w1 = fmaf(-err, sU[j * QB + lane + 64], w1);
        }
        // ---- write back
        if (in0) {
            const int64_t c = c0 + lane;
            Wrow[c] = w0;
            q.codes[i * n + c] = code0;
            q.E[i * bs + lane] = e0;
            if (q.Dhi) {
                uint16_t h, l;
                split_bf16(w0 - q.W0[i * n + c], h, l);
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
                split_bf16(w1 - q.W0[i * n + c], h, l);
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

}  // namespace realq
