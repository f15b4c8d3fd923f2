// bf16 MFMA "NT" GEMM for gfx950 with fused epilogues.
//
//   acc[i, j] = sum_k (Ahi[i, k] + Alo[i, k]) * B[j, k]          (fp32 accumulation)
//
// Both operands are K-contiguous (row i of A and row j of B hold consecutive k),
// which is the layout every contraction of the sweep is arranged into:
//   residual   R  = B0 + D_J Xhat_J^T      A = split(W - W0)[:, J], B = Xhat[:, J]   (K = |J|)
//   gradient   G  = (R o s) Xhat_J         A = split(R o s),        B = Xhat^T[J, :] (K = tokens)
//   Hessian    H += (s o Xhat)^T Xhat      A = split(s o Xhat^T),   B = Xhat^T       (K = tokens)
//   lock / init of the residual base       A = split(W - W0)[:, blk], B = Xhat[:, blk]
// The float32 operand is carried as a bf16 hi/lo pair and the bf16-exact operand
// (calibration activations) once; both passes reuse the same B fragments, so the
// product is accurate to about 2^-16 relative at twice the MFMA work.
//
// Tiling (two shapes, picked by problem size):
//   large: 256 x 256 block tile, 8 wave64s as 4 (M) x 2 (N), 64 x 128 per wave
//   small: 128 x 128 block tile, 4 wave64s as 2 x 2,        64 x 64 per wave
// with v_mfma_f32_32x32x16_bf16.  K advances in slices of 32 through a ring of three
// LDS stages filled by direct-to-LDS 16-byte loads with explicit vmcnt waits.  The large
// tile runs its K loop as a ping-pong of its two 4-wave groups (one wave of each per
// SIMD): between two barriers one group multiplies a slice from registers while the other
// reads the next fragments out of LDS and issues the next loads, so the matrix pipe of
// every SIMD stays fed while a wave waits on LDS.  The small tile keeps one barrier per
// slice with two slices in flight.  Blocks are renumbered
// so that each XCD (blocks are dealt round-robin over the 8 XCDs) owns a contiguous
// run of tiles, walked in groups of `group_m` row tiles for L2 reuse.  Split-K over
// gridDim.z with a fixed K range per split (deterministic).
#include "common.h"
#include "kernels.h"
#include "plan.h"

namespace realq {

namespace {

constexpr int BK = 32;
constexpr int LDS_STRIDE = BK;      // bf16 per LDS row (64 bytes, unpadded; 16-byte chunks XOR-swizzled)

// Chunk position of 16-byte chunk c of LDS row r.  Fragment reads touch 8 (or 16)
// consecutive rows at one chunk; the swizzle gives them distinct bank groups on both a
// 32- and a 64-bank LDS, and keeps each thread's stage writes conflict-free as well.
__device__ __forceinline__ int swz(int r, int c) { return (c ^ ((r >> 1) ^ (r >> 3))) & 3; }
constexpr int EPI_STRIDE = 36;      // floats per row of the epilogue restaging tile (16-byte aligned)

template <int BM_, int BN_, int WAVES_M_, int WAVES_N_>
struct Cfg {
    static constexpr int BM = BM_, BN = BN_, WAVES_M = WAVES_M_, WAVES_N = WAVES_N_;
    static constexpr int NT = WAVES_M * WAVES_N * 64;
    static constexpr int WTM = BM / WAVES_M, WTN = BN / WAVES_N;  // wave tile
    static constexpr int SM = WTM / 32, SN = WTN / 32;             // 32x32 MFMA tiles per wave
    static constexpr int A_CH = BM * BK / 8 / NT;                  // 16-byte chunks per thread
    static constexpr int B_CH = BN * BK / 8 / NT;
};
using CfgLarge = Cfg<256, 256, 4, 2>;
using CfgSmall = Cfg<128, 128, 2, 2>;
// The 8-wave tile runs its K loop as a ping-pong of two 4-wave groups.
template <class C>
constexpr bool kPingPong = C::WAVES_M == 4 && C::WAVES_N == 2;
__device__ __forceinline__ int64_t imin64(int64_t a, int64_t b) { return a < b ? a : b; }

// element offset of column k in a row: plain, or the blocked hi/lo layout (32 values a block)
__device__ __forceinline__ int64_t kofs_of(int64_t k, bool blk) { return blk ? ((k >> 5) << 6) + (k & 31) : k; }

template <int CH, int NT>
__device__ __forceinline__ void load_rows(u16x8 (&v)[CH], const uint16_t* __restrict__ P, int64_t ld, int64_t rows,
                                          int64_t r0, int64_t k0, int64_t kend, bool vec, bool blk = false) {
#pragma unroll
    for (int c = 0; c < CH; ++c) {
        const int chunk = threadIdx.x + c * NT;
        const int r = chunk >> 2;
        const int kc = (chunk & 3) * 8;
        const int64_t gr = r0 + r;
        const int64_t gk = k0 + kc;
        u16x8 x = {0, 0, 0, 0, 0, 0, 0, 0};
        if (gr < rows) {
            const uint16_t* p = P + gr * ld + kofs_of(gk, blk);
            if (vec && gk + 8 <= kend) {
                x = *reinterpret_cast<const u16x8*>(p);
            } else {
#pragma unroll
                for (int e = 0; e < 8; ++e)
                    if (gk + e < kend) x[e] = p[e];
            }
        }
        v[c] = x;
    }
}

template <int CH, int NT>
__device__ __forceinline__ void store_rows(const u16x8 (&v)[CH], uint16_t* lds) {
#pragma unroll
    for (int c = 0; c < CH; ++c) {
        const int chunk = threadIdx.x + c * NT;
        const int r = chunk >> 2;
        *reinterpret_cast<u16x8*>(lds + r * LDS_STRIDE + swz(r, chunk & 3) * 8) = v[c];
    }
}

__device__ __forceinline__ bf16x8 frag(const uint16_t* lds, int row, int k) {
    return __builtin_bit_cast(bf16x8,
                              *reinterpret_cast<const u16x8*>(lds + row * LDS_STRIDE + swz(row, k >> 3) * 8));
}

// 16-byte direct-to-LDS load: lane i reads sbase + voff (its own 32-bit byte offset) and
// fills LDS bytes [lds + 16i, lds + 16i + 16) (lds is wave-uniform).  Issued as inline
// assembly so the compiler does not insert conservative waits for it; every consumer is
// ordered by the explicit vmcnt waits and barriers of the K loop.
__device__ __forceinline__ void dma16(const void* sbase, uint32_t voff, uint32_t lds) {
    asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(voff), "s"(sbase), "s"(lds)
                 : "memory", "m0");
}
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}
__device__ __forceinline__ void wait_lgkm0() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }
// LDS byte address of a __shared__ object: the low 32 bits of its generic address.
__device__ __forceinline__ uint32_t lds_addr(const void* p) { return (uint32_t)(uintptr_t)p; }

// Tile coordinates of block b: XCD-contiguous renumbering, then grouped row-tile order.
__device__ __forceinline__ void tile_of_v(int64_t b, int64_t tiles_m, int64_t tiles_n, int64_t group_m, int64_t& tm,
                                          int64_t& tn) {
    const int64_t nblk = tiles_m * tiles_n;
    int64_t L = b;
    if ((nblk & 7) == 0) L = (b & 7) * (nblk >> 3) + (b >> 3);
    const int64_t per_group = group_m * tiles_n;
    const int64_t g = L / per_group;
    const int64_t first = g * group_m;
    const int64_t gs = min(group_m, tiles_m - first);
    const int64_t r = L - g * per_group;
    tm = first + r % gs;
    tn = r / gs;
}
__device__ __forceinline__ void tile_of(int64_t tiles_m, int64_t tiles_n, int64_t group_m, int64_t& tm, int64_t& tn) {
    tile_of_v(blockIdx.x, tiles_m, tiles_n, group_m, tm, tn);
}

}  // namespace

template <class C, class Epi, bool HAS_LO>
__global__ __launch_bounds__(C::NT) void gemm_nt_kernel(const uint16_t* __restrict__ Ahi,
                                                        const uint16_t* __restrict__ Alo, int64_t lda,
                                                        const uint16_t* __restrict__ B, int64_t ldb, int64_t M,
                                                        int64_t N, int64_t K, int64_t k_per_split, int vec_ok,
                                                        int64_t tiles_m, int64_t tiles_n, int64_t group_m, int a_blk,
                                                        Epi epi) {
    constexpr int A_ROWS = C::BM * (HAS_LO ? 2 : 1);
    constexpr int STAGE = (A_ROWS + C::BN) * LDS_STRIDE;  // bf16 elements per stage
    // Three LDS stages as separate arrays (the compiler can tell a stage being filled by the
    // direct-to-LDS loads from the one being read), plus epilogue scratch when a stage is
    // too small to hold it.
    constexpr int EPI_FLOATS = (C::NT / 64) * 32 * EPI_STRIDE;
    constexpr bool EPI_IN_STAGE = EPI_FLOATS * 4 <= STAGE * 2 && C::NT * 8 <= STAGE * 2;
    __shared__ __attribute__((aligned(16))) uint16_t st0[STAGE];
    __shared__ __attribute__((aligned(16))) uint16_t st1[STAGE];
    __shared__ __attribute__((aligned(16))) uint16_t st2[STAGE];
    __shared__ __attribute__((aligned(16))) float epi_extra[EPI_IN_STAGE ? 4 : EPI_FLOATS];
    float* const scratch = EPI_IN_STAGE ? reinterpret_cast<float*>(st0) : epi_extra;

    int64_t tm, tn;
    tile_of(tiles_m, tiles_n, group_m, tm, tn);
    const int64_t m0 = tm * C::BM, n0 = tn * C::BN;
    const int64_t kbeg = (int64_t)blockIdx.z * k_per_split;
    const int64_t kend = min(K, kbeg + k_per_split);
    const int64_t nk = kend > kbeg ? (kend - kbeg + BK - 1) / BK : 0;

    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int wm = wave / C::WAVES_N, wn = wave % C::WAVES_N;
    const bool vec = vec_ok != 0;

    f32x16 acc[C::SM][C::SN];
#pragma unroll
    for (int a = 0; a < C::SM; ++a)
#pragma unroll
        for (int b = 0; b < C::SN; ++b)
#pragma unroll
            for (int e = 0; e < 16; ++e) acc[a][b][e] = 0.f;

    // K pipeline.  Full, aligned 32-wide slices are fetched straight into LDS with
    // global_load_lds_dwordx4 (lane i of a wave instruction fills bytes [16i, 16i+16) of a
    // 1 KB run = 16 rows x 4 chunks); the lane picks the global chunk whose swizzled LDS
    // position that is.  Three stages rotate: slice s+2 is in flight while slice s is
    // multiplied and slice s+1 lands.  A partial last slice, or every slice of unaligned
    // operands, goes through the checked register path.
    constexpr int NW = C::NT / 64;
    constexpr int A_RUNS = C::BM / 16 / NW, B_RUNS = C::BN / 16 / NW;  // 1 KB runs per wave per slice
    constexpr int DMA_PER_SLICE = A_RUNS * (HAS_LO ? 2 : 1) + B_RUNS;
    static_assert(C::BM % (16 * NW) == 0 && C::BN % (16 * NW) == 0, "tile rows must split into wave runs");
    // Per-lane byte offsets (fixed for the whole K loop) from wave-uniform operand bases
    // that advance by one slice per step.  Rows past the end are clamped to the last row;
    // their products only reach accumulators the epilogue masks.
    const int wv = __builtin_amdgcn_readfirstlane(wave);
    uint32_t offA[A_RUNS], offB[B_RUNS];
    {
        const int lr = lane >> 2, pc = lane & 3;
#pragma unroll
        for (int q = 0; q < A_RUNS; ++q) {
            const int r = 16 * (wave + NW * q) + lr;
            const int c = pc ^ (((r >> 1) ^ (r >> 3)) & 3);
            const int64_t gr = min(m0 + r, M - 1) - m0;
            offA[q] = (uint32_t)((gr * lda + c * 8) * 2);
        }
#pragma unroll
        for (int q = 0; q < B_RUNS; ++q) {
            const int r = 16 * (wave + NW * q) + lr;
            const int c = pc ^ (((r >> 1) ^ (r >> 3)) & 3);
            const int64_t gr = min(n0 + r, N - 1) - n0;
            offB[q] = (uint32_t)((gr * ldb + c * 8) * 2);
        }
    }
    // A in the blocked hi/lo layout advances 64 values (hi and lo of 32) per slice
    const bool blk = a_blk != 0;
    const int a_sh = __builtin_amdgcn_readfirstlane(blk ? 1 : 0);  // kept scalar for the load addresses
    const int64_t a_step = (int64_t)(BK * 2) << a_sh;               // bytes of A per slice
    const char* const baseA = reinterpret_cast<const char*>(Ahi + m0 * lda + (kbeg << a_sh));
    const char* const baseAl = HAS_LO ? reinterpret_cast<const char*>(Alo + m0 * lda + (kbeg << a_sh)) : baseA;
    const char* const baseB = reinterpret_cast<const char*>(B + n0 * ldb + kbeg);
    const uint32_t lds_st[3] = {lds_addr(st0), lds_addr(st1), lds_addr(st2)};
    auto issue = [&](int64_t s, uint32_t stage) {
        const int64_t off = s * BK * 2;
        const int64_t offa = s * a_step;
#pragma unroll
        for (int q = 0; q < A_RUNS; ++q) {
            const uint32_t d = stage + (uint32_t)((wv + NW * q) * 16 * LDS_STRIDE * 2);
            dma16(baseA + offa, offA[q], d);
            if constexpr (HAS_LO) dma16(baseAl + offa, offA[q], d + C::BM * LDS_STRIDE * 2);
        }
#pragma unroll
        for (int q = 0; q < B_RUNS; ++q)
            dma16(baseB + off, offB[q], stage + (uint32_t)((A_ROWS + (wv + NW * q) * 16) * LDS_STRIDE * 2));
    };
    // wait until at most n direct-to-LDS loads of this wave are outstanding
    auto wait_vm = [](int n) {
        if (n >= DMA_PER_SLICE) wait_vmcnt<DMA_PER_SLICE>();
        else wait_vmcnt<0>();
    };
    struct Frags {
        bf16x8 a[C::SM], al[HAS_LO ? C::SM : 1], b[C::SN];
    };
    auto load_frags = [&](const uint16_t* sA, int kk, Frags& f) {
        const uint16_t* sAl = sA + C::BM * LDS_STRIDE;
        const uint16_t* sB = sA + A_ROWS * LDS_STRIDE;
        const int kofs = kk + 8 * (lane >> 5);
#pragma unroll
        for (int i = 0; i < C::SM; ++i) {
            f.a[i] = frag(sA, wm * C::WTM + i * 32 + (lane & 31), kofs);
            if constexpr (HAS_LO) f.al[i] = frag(sAl, wm * C::WTM + i * 32 + (lane & 31), kofs);
        }
#pragma unroll
        for (int j = 0; j < C::SN; ++j) f.b[j] = frag(sB, wn * C::WTN + j * 32 + (lane & 31), kofs);
    };
    auto mfmas = [&](const Frags& f) {
#pragma unroll
        for (int i = 0; i < C::SM; ++i)
#pragma unroll
            for (int j = 0; j < C::SN; ++j) {
                acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f.a[i], f.b[j], acc[i][j], 0, 0, 0);
                if constexpr (HAS_LO)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f.al[i], f.b[j], acc[i][j], 0, 0, 0);
            }
    };
    auto compute = [&](const uint16_t* sA) {
#pragma unroll
        for (int kk = 0; kk < BK; kk += 16) {
            Frags f;
            load_frags(sA, kk, f);
            mfmas(f);
        }
    };
    // Multiply one stage; the first fragments are read before the refill of another stage
    // is issued, so their LDS latency overlaps the issue of the direct-to-LDS loads.
    static_assert(BK == 32, "the slice step reads two 16-wide fragment sets");
    auto step = [&](int64_t s, bool refill, uint32_t fill, const uint16_t* read) {
        Frags f0, f1;
        load_frags(read, 0, f0);
        if (refill) issue(s, fill);
        load_frags(read, 16, f1);
        mfmas(f0);
        mfmas(f1);
    };
    const int64_t nfull = vec ? (kend - kbeg) / BK : 0;
    if constexpr (kPingPong<C>) {
        // Ping-pong over the two SIMD-sharing wave groups: waves 0-3 and 4-7 sit one per SIMD
        // each (group 0 owns rows 0..127 of the tile, group 1 rows 128..255).  Every wave runs
        // the same loop, "read slice s's fragments out of LDS and refill a stage | barrier |
        // multiply slice s from registers | barrier", but group 1 enters it one barrier later,
        // so between any two barriers one group multiplies while the other reads: on each SIMD
        // one wave keeps the matrix pipe busy while the other waits on LDS and memory.
        //   slice s lives in stage s % 3; each wave issues its share of slice s+2 in its read
        //   phase of slice s (into the stage of slice s-1, which both groups have read by then)
        //   and waits there until its share of slice s+1 has landed, which is before either
        //   group's read phase of slice s+1.
        const int grp = wv >> 2;
        auto mem = [&](int64_t s, const uint16_t* cur, uint32_t fill, Frags& f0, Frags& f1) {
            load_frags(cur, 0, f0);
            load_frags(cur, 16, f1);
            if (s + 2 < nfull) issue(s + 2, fill);
            wait_lgkm0();
            if (s + 2 < nfull) wait_vmcnt<DMA_PER_SLICE>();
            else wait_vmcnt<0>();
        };
        if (nfull > 0) issue(0, lds_st[0]);
        if (nfull > 1) issue(1, lds_st[1]);
        if (nfull > 1) wait_vmcnt<DMA_PER_SLICE>();
        else wait_vmcnt<0>();
        __builtin_amdgcn_s_barrier();
        if (grp == 1) __builtin_amdgcn_s_barrier();
        __builtin_amdgcn_sched_barrier(0);
#define RQ_PP_SLICE(S, CUR, FILL)                       \
    do {                                                \
        Frags f0, f1;                                   \
        mem((S), CUR, lds_st[FILL], f0, f1);            \
        __builtin_amdgcn_sched_barrier(0);              \
        __builtin_amdgcn_s_barrier();                   \
        __builtin_amdgcn_sched_barrier(0);              \
        mfmas(f0);                                      \
        mfmas(f1);                                      \
        __builtin_amdgcn_sched_barrier(0);              \
        __builtin_amdgcn_s_barrier();                   \
        __builtin_amdgcn_sched_barrier(0);              \
    } while (0)
        for (int64_t s = 0; s < nfull; s += 3) {
            RQ_PP_SLICE(s, st0, 2);
            if (s + 1 >= nfull) break;
            RQ_PP_SLICE(s + 1, st1, 0);
            if (s + 2 >= nfull) break;
            RQ_PP_SLICE(s + 2, st2, 1);
        }
#undef RQ_PP_SLICE
        if (grp == 0) __builtin_amdgcn_s_barrier();
    } else {
    // one slice: wait until this slice has landed (the next may stay in flight), barrier (all
    // waves' loads visible; the stage read two slices ago is free), refill it, multiply.
#define RQ_STEP(S, CUR, NXT2)                                      \
    do {                                                           \
        wait_vm((S) + 1 < nfull ? DMA_PER_SLICE : 0);              \
        __builtin_amdgcn_s_barrier();                              \
        step((S) + 2, (S) + 2 < nfull, lds_st[NXT2], CUR);         \
    } while (0)
    if (nfull > 0) issue(0, lds_st[0]);
    if (nfull > 1) issue(1, lds_st[1]);
    for (int64_t s = 0; s < nfull; s += 3) {
        RQ_STEP(s, st0, 2);
        if (s + 1 >= nfull) break;
        RQ_STEP(s + 1, st1, 0);
        if (s + 2 >= nfull) break;
        RQ_STEP(s + 2, st2, 1);
    }
#undef RQ_STEP
    }
    wait_vmcnt<0>();
    __syncthreads();
    for (int64_t s = nfull; s < nk; ++s) {  // checked tail, single-buffered in stage 0
        const int64_t k0 = kbeg + s * BK;
        u16x8 ra[C::A_CH], ral[HAS_LO ? C::A_CH : 1], rb[C::B_CH];
        load_rows<C::A_CH, C::NT>(ra, Ahi, lda, M, m0, k0, kend, vec, blk);
        if constexpr (HAS_LO) load_rows<C::A_CH, C::NT>(ral, Alo, lda, M, m0, k0, kend, vec, blk);
        load_rows<C::B_CH, C::NT>(rb, B, ldb, N, n0, k0, kend, vec);
        store_rows<C::A_CH, C::NT>(ra, st0);
        if constexpr (HAS_LO) store_rows<C::A_CH, C::NT>(ral, st0 + C::BM * LDS_STRIDE);
        store_rows<C::B_CH, C::NT>(rb, st0 + A_ROWS * LDS_STRIDE);
        __syncthreads();
        compute(st0);
        __syncthreads();
    }

    // Epilogue.  Element (row, col) of a 32x32 tile held by this lane in acc[e] is
    // row = 8*(e/4) + 4*(lane/32) + e%4, col = lane%32.  Each tile is restaged through
    // this wave's own LDS scratch so that a lane then owns 4 consecutive columns of a row
    // (16-byte accesses).  The global operands of the epilogue (residual base, per-token
    // weights, the accumulated output) are loaded one sub-tile ahead, so their latency
    // overlaps the restaging and the stores of the current sub-tile.  LDS accesses of one
    // wave complete in order; the wavefront fences only keep the compiler from moving the
    // scratch writes and reads across each other.
    float aux = 0.f;
    float* scr = scratch + wave * (32 * EPI_STRIDE);
    const int64_t z = blockIdx.z;
    // Full tiles of the large shape stream a residual-base epilogue's row operand into LDS with
    // direct-to-LDS loads, three 32x32 sub-tiles ahead per wave (a ring of 3 x 4 KB per wave in
    // stages 1 and 2, freed by the K loop): the register-held prefetch reaches one sub-tile ahead
    // only, and a tile's epilogue then waits out one memory latency per sub-tile.
    constexpr int RING = 3;
    constexpr bool kDma = Epi::kRowDma && C::NT == 512 && EPI_IN_STAGE && STAGE * 2 >= 4 * RING * 4096;
    bool dma_path = false;
    if constexpr (kDma) dma_path = m0 + C::BM <= M && n0 + C::BN <= N && epi.row_dma_ok();
    if constexpr (kDma) {
        if (dma_path) {
            constexpr int NSUB = C::SM * C::SN;
            const int cc = (lane & 7) * 4;
            const int wms = wv / C::WAVES_N, wns = wv % C::WAVES_N;  // scalar copies for the load bases
            // token weights of this wave's columns, consumed before the streamed loads start (the
            // compiler's own waits for them must not wait for those)
            typename Epi::Col cw[C::SN];
#pragma unroll
            for (int j = 0; j < C::SN; ++j) {
                cw[j] = epi.load_col(n0 + wn * C::WTN + j * 32 + cc);
                asm volatile("" ::"v"(cw[j].w[0]), "v"(cw[j].w[1]), "v"(cw[j].w[2]), "v"(cw[j].w[3]));
            }
            const float* const b0 = epi.row_base();
            const int64_t ldb0 = epi.row_ld();
            uint16_t* const ring16 = (wv < 4 ? st1 : st2) + (wv & 3) * (RING * 2048);
            const float* const ring = reinterpret_cast<const float*>(ring16);
            const uint32_t ring_lds = lds_addr(ring16);
            auto dma_sub = [&](int t) {
                const int64_t r0 = m0 + wms * C::WTM + (t / C::SN) * 32;
                const int64_t c0 = n0 + wns * C::WTN + (t % C::SN) * 32;
                const char* base = reinterpret_cast<const char*>(b0 + r0 * ldb0 + c0);
                const uint32_t slot = ring_lds + (uint32_t)((t % RING) * 4096);
#pragma unroll
                for (int q = 0; q < 4; ++q)
                    dma16(base, (uint32_t)(((int64_t)(q * 8 + (lane >> 3)) * ldb0 + (lane & 7) * 4) * 4),
                          slot + q * 1024);
            };
            // vector-memory operations of this lane issued after sub-tile t's streamed loads, at the
            // point where t is consumed (4 loads per sub-tile, kRowStores stores per sub-tile)
            auto after = [](int t) {
                int c = 0;
                if (t < RING) {
                    c += (RING - 1 - t) * 4;
                    for (int u = 0; u < t; ++u) c += Epi::kRowStores + (u + RING < NSUB ? 4 : 0);
                } else {
                    for (int u = t - RING + 1; u < t; ++u) c += Epi::kRowStores + (u + RING < NSUB ? 4 : 0);
                }
                return c;
            };
            static_assert(RING <= NSUB, "ring deeper than the sub-tiles");
#pragma unroll
            for (int t = 0; t < RING; ++t) dma_sub(t);
#pragma unroll
            for (int t = 0; t < NSUB; ++t) {
                switch (after(t)) {  // constant after unrolling
                    case 8: wait_vmcnt<8>(); break;
                    case 16: wait_vmcnt<16>(); break;
                    case 20: wait_vmcnt<20>(); break;
                    case 24: wait_vmcnt<24>(); break;
                    default: wait_vmcnt<0>(); break;
                }
                const int i = t / C::SN, j = t % C::SN;
#pragma unroll
                for (int e = 0; e < 16; ++e)
                    scr[(8 * (e >> 2) + 4 * (lane >> 5) + (e & 3)) * EPI_STRIDE + (lane & 31)] = acc[i][j][e];
                __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
                const int64_t r0 = m0 + wm * C::WTM + i * 32;
                const int64_t col = n0 + wn * C::WTN + j * 32 + cc;
                const float* slot = ring + (t % RING) * 1024;
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const int rr = q * 8 + (lane >> 3);
                    const f32x4 v = *reinterpret_cast<const f32x4*>(scr + rr * EPI_STRIDE + cc);
                    typename Epi::Row rw;
                    rw.b = *reinterpret_cast<const f32x4*>(slot + rr * 32 + cc);
                    rw.ok = true;
                    epi.vec4(r0 + rr, col, v, rw, cw[j], z, aux);
                }
                __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
                if (t + RING < NSUB) {
                    wait_lgkm0();  // this slot's reads are done before it is refilled
                    dma_sub(t + RING);
                }
            }
        }
    }
    if (!dma_path) {
    if constexpr (!Epi::kTransposed) {
        constexpr int NSUB = C::SM * C::SN;
        const int cc = (lane & 7) * 4;
        typename Epi::Row rcur[4], rnxt[4];
        typename Epi::Col ccur, cnxt;
        auto prefetch = [&](int t, typename Epi::Row(&R)[4], typename Epi::Col& Cl) {
            const int64_t r0 = m0 + wm * C::WTM + (t / C::SN) * 32;
            const int64_t col = n0 + wn * C::WTN + (t % C::SN) * 32 + cc;
            const bool colv = col + 3 < N;
            if (colv) Cl = epi.load_col(col);
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int64_t row = r0 + q * 8 + (lane >> 3);
                if (colv && row < M) R[q] = epi.load_row(row, col, z);
                else R[q].ok = false;
            }
        };
        prefetch(0, rcur, ccur);
#pragma unroll
        for (int t = 0; t < NSUB; ++t) {
            if (t + 1 < NSUB) prefetch(t + 1, rnxt, cnxt);
            const int i = t / C::SN, j = t % C::SN;
#pragma unroll
            for (int e = 0; e < 16; ++e)
                scr[(8 * (e >> 2) + 4 * (lane >> 5) + (e & 3)) * EPI_STRIDE + (lane & 31)] = acc[i][j][e];
            __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
            const int64_t r0 = m0 + wm * C::WTM + i * 32;
            const int64_t col = n0 + wn * C::WTN + j * 32 + cc;
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int rr = q * 8 + (lane >> 3);
                const int64_t row = r0 + rr;
                const f32x4 v = *reinterpret_cast<const f32x4*>(scr + rr * EPI_STRIDE + cc);
                if (row < M) {
                    if (rcur[q].ok) {
                        epi.vec4(row, col, v, rcur[q], ccur, z, aux);
                    } else {
#pragma unroll
                        for (int u = 0; u < 4; ++u)
                            if (col + u < N) epi(row, col + u, v[u], z, aux);
                    }
                }
            }
            __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
#pragma unroll
            for (int q = 0; q < 4; ++q) rcur[q] = rnxt[q];
            ccur = cnxt;
        }
    } else {
#pragma unroll
        for (int i = 0; i < C::SM; ++i)
#pragma unroll
            for (int j = 0; j < C::SN; ++j) {
#pragma unroll
                for (int e = 0; e < 16; ++e)
                    scr[(8 * (e >> 2) + 4 * (lane >> 5) + (e & 3)) * EPI_STRIDE + (lane & 31)] = acc[i][j][e];
                __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
                const int64_t r0 = m0 + wm * C::WTM + i * 32;
                const int64_t c0 = n0 + wn * C::WTN + j * 32;
                // lane owns 4 consecutive rows of one column (outputs stored column-major)
                const int rr = (lane & 7) * 4;
                const int64_t row = r0 + rr;
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const int cc = q * 8 + (lane >> 3);
                    const int64_t col = c0 + cc;
                    f32x4 v;
#pragma unroll
                    for (int u = 0; u < 4; ++u) v[u] = scr[(rr + u) * EPI_STRIDE + cc];
                    if (col < N) {
                        if (row + 3 < M) {
                            epi.vec4t(row, col, v, z, aux);
                        } else {
#pragma unroll
                            for (int u = 0; u < 4; ++u)
                                if (row + u < M) epi(row + u, col, v[u], z, aux);
                        }
                    }
                }
                __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
            }
    }
    }  // !dma_path
    if constexpr (Epi::kReduce) {
        // deterministic block reduction of the per-thread partial sums, in stage 0 past the
        // restaging scratch when it fits there (stages 1 and 2 may still feed other waves'
        // epilogues), else in stage 1
        constexpr bool RED0 = EPI_IN_STAGE && (C::NT / 64) * 32 * EPI_STRIDE * 4 + C::NT * 8 <= STAGE * 2;
        double* red = RED0 ? reinterpret_cast<double*>(reinterpret_cast<char*>(st0) + (C::NT / 64) * 32 * EPI_STRIDE * 4)
                           : reinterpret_cast<double*>(st1);
        red[threadIdx.x] = (double)aux;
        __syncthreads();
        for (int s = C::NT / 2; s > 0; s >>= 1) {
            if (threadIdx.x < s) red[threadIdx.x] += red[threadIdx.x + s];
            __syncthreads();
        }
        if (threadIdx.x == 0) epi.partial(blockIdx.x + (int64_t)blockIdx.z * gridDim.x, red[0]);
    }
}

// ---------------------------------------------------------------- epilogues
// Row-major epilogues: operator() handles one element.  The fast path handles columns
// j..j+3 of row i in three parts: load_col(j) and load_row(i, j, z) fetch the global
// operands ahead of time (ok = false sends the lane to operator() instead, e.g. for an
// unaligned address), vec4() combines them with the accumulators and stores.

__device__ __forceinline__ bool al16(const void* p) { return (((uintptr_t)p) & 15u) == 0; }
__device__ __forceinline__ bool al8(const void* p) { return (((uintptr_t)p) & 7u) == 0; }
typedef uint16_t u16x4 __attribute__((ext_vector_type(4)));

struct NoCol {};

struct EpiStoreF32 {  // C[z][i][j] = alpha * acc
    static constexpr bool kRowDma = false;
    static constexpr bool kReduce = false;
    static constexpr bool kTransposed = false;
    float* C;
    int64_t ldc, split_stride;
    float alpha;
    struct Row {
        bool ok;
    };
    using Col = NoCol;
    __device__ void operator()(int64_t i, int64_t j, float v, int64_t z, float&) const {
        C[z * split_stride + i * ldc + j] = alpha * v;
    }
    __device__ Col load_col(int64_t) const { return {}; }
    __device__ Row load_row(int64_t i, int64_t j, int64_t z) const {
        return {al16(C + z * split_stride + i * ldc + j)};
    }
    __device__ void vec4(int64_t i, int64_t j, f32x4 v, const Row&, const Col&, int64_t z, float&) const {
        *reinterpret_cast<f32x4*>(C + z * split_stride + i * ldc + j) = v * alpha;
    }
    __device__ void partial(int64_t, double) const {}
};

// Gradient slices of the split-K token reduction: G[z][i][j] = acc (same as EpiStoreF32,
// kept as its own type so the gradient GEMM is a kernel of its own in traces).
struct EpiGrad : EpiStoreF32 {};

struct EpiAccF32 {  // C[i][j] += alpha * acc
    static constexpr bool kRowDma = false;
    static constexpr bool kReduce = false;
    static constexpr bool kTransposed = false;
    float* C;
    int64_t ldc;
    float alpha;
    struct Row {
        f32x4 c;
        bool ok;
    };
    using Col = NoCol;
    __device__ void operator()(int64_t i, int64_t j, float v, int64_t, float&) const { C[i * ldc + j] += alpha * v; }
    __device__ Col load_col(int64_t) const { return {}; }
    __device__ Row load_row(int64_t i, int64_t j, int64_t) const {
        Row r;
        const float* p = C + i * ldc + j;
        r.ok = al16(p);
        if (r.ok) r.c = *reinterpret_cast<const f32x4*>(p);
        return r;
    }
    __device__ void vec4(int64_t i, int64_t j, f32x4 v, const Row& r, const Col&, int64_t, float&) const {
        *reinterpret_cast<f32x4*>(C + i * ldc + j) = r.c + v * alpha;
    }
    __device__ void partial(int64_t, double) const {}
};

struct EpiAccF64 {  // C[i][j] += acc   (float64 accumulator across chunks)
    static constexpr bool kRowDma = false;
    static constexpr bool kReduce = false;
    static constexpr bool kTransposed = false;
    double* C;
    int64_t ldc;
    struct Row {
        bool ok;
    };
    using Col = NoCol;
    __device__ void operator()(int64_t i, int64_t j, float v, int64_t, float&) const { C[i * ldc + j] += (double)v; }
    __device__ Col load_col(int64_t) const { return {}; }
    __device__ Row load_row(int64_t, int64_t, int64_t) const { return {false}; }
    __device__ void vec4(int64_t, int64_t, f32x4, const Row&, const Col&, int64_t, float&) const {}
    __device__ void partial(int64_t, double) const {}
};

// Per-token weights of columns t..t+3 (1 without weights).
struct TokW {
    f32x4 w;
    bool ok;
};
__device__ __forceinline__ TokW load_tokw(const float* s, int64_t t) {
    TokW c;
    c.w = f32x4{1.f, 1.f, 1.f, 1.f};
    c.ok = true;
    if (s) {
        c.ok = al16(s + t);
        if (c.ok) c.w = *reinterpret_cast<const f32x4*>(s + t);
    }
    return c;
}

// Residual: R = B0[i][t] + acc; writes split(R * s_t) and accumulates s_t R^2.
// With blk, split(R o s) goes to one array of 128-byte lines: 32 tokens' hi, then their lo.
struct EpiResid {
    static constexpr bool kRowDma = true;  // residual base streamed into LDS by full tiles
    static constexpr int kRowStores = 8;   // store instructions per lane and 32x32 sub-tile (4 rows x hi, lo)
    static constexpr bool kReduce = true;
    static constexpr bool kTransposed = false;
    const float* B0;
    int64_t ldb0;
    const float* s;
    uint16_t* Rhi;
    uint16_t* Rlo;
    int64_t ldr;
    double* partials;
    bool blk;
    struct Row {
        f32x4 b;
        bool ok;
    };
    using Col = TokW;
    __device__ uint16_t* hi_at(int64_t i, int64_t t) const {
        return blk ? Rhi + i * ldr + ((t >> 5) << 6) + (t & 31) : Rhi + i * ldr + t;
    }
    __device__ uint16_t* lo_at(int64_t i, int64_t t) const { return blk ? hi_at(i, t) + 32 : Rlo + i * ldr + t; }
    __device__ const float* row_base() const { return B0; }
    __device__ int64_t row_ld() const { return ldb0; }
    // every row of a full tile may take the streamed path: 16-byte base rows within 32-bit
    // offsets of a sub-tile's first row, 8-byte output quads
    __device__ bool row_dma_ok() const {
        const bool out = blk ? (al8(Rhi) && ldr % 64 == 0) : (al8(Rhi) && al8(Rlo) && ldr % 4 == 0);
        return al16(B0) && ldb0 % 4 == 0 && ldb0 < (int64_t(1) << 24) && out;
    }
    __device__ void operator()(int64_t i, int64_t t, float v, int64_t, float& aux) const {
        float r = B0[i * ldb0 + t] + v;
        float w = s ? s[t] : 1.f;
        float rs = r * w;
        uint16_t hi, lo;
        split_bf16(rs, hi, lo);
        *hi_at(i, t) = hi;
        *lo_at(i, t) = lo;
        aux += rs * r;
    }
    __device__ Col load_col(int64_t t) const { return load_tokw(s, t); }
    __device__ Row load_row(int64_t i, int64_t t, int64_t) const {
        Row r;
        const float* b = B0 + i * ldb0 + t;
        r.ok = al16(b) && al8(hi_at(i, t)) && al8(lo_at(i, t));
        if (r.ok) r.b = *reinterpret_cast<const f32x4*>(b);
        return r;
    }
    __device__ void vec4(int64_t i, int64_t t, f32x4 v, const Row& row, const Col& col, int64_t z, float& aux) const {
        if (!col.ok) {
            for (int u = 0; u < 4; ++u) (*this)(i, t + u, v[u], z, aux);
            return;
        }
        const f32x4 r = row.b + v;
        u16x4 h, l;
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const float rs = r[u] * col.w[u];
            uint16_t hh, ll;
            split_bf16(rs, hh, ll);
            h[u] = hh;
            l[u] = ll;
            aux += rs * r[u];
        }
        *reinterpret_cast<u16x4*>(hi_at(i, t)) = h;
        *reinterpret_cast<u16x4*>(lo_at(i, t)) = l;
    }
    __device__ void partial(int64_t b, double v) const { partials[b] = v; }
};

// A later step of a column block: acc = bf16(W_k - W_0) Xhat^T is the change of the residual since
// the block's first step.  Writes bf16(acc * s_t) row-major [i * ldq + t] for the gradient GEMM
// and accumulates s_t acc^2, the part of the step's loss that the block's first residual and
// gradient do not give (the caller adds them).
struct EpiResidInc {
    static constexpr bool kRowDma = false;
    static constexpr bool kReduce = true;
    static constexpr bool kTransposed = false;
    const float* s;
    uint16_t* Q;
    int64_t ldq;
    double* partials;
    struct Row {
        bool ok;
    };
    using Col = TokW;
    __device__ void operator()(int64_t i, int64_t t, float v, int64_t, float& aux) const {
        const float w = s ? s[t] : 1.f;
        const float vs = v * w;
        Q[i * ldq + t] = f2bf(vs);
        aux += vs * v;
    }
    __device__ Col load_col(int64_t t) const { return load_tokw(s, t); }
    __device__ Row load_row(int64_t i, int64_t t, int64_t) const { return {al8(Q + i * ldq + t)}; }
    __device__ void vec4(int64_t i, int64_t t, f32x4 v, const Row&, const Col& col, int64_t z, float& aux) const {
        if (!col.ok) {
            for (int u = 0; u < 4; ++u) (*this)(i, t + u, v[u], z, aux);
            return;
        }
        u16x4 q;
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const float vs = v[u] * col.w[u];
            q[u] = f2bf(vs);
            aux += vs * v[u];
        }
        *reinterpret_cast<u16x4*>(Q + i * ldq + t) = q;
    }
    __device__ void partial(int64_t b, double v) const { partials[b] = v; }
};

// Residual kept whole in float32: R[i][t] = B0[i][t] + acc (for the output-perturbation clip).
struct EpiResidF32 {
    static constexpr bool kRowDma = false;
    static constexpr bool kReduce = false;
    static constexpr bool kTransposed = false;
    const float* B0;
    int64_t ldb0;
    float* R;
    int64_t ldr;
    struct Row {
        f32x4 b;
        bool ok;
    };
    using Col = NoCol;
    __device__ void operator()(int64_t i, int64_t t, float v, int64_t, float&) const {
        R[i * ldr + t] = B0[i * ldb0 + t] + v;
    }
    __device__ Col load_col(int64_t) const { return {}; }
    __device__ Row load_row(int64_t i, int64_t t, int64_t) const {
        Row r;
        const float* b = B0 + i * ldb0 + t;
        r.ok = al16(b) && al16(R + i * ldr + t);
        if (r.ok) r.b = *reinterpret_cast<const f32x4*>(b);
        return r;
    }
    __device__ void vec4(int64_t i, int64_t t, f32x4 v, const Row& row, const Col&, int64_t, float&) const {
        *reinterpret_cast<f32x4*>(R + i * ldr + t) = row.b + v;
    }
    __device__ void partial(int64_t, double) const {}
};

// Residual loss only (no outputs besides the partial sums): s_t (B0 + acc)^2.
struct EpiLoss {
    static constexpr bool kRowDma = false;
    static constexpr bool kReduce = true;
    static constexpr bool kTransposed = false;
    const float* B0;
    int64_t ldb0;
    const float* s;
    double* partials;
    struct Row {
        f32x4 b;
        bool ok;
    };
    using Col = TokW;
    __device__ void operator()(int64_t i, int64_t t, float v, int64_t, float& aux) const {
        float r = B0[i * ldb0 + t] + v;
        float w = s ? s[t] : 1.f;
        aux += w * r * r;
    }
    __device__ Col load_col(int64_t t) const { return load_tokw(s, t); }
    __device__ Row load_row(int64_t i, int64_t t, int64_t) const {
        Row r;
        const float* b = B0 + i * ldb0 + t;
        r.ok = al16(b);
        if (r.ok) r.b = *reinterpret_cast<const f32x4*>(b);
        return r;
    }
    __device__ void vec4(int64_t i, int64_t t, f32x4 v, const Row& row, const Col& col, int64_t z, float& aux) const {
        if (!col.ok) {
            for (int u = 0; u < 4; ++u) (*this)(i, t + u, v[u], z, aux);
            return;
        }
        const f32x4 r = row.b + v;
#pragma unroll
        for (int u = 0; u < 4; ++u) aux += col.w[u] * r[u] * r[u];
    }
    __device__ void partial(int64_t b, double v) const { partials[b] = v; }
};

// Token-major outputs of the module hand-off (acc[i][j] is output channel i of token j):
// a lane holds rows i..i+3 of one column j and stores them contiguously at out[j*ld + i].

// out[j][i] = bf16(acc + add[j][i])   (add may be NULL; same layout as out)
struct EpiStoreBf16T {
    static constexpr bool kRowDma = false;
    static constexpr bool kReduce = false;
    static constexpr bool kTransposed = true;
    uint16_t* out;
    int64_t ld;
    const float* add;
    __device__ void operator()(int64_t i, int64_t j, float v, int64_t, float&) const {
        out[j * ld + i] = f2bf(add ? v + add[j * ld + i] : v);
    }
    __device__ void vec4t(int64_t i, int64_t j, f32x4 v, int64_t z, float& aux) const {
        uint16_t* p = out + j * ld + i;
        if (add) {
            const float* a = add + j * ld + i;
            if (!al16(a)) {
                for (int u = 0; u < 4; ++u) (*this)(i + u, j, v[u], z, aux);
                return;
            }
            const f32x4 av = *reinterpret_cast<const f32x4*>(a);
            for (int u = 0; u < 4; ++u) v[u] += av[u];
        }
        if (al8(p)) {
            u16x4 h = {f2bf(v[0]), f2bf(v[1]), f2bf(v[2]), f2bf(v[3])};
            *reinterpret_cast<u16x4*>(p) = h;
        } else {
            for (int u = 0; u < 4; ++u) (*this)(i + u, j, v[u], z, aux);
        }
    }
    __device__ void partial(int64_t, double) const {}
};

// out[j][i] = acc + add[j][i] (float32; the gate pre-activation of a SwiGLU hand-off; add may
// be NULL or equal to out: each element is read and written by the same lane)
struct EpiStoreF32T {
    static constexpr bool kRowDma = false;
    static constexpr bool kReduce = false;
    static constexpr bool kTransposed = true;
    float* out;
    int64_t ld;
    const float* add;
    __device__ void operator()(int64_t i, int64_t j, float v, int64_t, float&) const {
        out[j * ld + i] = add ? v + add[j * ld + i] : v;
    }
    __device__ void vec4t(int64_t i, int64_t j, f32x4 v, int64_t z, float& aux) const {
        float* p = out + j * ld + i;
        const float* a = add ? add + j * ld + i : nullptr;
        if (al16(p) && (!a || al16(a))) {
            if (a) {
                const f32x4 av = *reinterpret_cast<const f32x4*>(a);
                for (int u = 0; u < 4; ++u) v[u] += av[u];
            }
            *reinterpret_cast<f32x4*>(p) = v;
        } else {
            for (int u = 0; u < 4; ++u) (*this)(i + u, j, v[u], z, aux);
        }
    }
    __device__ void partial(int64_t, double) const {}
};

// SwiGLU hand-off: out[j][i] = bf16(silu(G[j][i]) * acc), silu(g) = g / (1 + e^-g).
struct EpiSwiGLUT {
    static constexpr bool kRowDma = false;
    static constexpr bool kReduce = false;
    static constexpr bool kTransposed = true;
    const float* G;
    int64_t ldg;
    uint16_t* out;
    int64_t ld;
    __device__ static float silu(float g) { return g / (1.f + expf(-g)); }
    __device__ void operator()(int64_t i, int64_t j, float v, int64_t, float&) const {
        out[j * ld + i] = f2bf(silu(G[j * ldg + i]) * v);
    }
    __device__ void vec4t(int64_t i, int64_t j, f32x4 v, int64_t z, float& aux) const {
        const float* g = G + j * ldg + i;
        uint16_t* p = out + j * ld + i;
        if (al16(g) && al8(p)) {
            const f32x4 gv = *reinterpret_cast<const f32x4*>(g);
            u16x4 h;
            for (int u = 0; u < 4; ++u) h[u] = f2bf(silu(gv[u]) * v[u]);
            *reinterpret_cast<u16x4*>(p) = h;
        } else {
            for (int u = 0; u < 4; ++u) (*this)(i + u, j, v[u], z, aux);
        }
    }
    __device__ void partial(int64_t, double) const {}
};

// ---------------------------------------------------------------- launchers

static inline bool aligned16(const void* p) { return (((uintptr_t)p) & 15u) == 0; }

// Tile choice and split-K arithmetic are the host-side plan's (plan.h), so that the
// workspace sizes the entry points derive from it describe exactly these launches.
static_assert(CfgLarge::BM == plan::kLargeBM && CfgLarge::BN == plan::kLargeBN, "large tile differs from the plan");
static_assert(CfgSmall::BM == plan::kSmallBM && CfgSmall::BN == plan::kSmallBN, "small tile differs from the plan");
static_assert(BK == plan::kBK, "K slice differs from the plan");

int64_t gemm_num_blocks(int64_t M, int64_t N, int tile) { return plan::num_blocks(M, N, tile); }

int64_t gemm_effective_splits(int64_t K, int64_t splits) { return plan::effective_splits(K, splits); }

template <class C, class Epi>
static hipError_t launch_cfg(const GemmArgs& g, const Epi& epi, hipStream_t stream) {
    const int64_t tiles_m = (g.M + C::BM - 1) / C::BM, tiles_n = (g.N + C::BN - 1) / C::BN;
    const int64_t kps = plan::k_per_split(g.K, g.splits);
    const int64_t splits = plan::effective_splits(g.K, g.splits);
    // The direct-to-LDS path addresses a tile's rows with 32-bit byte offsets from the tile's
    // first row; larger strides take the checked register path.
    const bool offsets32 = (int64_t)C::BM * g.lda * 2 < (int64_t(1) << 32) && (int64_t)C::BN * g.ldb * 2 < (int64_t(1) << 32);
    const bool vec = aligned16(g.Ahi) && (!g.Alo || aligned16(g.Alo)) && aligned16(g.B) && (g.lda % 8 == 0) &&
                     (g.ldb % 8 == 0) && offsets32;
    // row-tile group: enough row tiles per group that ~32 concurrent blocks of an XCD share operands
    int64_t group_m = tiles_n >= 32 ? 8 : (tiles_n >= 8 ? 2 : 1);
    if (g.group_m > 0) group_m = g.group_m;
    dim3 grid((unsigned)(tiles_m * tiles_n), 1, (unsigned)splits);
    if (g.Alo)
        hipLaunchKernelGGL((gemm_nt_kernel<C, Epi, true>), grid, dim3(C::NT), 0, stream, g.Ahi, g.Alo, g.lda, g.B,
                           g.ldb, g.M, g.N, g.K, kps, (int)vec, tiles_m, tiles_n, group_m, g.a_blocked, epi);
    else
        hipLaunchKernelGGL((gemm_nt_kernel<C, Epi, false>), grid, dim3(C::NT), 0, stream, g.Ahi, g.Alo, g.lda, g.B,
                           g.ldb, g.M, g.N, g.K, kps, (int)vec, tiles_m, tiles_n, group_m, g.a_blocked, epi);
    return hipGetLastError();
}

template <class Epi>
static hipError_t launch(const GemmArgs& g, const Epi& epi, hipStream_t stream) {
    if (g.M <= 0 || g.N <= 0) return hipSuccess;
    if (plan::pick_large(g.M, g.N, g.tile)) return launch_cfg<CfgLarge>(g, epi, stream);
    return launch_cfg<CfgSmall>(g, epi, stream);
}

hipError_t gemm_store_f32(const GemmArgs& g, float* C, int64_t ldc, int64_t split_stride, float alpha,
                          hipStream_t st) {
    return launch(g, EpiStoreF32{C, ldc, split_stride, alpha}, st);
}
int64_t gemm_grad_blocks(int64_t M, int64_t N) { return plan::tiles(M, N, true); }
hipError_t gemm_grad(const GemmArgs& g, float* C, int64_t ldc, int64_t split_stride, hipStream_t st) {
    if (g.M <= 0 || g.N <= 0) return hipSuccess;
    EpiGrad e;
    e.C = C;
    e.ldc = ldc;
    e.split_stride = split_stride;
    e.alpha = 1.f;
    return launch_cfg<CfgLarge>(g, e, st);  // always the large tile (split-K fills the chip)
}
hipError_t gemm_acc_f32(const GemmArgs& g, float* C, int64_t ldc, float alpha, hipStream_t st) {
    return launch(g, EpiAccF32{C, ldc, alpha}, st);
}
hipError_t gemm_acc_f64(const GemmArgs& g, double* C, int64_t ldc, hipStream_t st) {
    return launch(g, EpiAccF64{C, ldc}, st);
}
hipError_t gemm_resid_f32(const GemmArgs& g, const float* B0, int64_t ldb0, float* R, int64_t ldr, hipStream_t st) {
    return launch(g, EpiResidF32{B0, ldb0, R, ldr}, st);
}
hipError_t gemm_resid(const GemmArgs& g, const float* B0, int64_t ldb0, const float* s, uint16_t* Rhi, uint16_t* Rlo,
                      int64_t ldr, double* partials, hipStream_t st, bool blocked) {
    if (blocked && (ldr % 64 != 0 || g.N > ldr / 2)) return hipErrorInvalidValue;
    return launch(g, EpiResid{B0, ldb0, s, Rhi, Rlo, ldr, partials, blocked}, st);
}
hipError_t gemm_resid_inc(const GemmArgs& g, const float* s, uint16_t* Q, int64_t ldq, double* partials,
                          hipStream_t st) {
    return launch(g, EpiResidInc{s, Q, ldq, partials}, st);
}
hipError_t gemm_loss(const GemmArgs& g, const float* B0, int64_t ldb0, const float* s, double* partials,
                     hipStream_t st) {
    return launch(g, EpiLoss{B0, ldb0, s, partials}, st);
}
hipError_t gemm_store_bf16_t(const GemmArgs& g, uint16_t* out, int64_t ld, hipStream_t st, const float* add) {
    return launch(g, EpiStoreBf16T{out, ld, add}, st);
}
hipError_t gemm_store_f32_t(const GemmArgs& g, float* out, int64_t ld, hipStream_t st, const float* add) {
    return launch(g, EpiStoreF32T{out, ld, add}, st);
}
hipError_t gemm_swiglu_t(const GemmArgs& g, const float* G, int64_t ldg, uint16_t* out, int64_t ld, hipStream_t st) {
    return launch(g, EpiSwiGLUT{G, ldg, out, ld}, st);
}

}  // namespace realq
