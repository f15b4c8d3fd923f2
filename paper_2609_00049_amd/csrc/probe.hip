// realq_mfma_peak: the bf16 MFMA rate this GPU sustains on a register-resident loop, the
// achievable ceiling that the benchmark reports beside the data-sheet peak.  Every wave runs
// `iters` rounds of eight independent v_mfma_f32_32x32x16_bf16 chains (enough in flight to cover
// the instruction's latency), with no memory traffic inside the loop.
#include "common.h"
#include "ctx.h"
#include "../../include/realq.h"

namespace {

constexpr int kChains = 8;
constexpr int kWavesPerBlock = 8;   // two waves per SIMD, as the sweep's GEMM runs

__global__ __launch_bounds__(64 * kWavesPerBlock) void mfma_peak_kernel(int64_t iters, float* out) {
    using namespace realq;
    const int lane = threadIdx.x & 63;
    bf16x8 a, b;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        a[e] = (__bf16)(0.001f * (float)((lane * 8 + e) % 17));
        b[e] = (__bf16)(0.001f * (float)((lane * 5 + e) % 13));
    }
    f32x16 acc[kChains];
#pragma unroll
    for (int c = 0; c < kChains; ++c)
#pragma unroll
        for (int e = 0; e < 16; ++e) acc[c][e] = 0.f;
    for (int64_t it = 0; it < iters; ++it) {
#pragma unroll
        for (int c = 0; c < kChains; ++c) acc[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[c], 0, 0, 0);
    }
    float sum = 0.f;
#pragma unroll
    for (int c = 0; c < kChains; ++c)
#pragma unroll
        for (int e = 0; e < 16; ++e) sum += acc[c][e];
    // one value per wave keeps the loop live; the buffer holds gridDim.x * kWavesPerBlock floats
    if (lane == 0) out[(int64_t)blockIdx.x * kWavesPerBlock + (threadIdx.x >> 6)] = sum;
}

}  // namespace

extern "C" int realq_mfma_peak(realq_ctx* ctx, int64_t iters, double* tflops) {
    if (!ctx) return REALQ_ERR_INVALID_ARG;
    if (iters < 1 || iters > (int64_t(1) << 24) || !tflops)
        return realq::set_error(ctx, REALQ_ERR_INVALID_ARG, "mfma_peak: need 1 <= iters <= 2^24 and tflops");
    const int64_t blocks = (int64_t)ctx->cus * 4;   // four rounds of one block per CU
    void* out = nullptr;
    int rc = realq::get_ws(ctx, "probe_out", (size_t)blocks * kWavesPerBlock * 4, &out);
    if (rc) return rc;
    realq::EventPair ev;
    RQ_HIP(ctx, ev.create());
    // one short launch first (clocks ramp up, code object loaded)
    hipLaunchKernelGGL(mfma_peak_kernel, dim3((unsigned)blocks), dim3(64 * kWavesPerBlock), 0, ctx->stream,
                       iters / 8 + 1, (float*)out);
    RQ_LAUNCHED(ctx);
    RQ_HIP(ctx, hipEventRecord(ev.a, ctx->stream));
    hipLaunchKernelGGL(mfma_peak_kernel, dim3((unsigned)blocks), dim3(64 * kWavesPerBlock), 0, ctx->stream, iters,
                       (float*)out);
    RQ_LAUNCHED(ctx);
    RQ_HIP(ctx, hipEventRecord(ev.b, ctx->stream));
    RQ_HIP(ctx, hipEventSynchronize(ev.b));
    float ms = 0.f;
    RQ_HIP(ctx, hipEventElapsedTime(&ms, ev.a, ev.b));
    const double flops = (double)blocks * kWavesPerBlock * (double)iters * kChains * (2.0 * 32 * 32 * 16);
    *tflops = flops / ((double)ms * 1e-3) / 1e12;
    return REALQ_OK;
}
