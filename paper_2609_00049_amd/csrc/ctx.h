// Internal context of the REAL-Q library (not part of the C ABI): the stream, grow-only
// workspaces by slot name, and the optional per-kernel timing that realq_ctx_kernel_time reads.
#pragma once
#include <map>
#include <string>
#include <vector>

#include <rocprofiler-sdk-roctx/roctx.h>

#include "common.h"

struct realq_ctx {
    hipStream_t stream = nullptr;
    int device = 0;
    int cus = 256;  // compute units of the device (blocks of the 256x256 GEMM tile resident at once)
    std::string err;
    // grow-only workspaces, by slot name
    struct Buf {
        void* p = nullptr;
        size_t bytes = 0;
    };
    std::map<std::string, Buf> ws;
    // kernel timing
    bool timing = false;
    struct Stat {
        int64_t launches = 0;
        double ms = 0.0;
    };
    std::map<std::string, Stat> stats;
    struct Pending {
        std::string name;
        hipEvent_t a, b;
    };
    std::vector<Pending> pending;
    std::vector<std::pair<hipEvent_t, hipEvent_t>> free_events;
};

namespace realq {

// Device buffer of at least `bytes` for `slot` (grown by synchronising the stream and
// reallocating; contents are not kept across growth).
int get_ws(realq_ctx* ctx, const char* slot, size_t bytes, void** out);
// Folds finished timing events into ctx->stats (synchronises on the last one).
int harvest(realq_ctx* ctx);
}  // namespace realq

struct realq_qparams;
struct realq_bgd_params;

namespace realq {
// Argument checks shared by the entry points (REALQ_OK or an error set on ctx).
int validate_q(realq_ctx* ctx, const realq_qparams* qp);
int validate_bgd(realq_ctx* ctx, const realq_bgd_params* p);
// Token-chunked Hessian accumulation into H_acc with caller-provided staging buffers (n * tc bf16
// each; hi, lo, lo2 only used when s is given).
int hessian_accum_chunks(realq_ctx* ctx, const uint16_t* Xhat, const float* s, int64_t T, int64_t n, double* H_acc,
                         int64_t tc, uint16_t* xt, uint16_t* hi, uint16_t* lo, uint16_t* lo2, bool timed);

// A roctx range over a host scope: the launches it encloses show under its name in a
// `rocprofv3 --marker-trace` run (the push is a no-op call when no tool is attached).
struct Range {
    explicit Range(const char* n) { roctxRangePushA(n); }
    ~Range() { roctxRangePop(); }
    Range(const Range&) = delete;
    Range& operator=(const Range&) = delete;
};

// Brackets the launches of its scope with events on the context stream when timing is on, and
// with a roctx range of the same name.
struct Timed {
    realq_ctx* ctx;
    const char* name;
    hipEvent_t a = nullptr, b = nullptr;
    Range range;
    Timed(realq_ctx* c, const char* n) : ctx(c), name(n), range(n ? n : "realq") {
        if (!ctx->timing || !n) return;
        if (!ctx->free_events.empty()) {
            a = ctx->free_events.back().first;
            b = ctx->free_events.back().second;
            ctx->free_events.pop_back();
        } else {
            if (hipEventCreate(&a) != hipSuccess || hipEventCreate(&b) != hipSuccess) {
                a = b = nullptr;
                return;
            }
        }
        (void)hipEventRecord(a, ctx->stream);
    }
    ~Timed() {
        if (!a) return;
        (void)hipEventRecord(b, ctx->stream);
        ctx->pending.push_back({name, a, b});
    }
};

// Start/end events of a whole entry point, destroyed on every return path.
struct EventPair {
    hipEvent_t a = nullptr, b = nullptr;
    EventPair() = default;
    EventPair(const EventPair&) = delete;
    EventPair& operator=(const EventPair&) = delete;
    hipError_t create() {
        hipError_t e = hipEventCreate(&a);
        return e != hipSuccess ? e : hipEventCreate(&b);
    }
    ~EventPair() {
        if (a) (void)hipEventDestroy(a);
        if (b) (void)hipEventDestroy(b);
    }
};

}  // namespace realq
