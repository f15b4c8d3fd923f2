// realq_hessian_accum_noalloc: the Hessian accumulation of realq_hessian_accum with its token
// chunks staged in a fixed device array instead of context workspaces, for callers that cannot
// allocate device memory.  The array is file-scope device memory, one copy per GPU, held until the
// process ends; host code reaches it only through the address hipGetSymbolAddress returns for the
// current device (the array's own name is a host-side stand-in, not a device address).
#include <mutex>
#include <string>

#include "common.h"
#include "ctx.h"
#include "kernels.h"
#include "../../include/realq.h"

namespace {

static_assert(REALQ_NOALLOC_SCRATCH_BYTES % 4 == 0, "scratch splits into four staging buffers");
constexpr int64_t kStage = REALQ_NOALLOC_SCRATCH_BYTES / 4;  // bytes per staging buffer

// Staging for one token chunk: the transposed chunk and the three bf16 terms of s_t xhat_t.
static __device__ __align__(256) unsigned char scratch[REALQ_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_ptr[kMaxDevices] = {};
bool g_tried[kMaxDevices] = {};
hipError_t g_err[kMaxDevices] = {};

// Device address of this GPU's copy of `scratch`, looked up once per device with that device
// current (the first call on the device).
hipError_t scratch_of(int device, void** out) {
    std::lock_guard<std::mutex> lk(g_mu);
    if (!g_tried[device]) {
        g_tried[device] = true;
        void* p = nullptr;
        g_err[device] = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        g_ptr[device] = g_err[device] == hipSuccess ? p : nullptr;
        if (g_err[device] != hipSuccess) (void)hipGetLastError();
    }
    *out = g_ptr[device];
    return g_err[device];
}

}  // namespace

extern "C" int realq_hessian_accum_noalloc(realq_ctx* ctx, const uint16_t* Xhat, const float* s, int64_t T,
                                           int64_t n, double* H_acc) {
    if (!ctx) return REALQ_ERR_INVALID_ARG;
    if (T < 0 || n <= 0) return realq::set_error(ctx, REALQ_ERR_SHAPE, "hessian_accum_noalloc: need T >= 0, n > 0");
    if (n > REALQ_NOALLOC_MAX_N)
        return realq::set_error(ctx, REALQ_ERR_SHAPE,
                                "hessian_accum_noalloc: n = " + std::to_string(n) + " exceeds the scratch limit of " +
                                    std::to_string(REALQ_NOALLOC_MAX_N) + " input columns");
    if (T == 0) return REALQ_OK;
    if (!Xhat || !H_acc) return realq::set_error(ctx, REALQ_ERR_INVALID_ARG, "hessian_accum_noalloc: NULL Xhat or H_acc");
    int device = -1;
    RQ_HIP(ctx, hipGetDevice(&device));
    if (device < 0 || device >= kMaxDevices)
        return realq::set_error(ctx, REALQ_ERR_HIP, "hessian_accum_noalloc: device index out of range");
    void* base = nullptr;
    hipError_t e = scratch_of(device, &base);
    if (e != hipSuccess || !base)
        return realq::set_error(ctx, REALQ_ERR_HIP,
                                std::string("hessian_accum_noalloc: scratch address: ") + hipGetErrorString(e));
    // tokens per chunk: a multiple of 256 whose n x tc bf16 chunk fits one staging buffer
    // (n <= REALQ_NOALLOC_MAX_N keeps tc >= 256); a short input takes one chunk
    int64_t tc = (kStage / (2 * n)) / 256 * 256;
    if (tc > T) tc = ((T + 7) / 8) * 8;
    unsigned char* b = static_cast<unsigned char*>(base);
    uint16_t* xt = reinterpret_cast<uint16_t*>(b);
    uint16_t* hi = reinterpret_cast<uint16_t*>(b + kStage);
    uint16_t* lo = reinterpret_cast<uint16_t*>(b + 2 * kStage);
    uint16_t* lo2 = reinterpret_cast<uint16_t*>(b + 3 * kStage);
    // every staged element the GEMMs read is written by the transposes of the same chunk, so
    // nothing left in the array by an earlier call needs clearing
    return realq::hessian_accum_chunks(ctx, Xhat, s, T, n, H_acc, tc, xt, hi, lo, lo2, false);
}
