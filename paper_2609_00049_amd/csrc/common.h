// Shared helpers of the REAL-Q gfx950 library: bf16 storage, vector types,
// launch-check macros and the internal launcher declarations.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <string>

namespace realq {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef double f64x4 __attribute__((ext_vector_type(4)));
typedef uint16_t u16x8 __attribute__((ext_vector_type(8)));

// ---------------------------------------------------------------- bf16 storage
// Round to nearest, ties to even (finite inputs).
__device__ __forceinline__ uint16_t f2bf(float f) {
    uint32_t u = __float_as_uint(f);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}
__device__ __forceinline__ float bf2f(uint16_t b) { return __uint_as_float(((uint32_t)b) << 16); }

// hi + lo with hi = bf16(x), lo = bf16(x - hi): |x - hi - lo| <= 2^-16 |x| (roughly).
__device__ __forceinline__ void split_bf16(float x, uint16_t& hi, uint16_t& lo) {
    hi = f2bf(x);
    lo = f2bf(x - bf2f(hi));
}

__device__ __forceinline__ int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

}  // namespace realq

// ---------------------------------------------------------------- host-side error plumbing
struct realq_ctx;
namespace realq {
int set_error(realq_ctx* ctx, int code, const std::string& msg);
}

#define RQ_HIP(ctx, expr)                                                                  \
    do {                                                                                   \
        hipError_t _e = (expr);                                                            \
        if (_e != hipSuccess)                                                              \
            return realq::set_error((ctx), -4, std::string(#expr ": ") + hipGetErrorString(_e)); \
    } while (0)

#define RQ_LAUNCHED(ctx)                                                                   \
    do {                                                                                   \
        hipError_t _e = hipGetLastError();                                                 \
        if (_e != hipSuccess)                                                              \
            return realq::set_error((ctx), -4, std::string("kernel launch: ") + hipGetErrorString(_e)); \
    } while (0)
