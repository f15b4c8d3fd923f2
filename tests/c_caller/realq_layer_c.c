/* A plain C caller of librealq.so: device memory and the stream from the HIP runtime's C API,
 * one realq_quantize_layer call (the per-module sweep of Alg. 1), results written to a file.
 * Shows that the library's C ABI stands on its own, without PyTorch.
 *
 * usage: realq_layer_c IN OUT
 *   IN : int64 m, n, T, steps; float lr; float W0[m n]; uint16 X[T n], Xhat[T n] (bf16 bits);
 *        float s[T]
 *   OUT: uint8 codes[m n]; float scales[m g]; uint8 zeros[m g]; float W_hat[m n]; double loss_final
 *        (g = ceil(n / 128), the default group of 128 columns) */
#include <hip/hip_runtime_api.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

#include "realq.h"

#define HIP_OK(x)                                                                          \
    do {                                                                                   \
        hipError_t e_ = (x);                                                               \
        if (e_ != hipSuccess) {                                                            \
            fprintf(stderr, "%s:%d: %s\n", __FILE__, __LINE__, hipGetErrorString(e_));     \
            exit(2);                                                                       \
        }                                                                                  \
    } while (0)

static void* read_n(FILE* f, size_t bytes) {
    void* p = malloc(bytes ? bytes : 1);
    if (!p || fread(p, 1, bytes, f) != bytes) {
        fprintf(stderr, "short input\n");
        exit(2);
    }
    return p;
}

static void* to_device(const void* host, size_t bytes) {
    void* d = NULL;
    HIP_OK(hipMalloc(&d, bytes ? bytes : 1));
    if (bytes) HIP_OK(hipMemcpy(d, host, bytes, hipMemcpyHostToDevice));
    return d;
}

int main(int argc, char** argv) {
    if (argc != 3) {
        fprintf(stderr, "usage: %s IN OUT\n", argv[0]);
        return 2;
    }
    FILE* f = fopen(argv[1], "rb");
    if (!f) {
        perror(argv[1]);
        return 2;
    }
    int64_t dims[4];
    float lr;
    if (fread(dims, sizeof(int64_t), 4, f) != 4 || fread(&lr, sizeof(float), 1, f) != 1) {
        fprintf(stderr, "short header\n");
        return 2;
    }
    const int64_t m = dims[0], n = dims[1], T = dims[2];
    const int32_t steps = (int32_t)dims[3];
    if (m < 1 || n < 1 || T < 1 || m > (1 << 20) || n > (1 << 20) || T > (1 << 24)) {
        fprintf(stderr, "bad sizes\n");
        return 2;
    }
    const int64_t g = (n + 127) / 128;
    float* W0 = (float*)read_n(f, (size_t)(m * n) * 4);
    uint16_t* X = (uint16_t*)read_n(f, (size_t)(T * n) * 2);
    uint16_t* Xh = (uint16_t*)read_n(f, (size_t)(T * n) * 2);
    float* s = (float*)read_n(f, (size_t)T * 4);
    fclose(f);

    hipStream_t stream;
    HIP_OK(hipStreamCreate(&stream));
    realq_ctx* ctx = NULL;
    if (realq_ctx_create(&ctx, (void*)stream) != REALQ_OK) {
        fprintf(stderr, "realq_ctx_create failed\n");
        return 3;
    }
    realq_layer_desc d = {0};
    d.m = m;
    d.n = n;
    d.T = T;
    d.W0 = (const float*)to_device(W0, (size_t)(m * n) * 4);
    d.X = (const uint16_t*)to_device(X, (size_t)(T * n) * 2);
    d.Xhat = (const uint16_t*)to_device(Xh, (size_t)(T * n) * 2);
    d.s = (const float*)to_device(s, (size_t)T * 4);
    realq_qparams_default(&d.q);
    realq_bgd_params_default(&d.bgd);
    d.bgd.steps = steps;
    d.bgd.lr = lr;

    realq_layer_out o = {0};
    HIP_OK(hipMalloc((void**)&o.codes, (size_t)(m * n)));
    HIP_OK(hipMalloc((void**)&o.scales, (size_t)(m * g) * 4));
    HIP_OK(hipMalloc((void**)&o.zeros, (size_t)(m * g)));
    HIP_OK(hipMalloc((void**)&o.W_hat, (size_t)(m * n) * 4));
    const int rc = realq_quantize_layer(ctx, &d, &o);
    if (rc != REALQ_OK) {
        fprintf(stderr, "realq_quantize_layer: %d %s\n", rc, realq_last_error(ctx));
        return 3;
    }
    HIP_OK(hipStreamSynchronize(stream));

    uint8_t* codes = (uint8_t*)malloc((size_t)(m * n));
    float* scales = (float*)malloc((size_t)(m * g) * 4);
    uint8_t* zeros = (uint8_t*)malloc((size_t)(m * g));
    float* W_hat = (float*)malloc((size_t)(m * n) * 4);
    if (!codes || !scales || !zeros || !W_hat) return 2;
    HIP_OK(hipMemcpy(codes, o.codes, (size_t)(m * n), hipMemcpyDeviceToHost));
    HIP_OK(hipMemcpy(scales, o.scales, (size_t)(m * g) * 4, hipMemcpyDeviceToHost));
    HIP_OK(hipMemcpy(zeros, o.zeros, (size_t)(m * g), hipMemcpyDeviceToHost));
    HIP_OK(hipMemcpy(W_hat, o.W_hat, (size_t)(m * n) * 4, hipMemcpyDeviceToHost));
    FILE* out = fopen(argv[2], "wb");
    if (!out) {
        perror(argv[2]);
        return 2;
    }
    fwrite(codes, 1, (size_t)(m * n), out);
    fwrite(scales, 4, (size_t)(m * g), out);
    fwrite(zeros, 1, (size_t)(m * g), out);
    fwrite(W_hat, 4, (size_t)(m * n), out);
    fwrite(&o.loss_final, 8, 1, out);
    fclose(out);

    realq_ctx_destroy(ctx);
    HIP_OK(hipFree((void*)d.W0));
    HIP_OK(hipFree((void*)d.X));
    HIP_OK(hipFree((void*)d.Xhat));
    HIP_OK(hipFree((void*)d.s));
    HIP_OK(hipFree(o.codes));
    HIP_OK(hipFree(o.scales));
    HIP_OK(hipFree(o.zeros));
    HIP_OK(hipFree(o.W_hat));
    HIP_OK(hipStreamDestroy(stream));
    free(W0);
    free(X);
    free(Xh);
    free(s);
    free(codes);
    free(scales);
    free(zeros);
    free(W_hat);
    printf("realq_layer_c: m=%lld n=%lld T=%lld loss %.17g\n", (long long)m, (long long)n, (long long)T, o.loss_final);
    return 0;
}
