/*
 * Standalone use of the C ABI from C (no Python, no PyTorch): build an
 * IsoQuant-Full quantizer (d = 128, 3 bits, seeded rotations, Lloyd-Max
 * codebook), run isoq_quantize, isoq_dequantize and isoq_roundtrip on
 * 100,003 fp32 rows in device memory on a stream of its own, and check that
 * the fused path equals quantize followed by dequantize bit for bit, that a
 * zero row comes back as zero, that every other row's relative error lies
 * in the range a 3-bit Lloyd-Max quantizer produces, and that a bad argument
 * is refused before any launch.  Prints "abi_roundtrip ok" and exits 0 on
 * success.
 */
#include <hip/hip_runtime_api.h>
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "isoquant.h"

#define CHECK_HIP(call)                                                         \
    do {                                                                        \
        hipError_t e_ = (call);                                                 \
        if (e_ != hipSuccess) {                                                 \
            fprintf(stderr, "%s: %s\n", #call, hipGetErrorString(e_));          \
            return 1;                                                           \
        }                                                                       \
    } while (0)

#define CHECK_ISOQ(call)                                                        \
    do {                                                                        \
        isoq_status s_ = (call);                                                \
        if (s_ != ISOQ_OK) {                                                    \
            fprintf(stderr, "%s: %s (%s)\n", #call, isoq_status_string(s_),     \
                    isoq_last_hip_error());                                     \
            return 1;                                                           \
        }                                                                       \
    } while (0)

/* xorshift64* and Box-Muller: test input only */
static uint64_t rng_state = 0x9E3779B97F4A7C15ull;
static double uniform01(void)
{
    rng_state ^= rng_state >> 12;
    rng_state ^= rng_state << 25;
    rng_state ^= rng_state >> 27;
    return ((rng_state * 0x2545F4914F6CDD1Dull) >> 11) * (1.0 / 9007199254740992.0);
}
static double normal(void)
{
    double u = uniform01(), v = uniform01();
    if (u < 1e-300)
        u = 1e-300;
    return sqrt(-2.0 * log(u)) * cos(6.283185307179586 * v);
}

int main(void)
{
    const int d = 128, bits = 3;
    const int64_t n = 100003;
    const size_t rb = isoq_packed_bytes(d, bits);
    float *x = (float *)malloc(sizeof(float) * n * d);
    float *y1 = (float *)malloc(sizeof(float) * n * d);
    float *y2 = (float *)malloc(sizeof(float) * n * d);
    if (!x || !y1 || !y2)
        return 1;
    for (int64_t r = 0; r < n; r++) {
        double s = 0;
        for (int j = 0; j < d; j++) {
            const double v = normal();
            x[r * d + j] = (float)v;
            s += v * v;
        }
        for (int j = 0; j < d; j++)
            x[r * d + j] = (float)(x[r * d + j] / sqrt(s));
    }
    memset(x, 0, sizeof(float) * d); /* row 0 is zero */

    isoq_params *p = NULL;
    CHECK_ISOQ(isoq_params_init(&p, ISOQ_FULL, d, bits, 1, NULL, NULL, 1));

    hipStream_t stream;
    CHECK_HIP(hipStreamCreate(&stream));
    void *dx, *dy1, *dy2, *didx, *drho;
    CHECK_HIP(hipMalloc(&dx, sizeof(float) * n * d));
    CHECK_HIP(hipMalloc(&dy1, sizeof(float) * n * d));
    CHECK_HIP(hipMalloc(&dy2, sizeof(float) * n * d));
    CHECK_HIP(hipMalloc(&didx, rb * n));
    CHECK_HIP(hipMalloc(&drho, sizeof(float) * n));
    CHECK_HIP(hipMemcpyAsync(dx, x, sizeof(float) * n * d, hipMemcpyHostToDevice, stream));

    CHECK_ISOQ(isoq_quantize(p, ISOQ_F32, dx, n, 1, (uint8_t *)didx, (float *)drho, stream));
    CHECK_ISOQ(isoq_dequantize(p, ISOQ_F32, (const uint8_t *)didx, (const float *)drho, n, 1, dy1, stream));
    CHECK_ISOQ(isoq_roundtrip(p, ISOQ_F32, dx, n, 1, dy2, stream));
    CHECK_HIP(hipMemcpyAsync(y1, dy1, sizeof(float) * n * d, hipMemcpyDeviceToHost, stream));
    CHECK_HIP(hipMemcpyAsync(y2, dy2, sizeof(float) * n * d, hipMemcpyDeviceToHost, stream));
    CHECK_HIP(hipStreamSynchronize(stream));

    if (memcmp(y1, y2, sizeof(float) * n * d) != 0) {
        fprintf(stderr, "fused round trip differs from quantize + dequantize\n");
        return 1;
    }
    for (int j = 0; j < d; j++)
        if (y2[j] != 0.0f) {
            fprintf(stderr, "zero row not reconstructed as zero\n");
            return 1;
        }
    /* per-row squared error of a unit vector: about 0.034 on average at 3
     * bits (d times the per-coordinate MSE); every row well below 0.2 */
    double mean = 0, worst = 0;
    for (int64_t r = 1; r < n; r++) {
        double e = 0;
        for (int j = 0; j < d; j++) {
            const double t = (double)x[r * d + j] - (double)y2[r * d + j];
            e += t * t;
        }
        mean += e;
        if (e > worst)
            worst = e;
    }
    mean /= (double)(n - 1);
    if (!(mean > 0.025 && mean < 0.045) || !(worst < 0.2)) {
        fprintf(stderr, "unexpected error: mean %.5f worst %.5f\n", mean, worst);
        return 1;
    }
    /* a misaligned row pointer is refused before any launch */
    if (isoq_roundtrip(p, ISOQ_F32, (const char *)dx + 4, 4, 1, dy2, stream) != ISOQ_E_ALIGN) {
        fprintf(stderr, "misaligned input was not refused\n");
        return 1;
    }

    CHECK_HIP(hipFree(dx));
    CHECK_HIP(hipFree(dy1));
    CHECK_HIP(hipFree(dy2));
    CHECK_HIP(hipFree(didx));
    CHECK_HIP(hipFree(drho));
    CHECK_HIP(hipStreamDestroy(stream));
    CHECK_ISOQ(isoq_params_destroy(p));
    free(x);
    free(y1);
    free(y2);
    printf("abi_roundtrip ok: mean squared error per row %.5f\n", mean);
    return 0;
}
