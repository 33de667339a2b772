/*
 * Using librg from C through include/rg.h alone: device buffers from the HIP
 * runtime, one rg_linear call per shape, results checked on the host.
 *
 * The inputs are small integers (x in [-3, 3], W in [-2, 2], both exact in
 * bfloat16 and float32), so every partial sum is an exact integer and the
 * product has one correct value whatever the order; the host compares each
 * output with the integer dot product.  It also checks that rg_plan reports
 * the documented order and that a bad argument is rejected before any work.
 *
 * Build (done by the package build step):
 *   hipcc -x c ... linear_capi.c -L<package> -lrg -o linear_capi
 * Run: ./linear_capi   (exit status 0 when every check passes)
 */
#include <hip/hip_runtime_api.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "../../include/rg.h"

static uint16_t bf16_of_small_int(int v) {   /* exact: |v| <= 3 */
    float f = (float)v;
    uint32_t u;
    memcpy(&u, &f, 4);
    return (uint16_t)(u >> 16);
}

static int check_shape(int64_t M, int64_t N, int64_t K) {
    const size_t nx = (size_t)(M * K), nw = (size_t)(N * K), ny = (size_t)(M * N);
    float* hx = (float*)malloc(nx * sizeof(float));
    uint16_t* hw = (uint16_t*)malloc(nw * sizeof(uint16_t));
    float* hy = (float*)malloc(ny * sizeof(float));
    int* xi = (int*)malloc(nx * sizeof(int));
    int* wi = (int*)malloc(nw * sizeof(int));
    for (int64_t m = 0; m < M; ++m)
        for (int64_t k = 0; k < K; ++k) {
            xi[m * K + k] = (int)((3 * m + k) % 7) - 3;
            hx[m * K + k] = (float)xi[m * K + k];
        }
    for (int64_t n = 0; n < N; ++n)
        for (int64_t k = 0; k < K; ++k) {
            wi[n * K + k] = (int)((n + 2 * k) % 5) - 2;
            hw[n * K + k] = bf16_of_small_int(wi[n * K + k]);
        }
    float *dx = NULL, *dy = NULL;
    uint16_t* dw = NULL;
    if (hipMalloc((void**)&dx, nx * sizeof(float)) != hipSuccess ||
        hipMalloc((void**)&dw, nw * sizeof(uint16_t)) != hipSuccess ||
        hipMalloc((void**)&dy, ny * sizeof(float)) != hipSuccess) {
        fprintf(stderr, "hipMalloc failed\n");
        return 1;
    }
    hipMemcpy(dx, hx, nx * sizeof(float), hipMemcpyHostToDevice);
    hipMemcpy(dw, hw, nw * sizeof(uint16_t), hipMemcpyHostToDevice);
    int rc = rg_linear(dx, dw, dy, M, N, K, NULL);
    if (rc != RG_OK) {
        fprintf(stderr, "rg_linear(%lld,%lld,%lld): %s\n", (long long)M, (long long)N, (long long)K, rg_strerror(rc));
        return 1;
    }
    if (hipDeviceSynchronize() != hipSuccess) {
        fprintf(stderr, "hipDeviceSynchronize failed\n");
        return 1;
    }
    hipMemcpy(hy, dy, ny * sizeof(float), hipMemcpyDeviceToHost);
    int64_t bad = 0;
    for (int64_t m = 0; m < M; ++m)
        for (int64_t n = 0; n < N; ++n) {
            long long s = 0;
            for (int64_t k = 0; k < K; ++k) s += (long long)xi[m * K + k] * wi[n * K + k];
            if (hy[m * N + n] != (float)s) ++bad;
        }
    rg_plan_t p;
    rg_plan(M, N, K, &p);
    printf("rg_linear %lldx%lldx%lld kernel %d: %lld of %lld outputs wrong\n", (long long)M, (long long)N,
           (long long)K, p.kernel, (long long)bad, (long long)ny);
    hipFree(dx);
    hipFree(dw);
    hipFree(dy);
    free(hx); free(hw); free(hy); free(xi); free(wi);
    return bad != 0;
}

int main(void) {
    rg_plan_t p;
    if (rg_plan(3, 100, 1000, &p) != RG_OK || p.order_id != RG_ORDER_ID || p.chunk != RG_CHUNK || p.nchunks != 4) {
        fprintf(stderr, "rg_plan does not report the documented order\n");
        return 1;
    }
    if (rg_linear(NULL, NULL, NULL, 1, 1, 1, NULL) != RG_ERR_INVAL) {
        fprintf(stderr, "a NULL argument was not rejected\n");
        return 1;
    }
    int fails = 0;
    const int64_t shapes[][3] = {{1, 4096, 4096}, {1, 1030, 4352}, {3, 300, 1000}, {16, 515, 2048}, {70, 130, 264}};
    for (size_t i = 0; i < sizeof shapes / sizeof shapes[0]; ++i)
        fails += check_shape(shapes[i][0], shapes[i][1], shapes[i][2]);
    printf(fails ? "FAILED\n" : "all checks passed\n");
    return fails != 0;
}
