/*
 * rg_baseline.h -- the comparison point of librg: the scheme the fused layer
 * replaces (Design, eq. 1).  librg_baseline.so, a library of its own so that
 * librg.so keeps no BLAS dependency.
 *
 * W is first widened into a transient FP32 copy (w_tmp_f32, 4NK bytes, owned
 * by the caller), then y = x * w_tmp^T by the vendor FP32 GEMM (rocBLAS sgemm,
 * or sgemv for M = 1; a black box: its reduction order is the library's and may depend on the
 * device, the shape and the batch size, which is what the method removes).
 * It exists to time the scheme on the same buffers and stream as rg_linear;
 * it is never used by rg_linear.
 *
 *   x        float32 [M][K]  device, row-major
 *   w_bf16   bfloat16 bits [N][K] device, row-major
 *   w_tmp_f32 float32 [N][K] device scratch, overwritten (the transient copy)
 *   y        float32 [M][N] device, overwritten
 *   1 <= M, N, K <= 2^31 - 1 with N * K and M * N below 2^62; 4-byte alignment.
 *   stream: the HIP stream both steps are enqueued on (asynchronous).
 * The first call on a device creates that device's rocBLAS handle (which
 * allocates the library's own workspace); later calls allocate nothing.
 * Returns the rg_status codes of include/rg.h: RG_ERR_INVAL for bad sizes or
 * null pointers, RG_ERR_ALIGN, RG_ERR_ALIAS when w_tmp_f32 or y overlaps an
 * input or each other, RG_ERR_HIP when the cast, the handle or the GEMM fails.
 */
#ifndef RG_BASELINE_H
#define RG_BASELINE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

int rg_linear_cast_baseline(const float* x, const uint16_t* w_bf16, float* w_tmp_f32, float* y, int64_t M,
                            int64_t N, int64_t K, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* RG_BASELINE_H */
