/*
 * rg_negctl.h -- negative controls for the reproducibility tests (librg_negctl.so).
 *
 * NOT the method.  Two linear layers y = x * up(W)^T (same layouts as rg_linear:
 * x float32 [M][K], W bfloat16 bits [N][K], y float32 [M][N], all row-major,
 * device pointers, caller-owned) that each break one of the paper's design
 * rules, so that the tests can show the checks detect what the method removes
 * (paper: Supplement C, the R2 and R3 ablations; Design, rules R2 and R3).
 * Nothing in librg.so calls them.
 *
 * Errors: RG_NEGCTL_ERR_INVAL for a NULL pointer, M/N/K < 1, a size product that
 * overflows, x or y not 4-byte aligned, W not 2-byte aligned, more than
 * 16777215 * 256 outputs, or a bad split count; RG_NEGCTL_ERR_HIP when a HIP
 * call fails (rg_negctl_last_hip_error gives its code).  Nothing is enqueued on
 * error.  Calls are asynchronous and stream ordered; nothing is allocated.
 */
#ifndef RG_NEGCTL_H
#define RG_NEGCTL_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum { RG_NEGCTL_OK = 0, RG_NEGCTL_ERR_INVAL = 1, RG_NEGCTL_ERR_HIP = 4 };

/* Atomic split-K (breaks R3: the partials are combined in arrival order).
 * K is cut into `splits` contiguous ranges of ceil(K / splits) elements
 * (1 <= splits <= min(K, 65535)); each range's partial, one fmaf chain from +0,
 * is added into y with a float atomic add after y has been zeroed on the same
 * stream.  Repeated calls on the same inputs can return different bits. */
int rg_negctl_atomic_splitk(const float* x, const uint16_t* w_bf16, float* y, int64_t M, int64_t N, int64_t K,
                            int32_t splits, void* stream);

/* Machine-sized split (breaks R2: a configuration that depends on the device).
 * S = clamp(enabled CUs of `stream` / ceil(M*N / 256), 1, 64) (the null stream
 * counts every CU); K is cut into contiguous pieces of ceil(K / S) elements, each
 * summed by one fmaf chain from +0, and the pieces are added in ascending order.
 * Deterministic for one CU mask, but the bits change with the mask.  The split
 * actually used (the number of non-empty pieces) is written to *splits_out if
 * it is not NULL. */
int rg_negctl_cu_split(const float* x, const uint16_t* w_bf16, float* y, int64_t M, int64_t N, int64_t K,
                       void* stream, int32_t* splits_out);

/* hipError_t code of the last HIP call this thread made in this library. */
int rg_negctl_last_hip_error(void);

#ifdef __cplusplus
}
#endif

#endif /* RG_NEGCTL_H */
