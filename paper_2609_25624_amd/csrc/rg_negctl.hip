// Negative controls: two linear-layer kernels that break the design rules on
// purpose, so the tests can show that the reproducibility checks catch what
// the method removes (paper: Supplement C, the R2 and R3 ablations).  NOT the
// method and never called by rg_linear; built into a library of its own.
//
//  * atomic split-K (breaks R3): K is cut into `splits` ranges, each range's
//    partial is added into y with a floating-point atomic, so the order of the
//    additions is whatever order the workgroups reach memory in.
//  * machine-sized split (breaks R2/R3): the split factor is derived from the
//    number of compute units the stream may use, as an autotuner sizing split-K
//    to fill the device would; the summation order then depends on the CU mask.
//    The arithmetic of that split (contiguous pieces of ceil(K/S) elements, each
//    one fmaf chain from +0, the pieces added in ascending order) is carried out
//    inside one thread per output, which changes nothing in the bits it yields.
//
// Both use the exact BF16 upcast and binary32 fmaf like the library proper.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/rg_negctl.h"

namespace {

__device__ __forceinline__ float up1(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

__global__ void __launch_bounds__(256) zero_kernel(float* __restrict__ y, int64_t count) {
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < count; i += stride) y[i] = 0.0f;
}

// blockIdx.y = split s; thread = output (m, n).  Range s covers K elements
// [s*L, min(s*L + L, K)), summed by one fmaf chain, then added into y atomically.
__global__ void __launch_bounds__(256) atomic_splitk_kernel(const float* __restrict__ x, const uint16_t* __restrict__ w,
                                                           float* y, int64_t M, int64_t N, int64_t K, int64_t L) {
    const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= M * N) return;
    const int64_t m = idx / N, n = idx % N;
    const int64_t k0 = (int64_t)blockIdx.y * L;
    const int64_t k1 = (k0 + L < K) ? k0 + L : K;
    const float* xr = x + m * K;
    const uint16_t* wr = w + n * K;
    float p = 0.0f;
    for (int64_t k = k0; k < k1; ++k) p = __builtin_fmaf(xr[k], up1(wr[k]), p);
    atomicAdd(y + idx, p);
}

__global__ void __launch_bounds__(256) piece_split_kernel(const float* __restrict__ x, const uint16_t* __restrict__ w,
                                                         float* __restrict__ y, int64_t M, int64_t N, int64_t K,
                                                         int64_t L) {
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; idx < M * N; idx += stride) {
        const int64_t m = idx / N, n = idx % N;
        const float* xr = x + m * K;
        const uint16_t* wr = w + n * K;
        float acc = 0.0f;
        for (int64_t k0 = 0; k0 < K; k0 += L) {
            const int64_t k1 = (k0 + L < K) ? k0 + L : K;
            float p = 0.0f;
            for (int64_t k = k0; k < k1; ++k) p = __builtin_fmaf(xr[k], up1(wr[k]), p);
            acc = (k0 == 0) ? p : acc + p;
        }
        y[idx] = acc;
    }
}

thread_local int t_last_hip = 0;

int status_of(hipError_t e) {
    t_last_hip = (int)e;
    return e == hipSuccess ? RG_NEGCTL_OK : RG_NEGCTL_ERR_HIP;
}

// Grid limit of the one-output-per-thread launches (gridDim.x * 256 stays below 2^32).
constexpr int64_t kMaxBlocks = 16777215;

bool mul_ok(int64_t a, int64_t b) { return a <= 0 || b <= INT64_MAX / 4 / a; }

int check_args(const float* x, const uint16_t* w, const float* y, int64_t M, int64_t N, int64_t K) {
    if (!x || !w || !y || M < 1 || N < 1 || K < 1) return RG_NEGCTL_ERR_INVAL;
    if (!mul_ok(M, K) || !mul_ok(N, K) || !mul_ok(M, N)) return RG_NEGCTL_ERR_INVAL;
    if (((uintptr_t)x & 3) || ((uintptr_t)w & 1) || ((uintptr_t)y & 3)) return RG_NEGCTL_ERR_INVAL;
    if ((M * N + 255) / 256 > kMaxBlocks) return RG_NEGCTL_ERR_INVAL;
    return RG_NEGCTL_OK;
}

int device_cus(int* cus) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e == hipSuccess) e = hipDeviceGetAttribute(cus, hipDeviceAttributeMultiprocessorCount, dev);
    return status_of(e);
}

}  // namespace

extern "C" {

int rg_negctl_atomic_splitk(const float* x, const uint16_t* w, float* y, int64_t M, int64_t N, int64_t K,
                            int32_t splits, void* stream) {
    const int c = check_args(x, w, y, M, N, K);
    if (c != RG_NEGCTL_OK) return c;
    if (splits < 1 || splits > 65535 || splits > K) return RG_NEGCTL_ERR_INVAL;
    const int64_t L = (K + splits - 1) / splits;
    const int64_t blocks = (M * N + 255) / 256;
    hipStream_t st = (hipStream_t)stream;
    (void)hipGetLastError();
    const int64_t zb = blocks < 4096 ? blocks : 4096;
    hipLaunchKernelGGL(zero_kernel, dim3((unsigned)zb), dim3(256), 0, st, y, M * N);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return status_of(e);
    // Only splits that hold at least one element are launched (ceil rounding can leave the last empty).
    const int64_t used = (K + L - 1) / L;
    hipLaunchKernelGGL(atomic_splitk_kernel, dim3((unsigned)blocks, (unsigned)used), dim3(256), 0, st, x, w, y, M, N,
                       K, L);
    return status_of(hipGetLastError());
}

int rg_negctl_cu_split(const float* x, const uint16_t* w, float* y, int64_t M, int64_t N, int64_t K, void* stream,
                       int32_t* splits_out) {
    const int c = check_args(x, w, y, M, N, K);
    if (c != RG_NEGCTL_OK) return c;
    hipStream_t st = (hipStream_t)stream;
    int cus = 0;
    int d = device_cus(&cus);
    if (d != RG_NEGCTL_OK) return d;
    if (st) {   // a created stream may carry a CU mask; the null stream uses every CU
        uint32_t mask[32] = {0};
        const uint32_t words = (uint32_t)((cus + 31) / 32);
        if (words > 32) return RG_NEGCTL_ERR_INVAL;
        hipError_t e = hipExtStreamGetCUMask(st, words, mask);
        if (e != hipSuccess) return status_of(e);
        cus = 0;
        for (uint32_t i = 0; i < words; ++i) cus += __builtin_popcount(mask[i]);
    }
    // The split that gives every enabled CU one workgroup of 256 outputs.
    const int64_t tiles = (M * N + 255) / 256;
    int64_t S = cus / tiles;
    if (S < 1) S = 1;
    if (S > 64) S = 64;
    if (S > K) S = K;
    const int64_t L = (K + S - 1) / S;
    if (splits_out) *splits_out = (int32_t)((K + L - 1) / L);
    const int64_t blocks = tiles < 65536 ? tiles : 65536;
    (void)hipGetLastError();
    hipLaunchKernelGGL(piece_split_kernel, dim3((unsigned)blocks), dim3(256), 0, st, x, w, y, M, N, K, L);
    return status_of(hipGetLastError());
}

int rg_negctl_last_hip_error(void) { return t_last_hip; }

}  // extern "C"
