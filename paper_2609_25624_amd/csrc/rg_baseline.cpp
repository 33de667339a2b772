// The comparison point (Design, eq. 1): widen W into a caller-owned FP32 copy
// with librg's exact cast kernel, then the vendor FP32 GEMM (rocBLAS sgemm).
// See include/rg_baseline.h.

#include <hip/hip_runtime.h>
#include <rocblas/rocblas.h>

#include <cstdint>
#include <mutex>

#include "../../include/rg.h"
#include "../../include/rg_baseline.h"

namespace {

constexpr int kMaxDevices = 64;

struct Handle {
    std::once_flag once;
    rocblas_handle h = nullptr;
    bool ok = false;
};
Handle g_handles[kMaxDevices];

bool overlaps(const void* a, size_t an, const void* b, size_t bn) {
    const uintptr_t a0 = (uintptr_t)a, b0 = (uintptr_t)b;
    return a0 < b0 + bn && b0 < a0 + an;
}

}  // namespace

extern "C" int rg_linear_cast_baseline(const float* x, const uint16_t* w, float* wt, float* y, int64_t M, int64_t N,
                                       int64_t K, void* stream) {
    if (!x || !w || !wt || !y || M < 1 || N < 1 || K < 1) return RG_ERR_INVAL;
    const int64_t lim = 0x7fffffff;
    if (M > lim || N > lim || K > lim || N > ((int64_t)1 << 62) / K || M > ((int64_t)1 << 62) / N ||
        M > ((int64_t)1 << 62) / K)
        return RG_ERR_INVAL;
    if (((uintptr_t)x & 3) || ((uintptr_t)w & 1) || ((uintptr_t)wt & 3) || ((uintptr_t)y & 3)) return RG_ERR_ALIGN;
    const size_t xb = (size_t)(M * K) * 4, wb = (size_t)(N * K) * 2, tb = (size_t)(N * K) * 4, yb = (size_t)(M * N) * 4;
    if (overlaps(wt, tb, x, xb) || overlaps(wt, tb, w, wb) || overlaps(wt, tb, y, yb) || overlaps(y, yb, x, xb) ||
        overlaps(y, yb, w, wb))
        return RG_ERR_ALIAS;
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return RG_ERR_HIP;
    Handle& hd = g_handles[dev];
    std::call_once(hd.once, [&] { hd.ok = rocblas_create_handle(&hd.h) == rocblas_status_success; });
    if (!hd.ok) return RG_ERR_HIP;
    const int cs = rg_cast_bf16_f32(w, wt, N * K, stream);
    if (cs != RG_OK) return cs;
    if (rocblas_set_stream(hd.h, (hipStream_t)stream) != rocblas_status_success) return RG_ERR_HIP;
    const float one = 1.0f, zero = 0.0f;
    rocblas_status st;
    if (M == 1) {
        // one row of x: the vendor's matrix-vector product, y = (w_tmp viewed K x N column-major)^T x
        st = rocblas_sgemv(hd.h, rocblas_operation_transpose, (rocblas_int)K, (rocblas_int)N, &one, wt, (rocblas_int)K,
                           x, 1, &zero, y, 1);
    } else {
        // column-major view: y^T [N x M] = (w_tmp [N x K]) * (x^T [K x M]); w_tmp row-major is K x N column-major
        st = rocblas_sgemm(hd.h, rocblas_operation_transpose, rocblas_operation_none, (rocblas_int)N, (rocblas_int)M,
                           (rocblas_int)K, &one, wt, (rocblas_int)K, x, (rocblas_int)K, &zero, y, (rocblas_int)N);
    }
    return st == rocblas_status_success ? RG_OK : RG_ERR_HIP;
}
