// Internal interface of the wave-tile kernel (rg_wtile.hip) for the C-ABI (rg_api.cpp).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace rg {

constexpr int kWtileRows = 64;   // output tile: 64 rows of x by 64 rows of W
constexpr int kWtileK = 8;       // k per staged slab

// LDS bytes of one workgroup of `waves` waves (each wave its own double-buffered x and W
// slabs; one 64 x 64 tile of running totals).
constexpr int wtile_lds_bytes(int waves) {
    return waves * 2 * 2 * kWtileK * (kWtileRows + 4) * 4 + kWtileRows * kWtileRows * 4;
}

// waves: 4 (the planner's choice) or 8 (forced launches).  x [M][K] FP32, w [N][K] BF16 bits or FP32, y [M][N]; K % 8 == 0 (BF16)
// or K % 4 == 0 (FP32), x and w 16-byte aligned.  Grid: ceil(M / 64) * ceil(N / 64) workgroups.
hipError_t launch_wtile(const float* x, const uint16_t* w, const float* bias, float* y, int64_t M, int64_t N,
                        int64_t K, int waves, int reverse, hipStream_t stream);
hipError_t launch_wtile(const float* x, const float* w, const float* bias, float* y, int64_t M, int64_t N,
                        int64_t K, int waves, int reverse, hipStream_t stream);

}  // namespace rg
