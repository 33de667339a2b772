// Read-bandwidth probe (include/rg_probe.h): a kernel that reads and does nothing else.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/rg_probe.h"

namespace {

constexpr int kPiece = 8192;                 // bytes per wave piece: 8 loads of 1 KB per wave
constexpr int kLoads = kPiece / (64 * 16);   // 16-byte loads per lane per piece

// Wave v of W reads pieces v, v + W, v + 2W, ... two at a time (16 loads in flight per lane).
__global__ void __launch_bounds__(256) read_kernel(const uint4* __restrict__ src, int64_t pieces, uint32_t* sink) {
    const int lane = threadIdx.x & 63;
    const int64_t waves = (int64_t)gridDim.x * 4;
    const int64_t v = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    uint32_t acc = 0;
    int64_t p = v;
    for (; p + waves < pieces; p += 2 * waves) {
        uint4 a[kLoads], b[kLoads];
        const uint4* pa = src + p * (kPiece / 16) + lane;
        const uint4* pb = src + (p + waves) * (kPiece / 16) + lane;
#pragma unroll
        for (int i = 0; i < kLoads; ++i) a[i] = pa[64 * i];
#pragma unroll
        for (int i = 0; i < kLoads; ++i) b[i] = pb[64 * i];
#pragma unroll
        for (int i = 0; i < kLoads; ++i) acc ^= a[i].x ^ a[i].y ^ a[i].z ^ a[i].w ^ b[i].x ^ b[i].y ^ b[i].z ^ b[i].w;
    }
    for (; p < pieces; p += waves) {
        const uint4* pa = src + p * (kPiece / 16) + lane;
#pragma unroll
        for (int i = 0; i < kLoads; ++i) {
            const uint4 a = pa[64 * i];
            acc ^= a.x ^ a.y ^ a.z ^ a.w;
        }
    }
    sink[(int64_t)blockIdx.x * 256 + threadIdx.x] = acc;
}

}  // namespace

extern "C" int rg_probe_read(const void* src, int64_t bytes, uint32_t* sink, int32_t grid, void* stream) {
    if (!src || !sink || bytes < kPiece || bytes % kPiece != 0 || grid < 1 || grid > 65536) return 1;
    if (((uintptr_t)src & 15) || ((uintptr_t)sink & 3)) return 1;
    (void)hipGetLastError();
    hipLaunchKernelGGL(read_kernel, dim3((unsigned)grid), dim3(256), 0, (hipStream_t)stream,
                       static_cast<const uint4*>(src), bytes / kPiece, sink);
    return hipGetLastError() == hipSuccess ? 0 : 4;
}
