// Read-bandwidth probe (include/rg_probe.h): a kernel that reads and does nothing else.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/rg_probe.h"

namespace {

constexpr int kPiece = 8192;                 // bytes per wave piece: 8 loads of 1 KB per wave
constexpr int kLoads = kPiece / (64 * 16);   // 16-byte loads per lane per piece

// One 16-byte load, non-temporal (data read once; the linear-layer kernels stream weights so).
__device__ __forceinline__ uint4 ld(const uint4* p) {
    using E = __attribute__((ext_vector_type(4))) uint32_t;
    const E e = __builtin_nontemporal_load(reinterpret_cast<const E*>(p));
    return make_uint4(e.x, e.y, e.z, e.w);
}

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
        for (int i = 0; i < kLoads; ++i) a[i] = ld(pa + 64 * i);
#pragma unroll
        for (int i = 0; i < kLoads; ++i) b[i] = ld(pb + 64 * i);
#pragma unroll
        for (int i = 0; i < kLoads; ++i) acc ^= a[i].x ^ a[i].y ^ a[i].z ^ a[i].w ^ b[i].x ^ b[i].y ^ b[i].z ^ b[i].w;
    }
    for (; p < pieces; p += waves) {
        const uint4* pa = src + p * (kPiece / 16) + lane;
#pragma unroll
        for (int i = 0; i < kLoads; ++i) {
            const uint4 a = ld(pa + 64 * i);
            acc ^= a.x ^ a.y ^ a.z ^ a.w;
        }
    }
    sink[(int64_t)blockIdx.x * 256 + threadIdx.x] = acc;
}

// FMA issue-rate probe: CH independent accumulator chains per thread, each step one
// v_fmac_f32 per chain with its first operand read plainly (MODE 0), through a DPP row
// broadcast (MODE 1, row_newbcast), through a DPP quad broadcast (MODE 2, quad_perm), from
// an SGPR (MODE 3, a value the whole wave shares; a different SGPR for each chain) or from an
// SGPR and a VGPR in turn (MODE 4: even chains SGPR, odd chains plain).  The operands are non-trivial values near 1 (so the
// arithmetic switches as much as real data does).
template <int CH, int MODE>
__global__ void __launch_bounds__(256) fma_kernel(float* out, int iters) {
    float a[CH];
#pragma unroll
    for (int i = 0; i < CH; ++i) a[i] = threadIdx.x * 1e-3f + i;
    const float xs[4] = {1.0001f + threadIdx.x * 1e-9f, 0.9999f, 1.00002f, 0.99998f};
    const float w0 = 0.5f + threadIdx.x * 1e-7f, w1 = 0.25f;
    // wave-uniform operands, held in SGPRs (the empty asm keeps each in its own SGPR)
    int sx[CH];
#pragma unroll
    for (int j = 0; j < CH; ++j) {
        sx[j] = __builtin_amdgcn_readfirstlane(__float_as_int(xs[j & 3]) + j * 7);
        if constexpr (MODE >= 3) asm volatile("" : "+s"(sx[j]));
    }
    for (int it = 0; it < iters; ++it) {
#pragma unroll
        for (int r = 0; r < 64 / CH; ++r) {
            if (MODE == 1 || MODE == 2) asm volatile("s_nop 1");   // the wait states a DPP read of a fresh VGPR needs
#pragma unroll
            for (int i = 0; i < CH; ++i) {
                if constexpr (MODE == 0)
                    asm volatile("v_fmac_f32 %0, %1, %2" : "+v"(a[i]) : "v"(xs[i & 3]), "v"((i & 4) ? w0 : w1));
                else if constexpr (MODE == 1)
                    asm volatile("v_fmac_f32_dpp %0, %1, %2 row_newbcast:5 row_mask:0xf bank_mask:0xf"
                                 : "+v"(a[i]) : "v"(xs[i & 3]), "v"((i & 4) ? w0 : w1));
                else if constexpr (MODE == 2)
                    asm volatile("v_fmac_f32_dpp %0, %1, %2 quad_perm:[1,1,1,1] row_mask:0xf bank_mask:0xf bound_ctrl:1"
                                 : "+v"(a[i]) : "v"(xs[i & 3]), "v"((i & 4) ? w0 : w1));
                else if constexpr (MODE == 3)
                    asm volatile("v_fmac_f32 %0, %1, %2" : "+v"(a[i]) : "s"(sx[i]), "v"((i & 4) ? w0 : w1));
                else if (i & 1)
                    asm volatile("v_fmac_f32 %0, %1, %2" : "+v"(a[i]) : "v"(xs[i & 3]), "v"((i & 4) ? w0 : w1));
                else
                    asm volatile("v_fmac_f32 %0, %1, %2" : "+v"(a[i]) : "s"(sx[i]), "v"((i & 4) ? w0 : w1));
            }
        }
    }
    float s = 0.0f;
#pragma unroll
    for (int i = 0; i < CH; ++i) s += a[i];
    out[(int64_t)blockIdx.x * 256 + threadIdx.x] = s;
}

}  // namespace

extern "C" int rg_probe_fma(int32_t mode, int32_t chains, float* out, int32_t grid, int32_t iters, void* stream) {
    if (!out || ((uintptr_t)out & 3) || grid < 1 || grid > 65536 || iters < 1 || mode < 0 || mode > 4) return 1;
    if (chains != 8 && chains != 16) return 1;
    (void)hipGetLastError();
    const dim3 g((unsigned)grid), b(256);
    hipStream_t st = (hipStream_t)stream;
    switch (mode * 100 + chains) {
        case 8: hipLaunchKernelGGL((fma_kernel<8, 0>), g, b, 0, st, out, iters); break;
        case 16: hipLaunchKernelGGL((fma_kernel<16, 0>), g, b, 0, st, out, iters); break;
        case 108: hipLaunchKernelGGL((fma_kernel<8, 1>), g, b, 0, st, out, iters); break;
        case 116: hipLaunchKernelGGL((fma_kernel<16, 1>), g, b, 0, st, out, iters); break;
        case 208: hipLaunchKernelGGL((fma_kernel<8, 2>), g, b, 0, st, out, iters); break;
        case 216: hipLaunchKernelGGL((fma_kernel<16, 2>), g, b, 0, st, out, iters); break;
        case 308: hipLaunchKernelGGL((fma_kernel<8, 3>), g, b, 0, st, out, iters); break;
        case 316: hipLaunchKernelGGL((fma_kernel<16, 3>), g, b, 0, st, out, iters); break;
        case 408: hipLaunchKernelGGL((fma_kernel<8, 4>), g, b, 0, st, out, iters); break;
        default: hipLaunchKernelGGL((fma_kernel<16, 4>), g, b, 0, st, out, iters); break;
    }
    return hipGetLastError() == hipSuccess ? 0 : 4;
}

extern "C" int rg_probe_read(const void* src, int64_t bytes, uint32_t* sink, int32_t grid, void* stream) {
    if (!src || !sink || bytes < kPiece || bytes % kPiece != 0 || grid < 1 || grid > 65536) return 1;
    if (((uintptr_t)src & 15) || ((uintptr_t)sink & 3)) return 1;
    (void)hipGetLastError();
    hipLaunchKernelGGL(read_kernel, dim3((unsigned)grid), dim3(256), 0, (hipStream_t)stream,
                       static_cast<const uint4*>(src), bytes / kPiece, sink);
    return hipGetLastError() == hipSuccess ? 0 : 4;
}
