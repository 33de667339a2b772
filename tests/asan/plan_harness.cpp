// Host-side entry points of librg (the planner, launch settings, argument checks, workspace
// sizes) under AddressSanitizer and UndefinedBehaviorSanitizer, over many shapes and settings.
// Built with the library's own rg_api.cpp; the kernel launchers are stubs, and no call here
// reaches a launch or a device query (every rg_linear call below fails its argument checks).
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stdio.h>

#include "../../include/rg.h"
#include "../../include/rg_attn.h"
#include "../../paper_2609_25624_amd/csrc/rg_kernels.h"
#include "../../paper_2609_25624_amd/csrc/rg_wtile.h"

namespace rg {
static hipError_t stub() { return hipErrorInvalidValue; }
hipError_t launch_attn(const AttnArgs&, int, hipStream_t) { return stub(); }
hipError_t launch_cast(const uint16_t*, float*, int64_t, hipStream_t) { return stub(); }
hipError_t launch_argmax(const float*, int64_t*, int64_t, int64_t, hipStream_t) { return stub(); }
hipError_t launch_gemv(const GemvArgs&, int, int, hipStream_t) { return stub(); }
hipError_t launch_decode(const DecodeArgs&, int, int, int, int, hipStream_t) { return stub(); }
hipError_t launch_decode1(const DecodeArgs&, int, int, int, hipStream_t) { return stub(); }
hipError_t launch_skinny(const SkinnyArgs&, int, int, int, int, hipStream_t) { return stub(); }
hipError_t launch_stream(const StreamArgs&, bool, int, int, hipStream_t) { return stub(); }
hipError_t launch_ktile(const float*, const uint16_t*, const float*, float*, int64_t, int64_t, int64_t, int, int, int,
                        int, int, hipStream_t) { return stub(); }
hipError_t launch_ktile(const float*, const float*, const float*, float*, int64_t, int64_t, int64_t, int, int, int, int,
                        int, hipStream_t) { return stub(); }
hipError_t launch_tiled(const float*, const uint16_t*, const float*, float*, int64_t, int64_t, int64_t, int, int, int,
                        int, hipStream_t) { return stub(); }
hipError_t launch_tiled(const float*, const float*, const float*, float*, int64_t, int64_t, int64_t, int, int, int, int,
                        hipStream_t) { return stub(); }
hipError_t launch_wtile(const float*, const uint16_t*, const float*, float*, int64_t, int64_t, int64_t, int, int,
                        hipStream_t) { return stub(); }
hipError_t launch_wtile(const float*, const float*, const float*, float*, int64_t, int64_t, int64_t, int, int,
                        hipStream_t) { return stub(); }
hipError_t launch_generic(const float*, const uint16_t*, const float*, float*, int64_t, int64_t, int64_t, int, int,
                          hipStream_t) { return stub(); }
hipError_t launch_generic(const float*, const float*, const float*, float*, int64_t, int64_t, int64_t, int, int,
                          hipStream_t) { return stub(); }
}  // namespace rg

int main() {
    const int64_t Ms[] = {1, 2, 3, 4, 5, 8, 9, 16, 17, 24, 32, 33, 48, 64, 65, 128, 2048, 65536, 1 << 20};
    const int64_t Ns[] = {1, 7, 15, 16, 17, 300, 1030, 4096, 6144, 28672, 57344, 128256, 1048579, 1 << 28};
    const int64_t Ks[] = {1, 4, 7, 8, 255, 256, 264, 1000, 4096, 4352, 14336, 28672, 32776, 1 << 20, (1 << 26) + 8};
    rg_launch_t cfgs[24] = {};
    int nc = 1;                                                   // cfgs[0]: the defaults
    const int kernels[] = {1, 2, 3, 4, 5, 6, 7, 8, 9};
    for (int k : kernels) cfgs[nc++].kernel = k;                  // every kernel forced
    cfgs[nc].waves_per_wg = 3; cfgs[nc++].grid_wgs = 97;
    cfgs[nc].depth = 2; cfgs[nc++].grid_order = 1;
    cfgs[nc].kernel = 8; cfgs[nc++].slice_m = 1;
    cfgs[nc].kernel = 7; cfgs[nc++].tile_n = 64;
    cfgs[nc].kernel = 9; cfgs[nc++].waves_per_wg = 8;
    cfgs[nc].kernel = 3; cfgs[nc].depth = 3; cfgs[nc++].tile_n = 128;   // invalid tile: rejected
    cfgs[nc++].kernel = 10;                                             // no such kernel: rejected
    cfgs[nc++].grid_wgs = 65537;                                        // too many: rejected
    long plans = 0, rejected = 0;
    for (int c = 0; c < nc; ++c) {
        if (rg_linear_set_launch(c == 0 ? nullptr : &cfgs[c]) != RG_OK) {
            ++rejected;
            continue;
        }
        for (int64_t M : Ms)
            for (int64_t N : Ns)
                for (int64_t K : Ks) {
                    rg_plan_t p;
                    if (rg_plan(M, N, K, &p) == RG_OK) {
                        ++plans;
                        if (p.chunk != 256 || p.nchunks != (K + 255) / 256) return 2;
                    }
                    if (rg_plan_f32w(M, N, K, &p) == RG_OK) ++plans;
                }
    }
    rg_linear_set_launch(nullptr);
    // argument checks that fail before any device work
    float* x = reinterpret_cast<float*>(0x10000);
    uint16_t* w = reinterpret_cast<uint16_t*>(0x200000);
    float* y = reinterpret_cast<float*>(0x4000000);
    if (rg_linear(nullptr, w, y, 4, 4, 4, nullptr) != RG_ERR_INVAL) return 3;
    if (rg_linear(x, w, y, 0, 4, 4, nullptr) != RG_ERR_INVAL) return 3;
    if (rg_linear(x, w, y, (int64_t)1 << 40, (int64_t)1 << 40, 4, nullptr) != RG_ERR_INVAL) return 3;
    if (rg_linear(x + 1, w, reinterpret_cast<float*>(reinterpret_cast<char*>(y) + 2), 4, 4, 4, nullptr) != RG_ERR_ALIGN)
        return 3;
    if (rg_linear(x, w, x, 4, 4, 4, nullptr) != RG_ERR_ALIAS) return 3;
    for (int64_t B : {1, 16, 1 << 20})
        for (int64_t L : {1, 256, 4097, 1 << 22})
            for (int64_t D : {8, 64, 128, 256}) (void)rg_attn_workspace_size(B, 32, L, D);
    printf("ok: %ld plans, %ld launch settings rejected\n", plans, rejected);
    return 0;
}
