// Internal interface between the C-ABI (rg_api.cpp) and the kernels (rg_kernels.hip).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace rg {

constexpr int kChunk = 256;  // segment length C of the documented order

struct DecodeArgs {
    const float* x;
    const uint16_t* w;
    const float* bias;  // b[N] added after the fold, or null
    float* y;
    int64_t M, N, K;
    int64_t Q;          // quads of W rows: ceil(N / 4)
    int64_t qbase;      // Q / grid: quads per workgroup ...
    int qrem;           // ... plus one for the first Q % grid workgroups
    int J;              // segments: ceil(K / 256)
    uint32_t jmagic;    // ceil(2^32 / J) for J > 1: n / J = umulhi(n, jmagic) for n < 2^16
    int RQ;             // quads per round
    int reverse;        // 1: row group g takes the quads of row group groups-1-g
    int groups;         // row groups (workgroups per slice)
    int mslices;        // slices of MT rows of x (decode_kernel only; 1 otherwise)
    int max_rows_wg;    // 4 * ceil(Q / grid): rows staged per workgroup
    int round_major;    // 1: quads placed round-major over the grid, 0: one contiguous range each
};

// Arguments of the M == 1 dense-stream kernel (K % 256 == 0, K >= 4096).
struct GemvArgs {
    const float* x;
    const uint16_t* w;
    const float* bias;  // b[N] added after the fold, or null
    float* y;
    int64_t N, K;
    int64_t qbase;      // Q / V quads per wave (Q = ceil(N / 4), V = waves in the grid) ...
    int64_t qrem;       // ... plus one for waves v < Q % V
    int J;              // segments: K / 256
    int S;              // wave steps per quad: ceil(J / 16)
    int reverse;        // 1: workgroup b takes the quads of workgroup grid-1-b
};

// Streaming kernel through LDS (M <= mt <= 4; K % 8 == 0 for BF16 or K % 4 == 0
// for FP32 weights; x and w 16-byte aligned).
struct StreamArgs {
    const float* x;
    const void* w;        // uint16_t bfloat16 bits or float, [N][K]
    const float* bias;    // b[N] added after the fold, or null
    float* y;
    int64_t M, N, K;
    int J;                // ceil(K / kChunk)
    int reverse;          // reversed workgroup-to-block mapping
};

// Arguments of the skinny kernel (M >= 1, K % 8 == 0, K < 2^26, x and W 16-byte aligned).
struct SkinnyArgs {
    const float* x;
    const uint16_t* w;
    const float* bias;    // b[N] added after the fold, or null
    float* y;
    int64_t M, N, K;
    int64_t RG;           // row groups of 16 W rows: ceil(N / 16)
    int64_t groups;       // row-group walkers (workgroups) per slice
    int J;                // segments: ceil(K / 256)
    int NSG;              // segment groups of 4: ceil(J / 4)
    int JP;               // row stride of the partials in LDS: J, or J | 1 (odd: no bank conflicts)
    int mslices;          // slices of MT rows of x
    int reverse;          // 1: walker g takes the row groups of walker groups-1-g, mirrored
};

hipError_t launch_generic(const float* x, const uint16_t* w, const float* bias, float* y, int64_t M, int64_t N,
                          int64_t K, int grid, int reverse, hipStream_t stream);
hipError_t launch_generic(const float* x, const float* w, const float* bias, float* y, int64_t M, int64_t N,
                          int64_t K, int grid, int reverse, hipStream_t stream);
hipError_t launch_stream(const StreamArgs& a, bool f32_weights, int mt, int grid, hipStream_t stream);
hipError_t launch_decode(const DecodeArgs& a, int mt, int grid, int nw, int depth, hipStream_t stream);
hipError_t launch_decode1(const DecodeArgs& a, int grid, int nw, int depth, hipStream_t stream);
hipError_t launch_gemv(const GemvArgs& a, int grid, int nw, hipStream_t stream);
// occ: waves per SIMD of the 128 x 128 tile build (2 or 3; ignored by the other tiles)
hipError_t launch_tiled(const float* x, const uint16_t* w, const float* bias, float* y, int64_t M, int64_t N, int64_t K,
                        int bm, int bn, int occ, int reverse, hipStream_t stream);
hipError_t launch_tiled(const float* x, const float* w, const float* bias, float* y, int64_t M, int64_t N, int64_t K,
                        int bm, int bn, int occ, int reverse, hipStream_t stream);
hipError_t launch_ktile(const float* x, const uint16_t* w, const float* bias, float* y, int64_t M, int64_t N, int64_t K,
                        int bm, int bn, int nt, int cn, int reverse, hipStream_t stream);
hipError_t launch_ktile(const float* x, const float* w, const float* bias, float* y, int64_t M, int64_t N, int64_t K,
                        int bm, int bn, int nt, int cn, int reverse, hipStream_t stream);
// Fixed-order decode attention (include/rg_attn.h).  The workspace regions are
// carved by the caller: t [B][H][Lmax], segmax and spart [B][H][J], mmax [B][H],
// npart [B][H][J][D].  `cus`: compute units of the device (sizes the persistent grids).
struct AttnArgs {
    const float* q;
    const uint16_t* k;
    const uint16_t* v;
    const int32_t* lens;
    float* out;
    float* t;
    float* segmax;
    float* spart;
    float* mmax;
    float* npart;
    int64_t B, H, Hkv, Lmax, D, J;   // J = ceil(Lmax / 256)
    float scale;
    uint32_t vmagic;                 // ceil(2^32 / (D / 8)) for D / 8 > 1 (row of a 16-byte vector)
};
hipError_t launch_attn(const AttnArgs& a, int cus, hipStream_t stream);

// LDS bytes of a skinny launch (DEPTH steps of 8 KB per wave, then two sets of partials).
inline size_t skinny_lds_bytes(int mt, int nw, int depth, int JP) {
    return (size_t)nw * depth * 8192 + (size_t)2 * mt * 16 * JP * sizeof(float);
}
hipError_t launch_skinny(const SkinnyArgs& a, int mt, int spw, int nw, int depth, hipStream_t stream);

hipError_t launch_cast(const uint16_t* w, float* o, int64_t count, hipStream_t stream);
hipError_t launch_argmax(const float* y, int64_t* out, int64_t M, int64_t N, hipStream_t stream);

}  // namespace rg
