// Wave-tile kernel for the fused-upcast linear layer (gfx950): 32 < M <= 64 on wide layers.
//
// Same order as every kernel of the library (include/rg.h, RG-ORDER-1; paper: Design,
// eq. 2 and rules R1-R4): 256-wide K segments, each a chain of fmaf from +0 in ascending
// k, the segment partials folded left to right in ascending segment order.
//
// Work split.  A workgroup owns a 64 x 64 output tile (64 rows of x by 64 rows of W) and
// all of K.  Each of its KS waves holds the whole tile for one segment at a time: lane
// (mi, ni) = (lane % 8, lane / 8) runs the 8 x 8 chains of x rows {4mi .. 4mi+3, 32+4mi ..
// 32+4mi+3} and W rows {4ni .. 4ni+3, 32+4ni .. 32+4ni+3}.  Wave g runs segments g, g + KS,
// g + 2KS, ...; each wave stages the 8-k slabs of its own segment (x, and W widened once)
// through its own double-buffered LDS region, so a segment runs without any barrier.
// Per k a lane reads two float4 of x and two of W (the eight lanes that share an address
// get it by broadcast) and issues 64 plain FMAs: one LDS byte per FMA.
//
// Fold.  After each round the waves add their segment partials to the tile's running
// totals in LDS one after another, in ascending segment order (the first partial starts
// the sum); the wave that adds the last segment writes y (+ b).  No atomics, no workspace,
// no second launch.
//
// Arithmetic: only v_fmac_f32 / v_fma_f32 and v_add_f32 (the library is built with
// -ffp-contract=off and packed FP32 disabled), binary32 denormals preserved.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "rg_kernels.h"
#include "rg_wtile.h"

namespace rg {
namespace {

// Weight elements of a 16-byte vector: bfloat16 bit patterns widened exactly (bits << 16;
// element k at the lower address in the low half of a dword), float32 weights as they are.
template <typename WT>
struct WtVec;
template <>
struct WtVec<uint16_t> {
    using V = uint4;
    static constexpr int E = 8;
    static __device__ __forceinline__ V zero() { return make_uint4(0u, 0u, 0u, 0u); }
    static __device__ __forceinline__ float get(const V& v, int h) {
        const uint32_t d[4] = {v.x, v.y, v.z, v.w};
        const uint32_t u = d[h >> 1];
        return __uint_as_float((h & 1) ? (u & 0xffff0000u) : (u << 16));
    }
};
template <>
struct WtVec<float> {
    using V = float4;
    static constexpr int E = 4;
    static __device__ __forceinline__ V zero() { return make_float4(0.f, 0.f, 0.f, 0.f); }
    static __device__ __forceinline__ float get(const V& v, int h) {
        const float d[4] = {v.x, v.y, v.z, v.w};
        return d[h];
    }
};

constexpr int kT = kWtileRows;        // tile rows (x) = tile rows (W)
constexpr int kPad = kWtileRows + 4;  // LDS row of one k: 64 values and 4 of padding
constexpr int kKT = kWtileK;          // k per slab

}  // namespace

template <int KS, typename WT>
__global__ void __launch_bounds__(64 * KS) wtile_kernel(const float* __restrict__ x, const WT* __restrict__ w,
                                                        const float* __restrict__ bias, float* __restrict__ y,
                                                        int64_t M, int64_t N, int64_t K, int reverse) {
    using WV = WtVec<WT>;
    constexpr int NSL = kChunk / kKT;             // slabs per segment
    constexpr int WPR = kKT / WV::E;              // weight vectors per slab row
    constexpr int XPT = kT * kKT / 4 / 64;        // float4 x loads per lane per slab
    constexpr int WPT = kT * WPR / 64;            // weight vector loads per lane per slab
    static_assert(XPT * 64 * 4 == kT * kKT && WPT * 64 == kT * WPR && WPR >= 1, "slab split");
    static_assert(NSL % 2 == 0, "slabs of a segment alternate between the two buffers");
    __shared__ __attribute__((aligned(16))) float xs[KS][2][kKT][kPad];
    __shared__ __attribute__((aligned(16))) float ws[KS][2][kKT][kPad];
    __shared__ __attribute__((aligned(16))) float4 tots[16][64];   // running totals, lane-major

    const int lane = threadIdx.x & 63, g = threadIdx.x >> 6;
    const int mi = lane & 7, ni = lane >> 3;
    const int64_t tiles_n = (N + kT - 1) / kT;
    const int64_t b = reverse ? (int64_t)(gridDim.x - 1 - blockIdx.x) : (int64_t)blockIdx.x;
    const int64_t m0 = (b / tiles_n) * kT, n0 = (b % tiles_n) * kT;
    const int J = (int)((K + kChunk - 1) / kChunk);
    const int rounds = (J + KS - 1) / KS;

    // two register sets: slab s of this wave (its slabs numbered across rounds) lives in set
    // s % 2, loaded three slabs before it is computed and stored to LDS one slab before
    float4 xr[2][XPT];
    typename WV::V wr[2][WPT];
    // this wave's slab s into register set R.  Every lane loads, from an address clamped into
    // x and W: rows past M or N then hold copies of the last row (their outputs are never
    // stored) and k past K or past the last segment copies of the first (never multiplied:
    // a short slab runs only its valid k).  Unconditional loads let the compiler's waits count
    // exactly the slabs still in flight.
    auto load_slab = [&](auto R, int s) {
        const int t = s / NSL, sl = s % NSL;
        const int64_t j = (int64_t)t * KS + g;
        const int64_t k0 = j * kChunk + (int64_t)sl * kKT;
#pragma unroll
        for (int u = 0; u < XPT; ++u) {
            const int idx = lane + 64 * u;               // over 64 rows x kKT/4 float4
            const int row = idx / (kKT / 4), kq = idx % (kKT / 4);
            const int64_t gm = m0 + row, gk = k0 + 4 * kq;
            const bool kok = j < J && gk + 4 <= K;
            xr[R][u] = *reinterpret_cast<const float4*>(x + (gm < M ? gm : M - 1) * K + (kok ? gk : 0));
        }
#pragma unroll
        for (int u = 0; u < WPT; ++u) {
            const int idx = lane + 64 * u;               // over 64 rows x WPR vectors
            const int row = idx / WPR, kh = idx % WPR;
            const int64_t gn = n0 + row, gk = k0 + WV::E * kh;
            const bool kok = j < J && gk + WV::E <= K;
            // (a normal load: a slab reads 16 or 32 bytes of each 128-byte line of a row and the
            // next slabs the rest, which a non-temporal load would not find in the cache)
            wr[R][u] = *reinterpret_cast<const typename WV::V*>(w + (gn < N ? gn : N - 1) * K + (kok ? gk : 0));
        }
    };
    // register set R into this wave's LDS buffer R, transposed to [k][row]
    auto store_slab = [&](auto R) {
        constexpr int buf = decltype(R)::value;
#pragma unroll
        for (int u = 0; u < XPT; ++u) {
            const int idx = lane + 64 * u;
            const int row = idx / (kKT / 4), kq = idx % (kKT / 4);
            xs[g][buf][4 * kq + 0][row] = xr[buf][u].x;
            xs[g][buf][4 * kq + 1][row] = xr[buf][u].y;
            xs[g][buf][4 * kq + 2][row] = xr[buf][u].z;
            xs[g][buf][4 * kq + 3][row] = xr[buf][u].w;
        }
#pragma unroll
        for (int u = 0; u < WPT; ++u) {
            const int idx = lane + 64 * u;
            const int row = idx / WPR, kh = idx % WPR;
#pragma unroll
            for (int h = 0; h < WV::E; ++h) ws[g][buf][WV::E * kh + h][row] = WV::get(wr[buf][u], h);
        }
    };

    float acc[64];
    // the operands of one k: x rows {4mi .. 4mi+3, 32+4mi ..} and W rows {4ni .., 32+4ni ..}
    struct Ops {
        float4 x0, x1, w0, w1;
    };
    auto read_k = [&](int buf, int kk) {
        Ops o;
        o.x0 = *reinterpret_cast<const float4*>(&xs[g][buf][kk][4 * mi]);
        o.x1 = *reinterpret_cast<const float4*>(&xs[g][buf][kk][32 + 4 * mi]);
        o.w0 = *reinterpret_cast<const float4*>(&ws[g][buf][kk][4 * ni]);
        o.w1 = *reinterpret_cast<const float4*>(&ws[g][buf][kk][32 + 4 * ni]);
        return o;
    };
    // one k of the 8 x 8 chains: acc[8r + c] += x[row r] * w[row c]
    auto fma_ops = [&](const Ops& o) {
        const float xa[8] = {o.x0.x, o.x0.y, o.x0.z, o.x0.w, o.x1.x, o.x1.y, o.x1.z, o.x1.w};
        const float wa[8] = {o.w0.x, o.w0.y, o.w0.z, o.w0.w, o.w1.x, o.w1.y, o.w1.z, o.w1.w};
#pragma unroll
        for (int r = 0; r < 8; ++r)
#pragma unroll
            for (int c = 0; c < 8; ++c) acc[8 * r + c] = __builtin_fmaf(xa[r], wa[c], acc[8 * r + c]);
    };
    auto fma_k = [&](int buf, int kk) { fma_ops(read_k(buf, kk)); };

    using R0 = std::integral_constant<int, 0>;
    using R1 = std::integral_constant<int, 1>;
    load_slab(R0{}, 0);
    store_slab(R0{});
    load_slab(R1{}, 1);
    load_slab(R0{}, 2);
    // move slab s + 1 from registers to the other LDS buffer, load slab s + 3 into the
    // registers it freed, then compute slab s from buffer s % 2 with the next k's operands
    // read while the current k's FMAs run (a wave's LDS operations run in order and only this
    // wave touches its buffers, so no barrier is needed)
    auto slab = [&](auto R, int s, int len, int sl) {
        constexpr int buf = decltype(R)::value;
        using RN = std::integral_constant<int, 1 - buf>;
        store_slab(RN{});
        load_slab(RN{}, s + 3);
        const int kvalid = max(0, min(kKT, len - sl * kKT));
        if (kvalid == kKT) {
            Ops cur = read_k(buf, 0);
#pragma unroll
            for (int kk = 0; kk < kKT; ++kk) {
                Ops nxt;
                if (kk + 1 < kKT) nxt = read_k(buf, kk + 1);
                __builtin_amdgcn_sched_barrier(0);
                fma_ops(cur);
                __builtin_amdgcn_sched_barrier(0);
                if (kk + 1 < kKT) cur = nxt;
            }
        } else {
            for (int kk = 0; kk < kvalid; ++kk) fma_k(buf, kk);
        }
    };
    for (int t = 0; t < rounds; ++t) {
        const int64_t j = (int64_t)t * KS + g;
#pragma unroll
        for (int i = 0; i < 64; ++i) acc[i] = 0.0f;
        if (j < J) {
            const int len = (int)min((int64_t)kChunk, K - j * kChunk);   // this segment's length
            for (int sl = 0; sl < NSL; sl += 2) {
                slab(R0{}, t * NSL + sl, len, sl);
                slab(R1{}, t * NSL + sl + 1, len, sl + 1);
            }
        }
        // the round's partials join the totals wave by wave, in ascending segment order
        for (int gg = 0; gg < KS; ++gg) {
            __syncthreads();
            if (g == gg && j < J) {
                if (j > 0) {
#pragma unroll
                    for (int q = 0; q < 16; ++q) {
                        const float4 tv = tots[q][lane];
                        acc[4 * q + 0] = tv.x + acc[4 * q + 0];
                        acc[4 * q + 1] = tv.y + acc[4 * q + 1];
                        acc[4 * q + 2] = tv.z + acc[4 * q + 2];
                        acc[4 * q + 3] = tv.w + acc[4 * q + 3];
                    }
                }
                if (j + 1 < J) {
#pragma unroll
                    for (int q = 0; q < 16; ++q)
                        tots[q][lane] = make_float4(acc[4 * q], acc[4 * q + 1], acc[4 * q + 2], acc[4 * q + 3]);
                } else {
                    // the last segment: the totals are the outputs
#pragma unroll
                    for (int r = 0; r < 8; ++r) {
                        const int64_t gm = m0 + (r < 4 ? 4 * mi + r : 32 + 4 * mi + (r - 4));
                        if (gm >= M) continue;
#pragma unroll
                        for (int c = 0; c < 8; ++c) {
                            const int64_t gn = n0 + (c < 4 ? 4 * ni + c : 32 + 4 * ni + (c - 4));
                            if (gn < N) y[gm * N + gn] = bias ? acc[8 * r + c] + bias[gn] : acc[8 * r + c];
                        }
                    }
                }
            }
        }
    }
}

namespace {

template <typename WT>
hipError_t launch_wtile_t(const float* x, const WT* w, const float* bias, float* y, int64_t M, int64_t N,
                          int64_t K, int waves, int reverse, hipStream_t stream) {
    const int64_t tiles = ((M + kT - 1) / kT) * ((N + kT - 1) / kT);
    if (tiles < 1 || tiles > 0x7fffffff || (waves != 4 && waves != 8)) return hipErrorInvalidValue;
    if (waves == 4)
        hipLaunchKernelGGL((wtile_kernel<4, WT>), dim3((unsigned)tiles), dim3(256), 0, stream, x, w, bias, y, M, N, K,
                           reverse);
    else
        hipLaunchKernelGGL((wtile_kernel<8, WT>), dim3((unsigned)tiles), dim3(512), 0, stream, x, w, bias, y, M, N, K,
                           reverse);
    return hipGetLastError();
}

}  // namespace

static_assert(wtile_lds_bytes(4) == sizeof(float) * (4 * 2 * kKT * kPad * 2 + 16 * 64 * 4), "LDS size");

hipError_t launch_wtile(const float* x, const uint16_t* w, const float* bias, float* y, int64_t M, int64_t N,
                        int64_t K, int waves, int reverse, hipStream_t stream) {
    return launch_wtile_t(x, w, bias, y, M, N, K, waves, reverse, stream);
}

hipError_t launch_wtile(const float* x, const float* w, const float* bias, float* y, int64_t M, int64_t N,
                        int64_t K, int waves, int reverse, hipStream_t stream) {
    return launch_wtile_t(x, w, bias, y, M, N, K, waves, reverse, stream);
}

}  // namespace rg
