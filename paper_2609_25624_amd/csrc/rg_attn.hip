// Fixed-order decode attention kernels for gfx950 (MI355X): the order
// RG-ATTN-1 and its exponential EXP1, both defined in include/rg_attn.h.
//
// Three launches, each deterministic by construction (no atomics, no order
// that depends on the grid):
//   1. scores:   workgroup (b, g, j) stages the keys of positions
//                [256j, 256j + 256) of kv head g in LDS; thread l runs the dot
//                product chain of position l for every query head of the
//                group, scales it, writes t, and the workgroup writes the
//                segment's maximum per head (max is exact, so its tree shape
//                does not matter).
//   2. partials: workgroup (b, g, j) takes m = the maximum of the segment
//                maxima, computes e_l = EXP1(t_l - m) for its positions, the
//                segment sum S_j (one sequential chain per head) and the
//                segment numerators n_j[d] (one fmaf chain per head and d over
//                the positions in ascending order, values staged in LDS).
//   3. fold:     workgroup (b, h) folds the S_j and n_j[d] in ascending j and
//                divides.
// Arithmetic: binary32 fmaf / add / multiply / correctly rounded divide,
// denormals kept, no contraction (the build uses -ffp-contract=off).

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "rg_kernels.h"

namespace rg {
namespace {

constexpr int kAttnSeg = 256;                 // positions per segment

__device__ __forceinline__ float up_bf16(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

// EXP1 of include/rg_attn.h.
__device__ __forceinline__ float exp1(float u) {
    if (u != u) return u;
    if (u < -87.0f) return 0.0f;
    const float k = __builtin_rintf(u * 0x1.715476p+0f);
    float r = __builtin_fmaf(-k, 0x1.62e4p-1f, u);
    r = __builtin_fmaf(-k, 0x1.7f7d1cp-20f, r);
    float p = 0x1.a01a02p-13f;
    p = __builtin_fmaf(p, r, 0x1.6c16c2p-10f);
    p = __builtin_fmaf(p, r, 0x1.111112p-7f);
    p = __builtin_fmaf(p, r, 0x1.555556p-5f);
    p = __builtin_fmaf(p, r, 0x1.555556p-3f);
    p = __builtin_fmaf(p, r, 0.5f);
    p = __builtin_fmaf(p, r, 1.0f);
    p = __builtin_fmaf(p, r, 1.0f);
    return p * __uint_as_float((uint32_t)((int)k + 127) << 23);
}

__device__ __forceinline__ int clamp_len(const int32_t* lens, int64_t b, int64_t Lmax) {
    const int64_t L = lens[b];
    return (int)(L < 0 ? 0 : (L > Lmax ? Lmax : L));
}

// Stage rows [0, rows) of a [*, D] bf16 block (contiguous) into LDS at a row
// stride of D + 8 (16 bytes of pad: the lanes that read one row each hit
// different banks).  D % 8 == 0.
__device__ __forceinline__ void stage_rows(const uint16_t* __restrict__ src, uint16_t* dst, int rows, int D) {
    const int vpr = D / 8;                    // 16-byte vectors per row
    const int total = rows * vpr;
    for (int i = threadIdx.x; i < total; i += blockDim.x) {
        const int r = i / vpr, c = i % vpr;
        *reinterpret_cast<uint4*>(dst + r * (D + 8) + 8 * c) = *reinterpret_cast<const uint4*>(src + (int64_t)r * D + 8 * c);
    }
}

// G query heads per kv head; DM >= D bounds the LDS tiles (64, 128 or 256).
template <int G, int DM>
__global__ void __launch_bounds__(256) attn_scores_kernel(AttnArgs a) {
    __shared__ __attribute__((aligned(16))) float qs[G * DM];                 // [G][D]
    __shared__ __attribute__((aligned(16))) uint16_t ks[kAttnSeg * (DM + 8)]; // [256][D + 8]
    __shared__ float red[G][256];
    const int D = a.D;

    const int64_t j = blockIdx.x % a.J, bg = blockIdx.x / a.J;
    const int64_t b = bg / a.Hkv, g = bg % a.Hkv;
    const int L = clamp_len(a.lens, b, a.Lmax);
    const int l0 = (int)(j * kAttnSeg);
    if (l0 >= L) return;                          // the whole workgroup: no barrier below is skipped by part of it
    const int rows = min(kAttnSeg, L - l0);
    const int64_t h0 = g * G;
    for (int i = threadIdx.x; i < G * D; i += blockDim.x) qs[i] = a.q[(b * a.H + h0) * D + i];
    stage_rows(a.k + ((b * a.Hkv + g) * a.Lmax + l0) * D, ks, rows, D);
    __syncthreads();

    const int l = threadIdx.x;
    float t[G];
    if (l < rows) {
        float z[G];
#pragma unroll
        for (int i = 0; i < G; ++i) z[i] = 0.0f;
        const uint16_t* kr = ks + l * (D + 8);
        for (int d = 0; d < D; d += 8) {
            const uint4 kv = *reinterpret_cast<const uint4*>(kr + d);
            const uint32_t w4[4] = {kv.x, kv.y, kv.z, kv.w};
            float kf[8];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                kf[2 * e] = __uint_as_float(w4[e] << 16);
                kf[2 * e + 1] = __uint_as_float(w4[e] & 0xffff0000u);
            }
#pragma unroll
            for (int i = 0; i < G; ++i)
#pragma unroll
                for (int e = 0; e < 8; ++e) z[i] = __builtin_fmaf(qs[i * D + d + e], kf[e], z[i]);
        }
#pragma unroll
        for (int i = 0; i < G; ++i) {
            t[i] = z[i] * a.scale;
            a.t[((b * a.H + h0 + i) * a.Lmax) + l0 + l] = t[i];
        }
    } else {
#pragma unroll
        for (int i = 0; i < G; ++i) t[i] = -__builtin_inff();
    }
    // segment maximum per head: a fixed tree of fmaxf (exact; NaN never wins)
#pragma unroll
    for (int i = 0; i < G; ++i) red[i][l] = t[i];
    __syncthreads();
    for (int s = 128; s > 0; s >>= 1) {
        if (l < s) {
#pragma unroll
            for (int i = 0; i < G; ++i) red[i][l] = __builtin_fmaxf(red[i][l], red[i][l + s]);
        }
        __syncthreads();
    }
    if (l < G) a.segmax[(b * a.H + h0 + l) * a.J + j] = red[l][0];
}

template <int G, int DM>
__global__ void __launch_bounds__(256) attn_partials_kernel(AttnArgs a) {
    __shared__ __attribute__((aligned(16))) float es[G * kAttnSeg];           // [G][256]
    __shared__ __attribute__((aligned(16))) uint16_t vs[kAttnSeg * (DM + 8)]; // [256][D + 8]
    __shared__ float mh[G];
    const int D = a.D;

    const int64_t j = blockIdx.x % a.J, bg = blockIdx.x / a.J;
    const int64_t b = bg / a.Hkv, g = bg % a.Hkv;
    const int L = clamp_len(a.lens, b, a.Lmax);
    const int l0 = (int)(j * kAttnSeg);
    if (l0 >= L) return;
    const int rows = min(kAttnSeg, L - l0);
    const int Jb = (L + kAttnSeg - 1) / kAttnSeg;
    const int64_t h0 = g * G;
    const int tid = threadIdx.x;
    stage_rows(a.v + ((b * a.Hkv + g) * a.Lmax + l0) * D, vs, rows, D);
    if (tid < G) {
        const float* sm = a.segmax + (b * a.H + h0 + tid) * a.J;
        float m = sm[0];
        for (int jj = 1; jj < Jb; ++jj) m = __builtin_fmaxf(m, sm[jj]);
        mh[tid] = m;
    }
    __syncthreads();
    if (tid < rows) {
#pragma unroll
        for (int i = 0; i < G; ++i)
            es[i * kAttnSeg + tid] = exp1(a.t[(b * a.H + h0 + i) * a.Lmax + l0 + tid] - mh[i]);
    }
    __syncthreads();
    // segment sums: one sequential chain per head
    if (tid < G) {
        float s = 0.0f;
        for (int l = 0; l < rows; ++l) s = s + es[tid * kAttnSeg + l];
        a.spart[(b * a.H + h0 + tid) * a.J + j] = s;
    }
    // segment numerators: thread handles (head, d) pairs p = tid, tid + 256, ... as independent chains
    constexpr int kMaxPairs = (G * DM + 255) / 256;
    const int npairs = G * D;
    float n[kMaxPairs];
    int hh[kMaxPairs], dd[kMaxPairs];
#pragma unroll
    for (int u = 0; u < kMaxPairs; ++u) {
        const int p = tid + 256 * u;
        hh[u] = p < npairs ? p / D : 0;
        dd[u] = p < npairs ? p % D : 0;
        n[u] = 0.0f;
    }
    const int nu = (npairs - tid + 255) / 256;       // pairs of this thread
    for (int l = 0; l < rows; ++l) {
        const uint16_t* vr = vs + l * (D + 8);
#pragma unroll
        for (int u = 0; u < kMaxPairs; ++u)
            if (u < nu) n[u] = __builtin_fmaf(es[hh[u] * kAttnSeg + l], up_bf16(vr[dd[u]]), n[u]);
    }
#pragma unroll
    for (int u = 0; u < kMaxPairs; ++u)
        if (u < nu) a.npart[((b * a.H + h0 + hh[u]) * a.J + j) * D + dd[u]] = n[u];
}

__global__ void __launch_bounds__(256) attn_fold_kernel(AttnArgs a) {
    const int64_t bh = blockIdx.x, b = bh / a.H;
    const int L = clamp_len(a.lens, b, a.Lmax);
    const int Jb = (L + kAttnSeg - 1) / kAttnSeg;
    const int D = a.D;
    for (int d = threadIdx.x; d < D; d += blockDim.x) {
        float S = 0.0f, N = 0.0f;
        const float* sp = a.spart + bh * a.J;
        const float* np = a.npart + bh * a.J * D + d;
        for (int jj = 0; jj < Jb; ++jj) {
            S = (jj == 0) ? sp[0] : S + sp[jj];
            N = (jj == 0) ? np[0] : N + np[(int64_t)jj * D];
        }
        a.out[bh * D + d] = N / S;
    }
}

template <int G, int DM>
hipError_t launch_group(const AttnArgs& a, hipStream_t stream) {
    const int64_t wgs = a.B * a.Hkv * a.J;
    hipLaunchKernelGGL((attn_scores_kernel<G, DM>), dim3((unsigned)wgs), dim3(256), 0, stream, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL((attn_partials_kernel<G, DM>), dim3((unsigned)wgs), dim3(256), 0, stream, a);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(attn_fold_kernel, dim3((unsigned)(a.B * a.H)), dim3(256), 0, stream, a);
    return hipGetLastError();
}

template <int G>
hipError_t launch_dm(const AttnArgs& a, hipStream_t stream) {
    if (a.D <= 64) return launch_group<G, 64>(a, stream);
    if (a.D <= 128) return launch_group<G, 128>(a, stream);
    return launch_group<G, 256>(a, stream);
}

}  // namespace

hipError_t launch_attn(const AttnArgs& a, hipStream_t stream) {
    if (a.D < 8 || a.D > 256 || a.D % 8 != 0 || a.Hkv < 1 || a.H % a.Hkv != 0) return hipErrorInvalidValue;
    switch (a.H / a.Hkv) {
        case 1: return launch_dm<1>(a, stream);
        case 2: return launch_dm<2>(a, stream);
        case 3: return launch_dm<3>(a, stream);
        case 4: return launch_dm<4>(a, stream);
        case 5: return launch_dm<5>(a, stream);
        case 6: return launch_dm<6>(a, stream);
        case 7: return launch_dm<7>(a, stream);
        case 8: return launch_dm<8>(a, stream);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace rg
