// Fixed-order decode attention kernels for gfx950 (MI355X): the order
// RG-ATTN-1 and its exponential EXP1, both defined in include/rg_attn.h.
//
// Four launches (three when the partials kernel takes the row maxima itself),
// each deterministic by construction (no atomics, no order that depends on the
// grid):
//   1. scores:   work item (b, g, j) = segment j (positions [256j, 256j + 256))
//                of kv head g of sequence b; its keys are staged in LDS and
//                thread l runs the dot product chain of position l for every
//                query head of the group, scales it, writes t, and the
//                workgroup writes the segment's maximum per head (max is
//                exact, so its tree shape does not matter).
//   2. max:      m[b][h] = the largest segment maximum (exact, so it is the same
//                value when the partials kernel reduces it per item instead).
//   3. partials: per work item, e_l = EXP1(t_l - m), the segment sum S_j (one
//                addition chain per head) and the segment numerators n_j[d]
//                (one fmaf chain per head and d over the positions in
//                ascending order; values and e staged in LDS).
//   4. fold:     workgroup (b, h) folds the S_j and n_j[d] in ascending j and
//                divides.
// Kernels 1 and 3 are persistent: a workgroup (kernel 1; kernel 3 for head dims
// other than 128 and 256) walks work items it, it + grid, ... in steps of one
// 32 KB tile (for the usual head dims), or for kernel 3 with head dims 128 and
// 256 a single wave walks them in 8 KB steps; either fetches the next step into
// registers while it computes the current one from LDS.
// Arithmetic: binary32 fmaf / add / multiply / correctly rounded divide,
// denormals kept, no contraction (the build uses -ffp-contract=off).

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "rg_kernels.h"

namespace rg {

// A 16-byte non-temporal load (key and value rows that a pass reads whole, once per call).
__device__ __forceinline__ uint4 ldnt(const uint4* p) {
    using E = __attribute__((ext_vector_type(4))) uint32_t;
    const E e = __builtin_nontemporal_load(reinterpret_cast<const E*>(p));
    return make_uint4(e.x, e.y, e.z, e.w);
}

namespace {

constexpr int kAttnSeg = 256;                 // positions per segment

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

// A step's tile: `rows` rows of VPR 16-byte vectors (8 bf16 each) taken from a
// [*, D] bf16 block at row stride D, staged in LDS at a row stride of
// 8 * VPR + 8 (16 bytes of pad: lanes that read one row each hit different
// banks).  It is fetched into registers one step ahead (every load issued
// before the first use) and stored to LDS between barriers; rows past the
// sequence are +0.  Thread t holds vectors t, t + 256, ...; the row of vector i
// is i / VPR (a shift for the fixed shapes, else a multiply by `vmagic` =
// ceil(2^32 / vpr), exact for i < 8192).
template <int NV, int VPR>   // VPR > 0: fixed vectors per row; 0: vpr at run time
struct Tile {
    uint4 r[NV];
    __device__ __forceinline__ static int row_of(int i, int vpr, uint32_t vmagic) {
        if constexpr (VPR > 0) return i / VPR;
        return vpr == 1 ? i : (int)__umulhi((uint32_t)i, vmagic);
    }
    __device__ __forceinline__ void fetch(const uint16_t* __restrict__ src, int64_t stride, int rows, int vpr,
                                          uint32_t vmagic) {
        if constexpr (VPR > 0) vpr = VPR;
        const int limit = rows * vpr;
#pragma unroll
        for (int u = 0; u < NV; ++u) {
            const int i = (int)threadIdx.x + 256 * u;
            const int row = row_of(i, vpr, vmagic);
            r[u] = i < limit ? ldnt(reinterpret_cast<const uint4*>(src + row * stride + 8 * (i - row * vpr)))
                             : make_uint4(0u, 0u, 0u, 0u);
        }
    }
    __device__ __forceinline__ void store(uint16_t* dst, int rows_total, int vpr, uint32_t vmagic) const {
        if constexpr (VPR > 0) vpr = VPR;
#pragma unroll
        for (int u = 0; u < NV; ++u) {
            const int i = (int)threadIdx.x + 256 * u;
            if (VPR > 0 || i < rows_total * vpr) {
                const int row = row_of(i, vpr, vmagic);
                *reinterpret_cast<uint4*>(dst + 8 * (i + row)) = r[u];   // row * (8 vpr + 8) + 8 (i % vpr)
            }
        }
    }
};

// Work item it = (b * Hkv + g) * J + j: segment j of kv head g of sequence b.
struct Item {
    int b, g, j;
    int L, l0, rows;
};

__device__ __forceinline__ Item item_of(const AttnArgs& a, int it) {
    Item w;
    const int J = (int)a.J, Hkv = (int)a.Hkv;
    const int bg = it / J;
    w.j = it - bg * J;
    w.b = bg / Hkv;
    w.g = bg - w.b * Hkv;
    w.L = clamp_len(a.lens, w.b, a.Lmax);
    w.l0 = w.j * kAttnSeg;
    w.rows = w.L - w.l0 < kAttnSeg ? w.L - w.l0 : kAttnSeg;
    return w;
}

// The first item at or after `it`, stepping by the grid, that holds positions.
__device__ __forceinline__ int next_item(const AttnArgs& a, int it, int items) {
    while (it < items && item_of(a, it).rows <= 0) it += (int)gridDim.x;
    return it;
}

typedef const __attribute__((address_space(4))) float cfloat;   // read-only: uniform loads go to SGPRs

// Exact maximum over the workgroup of one value per thread: lanes by xor
// shuffles, then the four waves through LDS (fmaxf is exact and NaN never
// wins, so any tree gives the same value).
template <int G>
__device__ __forceinline__ void block_max(float (&v)[G], float (*wred)[G]) {
#pragma unroll
    for (int sh = 32; sh > 0; sh >>= 1)
#pragma unroll
        for (int i = 0; i < G; ++i) v[i] = __builtin_fmaxf(v[i], __shfl_xor(v[i], sh, 64));
    if ((threadIdx.x & 63) == 0) {
#pragma unroll
        for (int i = 0; i < G; ++i) wred[threadIdx.x >> 6][i] = v[i];
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < G; ++i)
        v[i] = __builtin_fmaxf(__builtin_fmaxf(wred[0][i], wred[1][i]), __builtin_fmaxf(wred[2][i], wred[3][i]));
}

// 1. scores and segment maxima.  Work item = segment; its NC steps take the keys'
// columns [c DC, c DC + DC) in turn (DC = 64 for the fixed head dims, else DC = D
// in one step), so each thread's dot product chain of position l continues across
// the steps in ascending d.  G query heads per kv head, their chains interleaved;
// q is read with uniform (scalar) loads.
template <int G, int DC, int NC, bool EXACT>
__global__ void __launch_bounds__(256) attn_scores_kernel(AttnArgs a) {
    constexpr int VPR = EXACT ? DC / 8 : 0;
    constexpr int NV = DC / 8;                                                // vectors per thread (256 rows)
    __shared__ __attribute__((aligned(16))) uint16_t ks[kAttnSeg * (DC + 8)]; // [256][DC + 8]
    __shared__ float wred[4][G];
    const int D = EXACT ? DC * NC : (int)a.D, l = threadIdx.x;
    const int dc = EXACT ? DC : D;                    // columns per step
    const int vpr = dc / 8;
    const int items = (int)(a.B * a.Hkv * a.J);
    cfloat* q4 = (cfloat*)a.q;
    Tile<NV, VPR> tile;
    auto fetch = [&](const Item& w, int c) {
        tile.fetch(a.k + (((int64_t)w.b * a.Hkv + w.g) * a.Lmax + w.l0) * D + c * dc, D, w.rows, vpr, a.vmagic);
    };
    int it = next_item(a, (int)blockIdx.x, items);
    Item w;
    int c = 0;
    if (it < items) {
        w = item_of(a, it);
        fetch(w, 0);
    }
    float z[G];
    while (it < items) {
        __syncthreads();                              // the previous step's reads of LDS are done
        tile.store(ks, kAttnSeg, vpr, a.vmagic);
        __syncthreads();
        const Item cur = w;
        const int cc = c;
        if (c + 1 < NC) {
            ++c;
        } else {
            c = 0;
            it = next_item(a, it + (int)gridDim.x, items);
            if (it < items) w = item_of(a, it);
        }
        if (it < items) fetch(w, c);                  // in flight during this step's chains
        if (cc == 0) {
#pragma unroll
            for (int i = 0; i < G; ++i) z[i] = 0.0f;
        }
        const int64_t h0 = (int64_t)cur.g * G;
        const int64_t qbase = ((int64_t)cur.b * a.H + h0) * D + cc * dc;
        if (l < cur.rows) {
            const uint16_t* kr = ks + l * (dc + 8);
#pragma unroll 1
            for (int d = 0; d < DC; d += 8) {
                if (!EXACT && d >= dc) break;
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
                    for (int e = 0; e < 8; ++e) z[i] = __builtin_fmaf(q4[qbase + i * D + d + e], kf[e], z[i]);
            }
        }
        if (cc == NC - 1) {
            float t[G];
#pragma unroll
            for (int i = 0; i < G; ++i) {
                t[i] = l < cur.rows ? z[i] * a.scale : -__builtin_inff();
                if (l < cur.rows) a.t[(((int64_t)cur.b * a.H + h0 + i) * a.Lmax) + cur.l0 + l] = t[i];
            }
            block_max<G>(t, wred);
            float mine = t[0];                        // thread l < G writes head l's maximum
#pragma unroll
            for (int i = 1; i < G; ++i) mine = (l == i) ? t[i] : mine;
            if (l < G) a.segmax[((int64_t)cur.b * a.H + h0 + l) * a.J + cur.j] = mine;
        }
    }
}

// 1'. the same scores with 128 threads per workgroup, thread l holding positions
// l and l + 128 (head dims 64, 128, 256; 32-column key steps).  Each q value
// (read with uniform loads) then feeds two FMAs per thread, which halves the
// scalar-load traffic per FMA of the 256-thread kernel.
template <int G, int D>
__global__ void __launch_bounds__(128) attn_scores2_kernel(AttnArgs a) {
    constexpr int DC = 32, NC = D / DC, PAD = DC + 8;
    constexpr int NV = kAttnSeg * DC / 8 / 128;       // 16-byte vectors per thread per step (8)
    __shared__ __attribute__((aligned(16))) uint16_t ks[kAttnSeg * PAD];   // [256][DC + 8]
    __shared__ float wred[2][G];
    const int tid = threadIdx.x;
    const int items = (int)(a.B * a.Hkv * a.J);
    cfloat* q4 = (cfloat*)a.q;
    uint4 kr[NV];
    auto fetch = [&](const Item& w, int c) {
        const uint16_t* src = a.k + (((int64_t)w.b * a.Hkv + w.g) * a.Lmax + w.l0) * D + c * DC;
#pragma unroll
        for (int u = 0; u < NV; ++u) {
            const int i = tid + 128 * u;               // vector i: row i / 4, columns 8 (i % 4)
            const int row = i >> 2;
            // a normal load: each pass reads 64 bytes of a row whose other bytes the next
            // passes read (non-temporal here measured slower on the 70B-shaped heads)
            kr[u] = row < w.rows ? *reinterpret_cast<const uint4*>(src + (int64_t)row * D + 8 * (i & 3))
                                 : make_uint4(0u, 0u, 0u, 0u);
        }
    };
    int it = next_item(a, (int)blockIdx.x, items);
    Item w;
    int c = 0;
    if (it < items) {
        w = item_of(a, it);
        fetch(w, 0);
    }
    float z0[G], z1[G];
    while (it < items) {
        __syncthreads();                              // the previous step's reads of LDS are done
#pragma unroll
        for (int u = 0; u < NV; ++u) {
            const int i = tid + 128 * u;
            *reinterpret_cast<uint4*>(ks + (i >> 2) * PAD + 8 * (i & 3)) = kr[u];
        }
        __syncthreads();
        const Item cur = w;
        const int cc = c;
        if (c + 1 < NC) {
            ++c;
        } else {
            c = 0;
            it = next_item(a, it + (int)gridDim.x, items);
            if (it < items) w = item_of(a, it);
        }
        if (it < items) fetch(w, c);                  // in flight during this step's chains
        if (cc == 0) {
#pragma unroll
            for (int i = 0; i < G; ++i) z0[i] = z1[i] = 0.0f;
        }
        const int64_t h0 = (int64_t)cur.g * G;
        const int64_t qbase = ((int64_t)cur.b * a.H + h0) * D + cc * DC;
        const uint16_t* kp0 = ks + tid * PAD;
        const uint16_t* kp1 = ks + (tid + 128) * PAD;
#pragma unroll 1
        for (int d = 0; d < DC; d += 8) {
            const uint4 k0 = *reinterpret_cast<const uint4*>(kp0 + d);
            const uint4 k1 = *reinterpret_cast<const uint4*>(kp1 + d);
            const uint32_t a4[4] = {k0.x, k0.y, k0.z, k0.w}, b4[4] = {k1.x, k1.y, k1.z, k1.w};
            float f0[8], f1[8];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                f0[2 * e] = __uint_as_float(a4[e] << 16);
                f0[2 * e + 1] = __uint_as_float(a4[e] & 0xffff0000u);
                f1[2 * e] = __uint_as_float(b4[e] << 16);
                f1[2 * e + 1] = __uint_as_float(b4[e] & 0xffff0000u);
            }
#pragma unroll
            for (int i = 0; i < G; ++i)
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const float qv = q4[qbase + i * D + d + e];
                    z0[i] = __builtin_fmaf(qv, f0[e], z0[i]);
                    z1[i] = __builtin_fmaf(qv, f1[e], z1[i]);
                }
        }
        if (cc == NC - 1) {
            // t for the valid positions; the segment maximum per head over them (exact)
            const int l0 = tid, l1 = tid + 128;
            float t[G];
#pragma unroll
            for (int i = 0; i < G; ++i) {
                const float t0 = l0 < cur.rows ? z0[i] * a.scale : -__builtin_inff();
                const float t1 = l1 < cur.rows ? z1[i] * a.scale : -__builtin_inff();
                float* tp = a.t + (((int64_t)cur.b * a.H + h0 + i) * a.Lmax) + cur.l0;
                if (l0 < cur.rows) tp[l0] = t0;
                if (l1 < cur.rows) tp[l1] = t1;
                t[i] = __builtin_fmaxf(t0, t1);
            }
#pragma unroll
            for (int sh = 32; sh > 0; sh >>= 1)
#pragma unroll
                for (int i = 0; i < G; ++i) t[i] = __builtin_fmaxf(t[i], __shfl_xor(t[i], sh, 64));
            if ((tid & 63) == 0) {
#pragma unroll
                for (int i = 0; i < G; ++i) wred[tid >> 6][i] = t[i];
            }
            __syncthreads();
            if (tid < G) {
                float mine = wred[0][0];
#pragma unroll
                for (int i = 0; i < G; ++i) mine = (tid == i) ? __builtin_fmaxf(wred[0][i], wred[1][i]) : mine;
                a.segmax[((int64_t)cur.b * a.H + h0 + tid) * a.J + cur.j] = mine;
            }
        }
    }
}

// 2. m[b][h] = the largest segment maximum (exact).  One thread per (b, h).
__global__ void __launch_bounds__(256) attn_max_kernel(AttnArgs a) {
    const int64_t bh = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (bh >= a.B * a.H) return;
    const int L = clamp_len(a.lens, bh / a.H, a.Lmax);
    const int Jb = (L + kAttnSeg - 1) / kAttnSeg;
    const float* sm = a.segmax + bh * a.J;
    float m = -__builtin_inff();
    int jj = 0;
    for (; jj + 8 <= Jb; jj += 8) {
        float v[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) v[i] = sm[jj + i];
#pragma unroll
        for (int i = 0; i < 8; ++i) m = __builtin_fmaxf(m, v[i]);
    }
    for (; jj < Jb; ++jj) m = __builtin_fmaxf(m, sm[jj]);
    a.mmax[bh] = m;
}

// 3. exponentials and the segment partials S_j and n_j[d].  Work item = segment;
// its NS steps take positions [l0 + s RS, l0 + s RS + RS) in turn (RS = 16384 / D
// rows for the fixed head dims, else all 256 in one step), so every chain below
// continues across the steps in ascending l.  e for the segment is computed at
// its first step into LDS ([head][position], -0 past the sequence).  Unit u =
// (head, pair of adjacent d): two fmaf chains over the positions; threads tid < G
// also run the segment sum of head tid (an addition chain).  Chains run over all
// 256 positions of the segment: past the sequence e = -0 and the values are +0,
// so a padded step is fmaf(-0, +0, n) = -0 + n = n and s + (-0) = s for every n and
// s, including a numerator that is -0 (a negative product e * v that underflows).
// (A +0 pad would turn such a -0 numerator into +0.)
template <int G, int DM, int RS, bool EXACT>
__global__ void __launch_bounds__(256) attn_partials_kernel(AttnArgs a) {
    constexpr int NS = kAttnSeg / RS;                 // steps per item
    constexpr int VPR = EXACT ? DM / 8 : 0;
    constexpr int NV = RS * DM / 8 / 256;             // vectors per thread
    constexpr int UPT = (G * DM / 2 + 255) / 256;     // units per thread
    __shared__ __attribute__((aligned(16))) float es[G * kAttnSeg];           // [G][256]
    __shared__ __attribute__((aligned(16))) uint16_t vs[RS * (DM + 8)];       // [RS][D + 8]
    const int D = EXACT ? DM : (int)a.D, tid = threadIdx.x;
    const int vpr = D / 8;
    const int items = (int)(a.B * a.Hkv * a.J);
    Tile<NV, VPR> tile;
    float tr[G], mr[G];
    auto fetch = [&](const Item& w, int s) {
        const int r0 = s * RS;
        const int rows = w.rows - r0 < RS ? w.rows - r0 : RS;
        tile.fetch(a.v + (((int64_t)w.b * a.Hkv + w.g) * a.Lmax + w.l0 + r0) * D, D, rows, vpr, a.vmagic);
        if (s == 0) {
            const int64_t h0 = (int64_t)w.g * G;
#pragma unroll
            for (int i = 0; i < G; ++i) {
                tr[i] = tid < w.rows ? a.t[((int64_t)w.b * a.H + h0 + i) * a.Lmax + w.l0 + tid] : 0.0f;
                mr[i] = a.mmax[(int64_t)w.b * a.H + h0 + i];
            }
        }
    };
    int it = next_item(a, (int)blockIdx.x, items);
    Item w;
    int st = 0;
    if (it < items) {
        w = item_of(a, it);
        fetch(w, 0);
    }
    const int npd = D / 2;
    const int nunits = G * npd;
    float n0[UPT], n1[UPT], ssum = 0.0f;
    while (it < items) {
        __syncthreads();
        tile.store(vs, RS, vpr, a.vmagic);
        if (st == 0) {
#pragma unroll
            for (int i = 0; i < G; ++i) es[i * kAttnSeg + tid] = tid < w.rows ? exp1(tr[i] - mr[i]) : -0.0f;
        }
        __syncthreads();
        const Item cur = w;
        const int ss = st;
        if (st + 1 < NS) {
            ++st;
        } else {
            st = 0;
            it = next_item(a, it + (int)gridDim.x, items);
            if (it < items) w = item_of(a, it);
        }
        if (it < items) fetch(w, st);                 // in flight during this step's chains
        if (ss == 0) {
#pragma unroll
            for (int k = 0; k < UPT; ++k) n0[k] = n1[k] = 0.0f;
            ssum = 0.0f;
        }
        const int lb = ss * RS;                        // first position of this step in the segment
#pragma unroll
        for (int k = 0; k < UPT; ++k) {
            const int u = tid + 256 * k;
            if (u < nunits) {
                const int hh = u / npd, d = 2 * (u - hh * npd);
                const bool sums = k == 0 && tid < G;
                const float* ep = es + hh * kAttnSeg + lb;
                const float* sp = es + (tid < G ? tid : 0) * kAttnSeg + lb;
                const uint16_t* vp = vs + d;
                float x0 = n0[k], x1 = n1[k], sm = ssum;
#pragma unroll 2
                for (int l = 0; l < RS; l += 8) {
                    const float4 e0 = *reinterpret_cast<const float4*>(ep + l);
                    const float4 e1 = *reinterpret_cast<const float4*>(ep + l + 4);
                    const float ev[8] = {e0.x, e0.y, e0.z, e0.w, e1.x, e1.y, e1.z, e1.w};
                    uint32_t vv[8];
#pragma unroll
                    for (int i = 0; i < 8; ++i) vv[i] = *reinterpret_cast<const uint32_t*>(vp + (l + i) * (D + 8));
#pragma unroll
                    for (int i = 0; i < 8; ++i) {
                        x0 = __builtin_fmaf(ev[i], __uint_as_float(vv[i] << 16), x0);
                        x1 = __builtin_fmaf(ev[i], __uint_as_float(vv[i] & 0xffff0000u), x1);
                    }
                    if (sums) {
                        const float4 s0 = *reinterpret_cast<const float4*>(sp + l);
                        const float4 s1 = *reinterpret_cast<const float4*>(sp + l + 4);
                        sm = sm + s0.x; sm = sm + s0.y; sm = sm + s0.z; sm = sm + s0.w;
                        sm = sm + s1.x; sm = sm + s1.y; sm = sm + s1.z; sm = sm + s1.w;
                    }
                }
                n0[k] = x0;
                n1[k] = x1;
                if (sums) ssum = sm;
                if (ss == NS - 1) {
                    float* np = a.npart + (((int64_t)cur.b * a.H + cur.g * G + hh) * a.J + cur.j) * D + d;
                    np[0] = x0;
                    np[1] = x1;
                    if (sums) a.spart[((int64_t)cur.b * a.H + cur.g * G + tid) * a.J + cur.j] = sm;
                }
            }
        }
    }
}

// 3'. the same partials with one wave per work item (head dims 128 and 256).
// Lane p owns the value columns 2p, 2p + 1 (and 2p + 128, 2p + 129 for D = 256)
// for all G query heads of the group, so a value pair is read from LDS and
// widened once and feeds 2G fmaf chains.  The item's positions are taken in
// steps of RS = 32 (D = 128) or 16 (D = 256) rows (8 KB); the wave loads the
// next step's value rows and scores into registers while it computes the
// current step, and stages them in its own LDS region (waves never wait for
// each other).  e for a step is computed into LDS as [position][head].  The
// chains run over the valid positions only (the same values as chains over the
// +0-padded segment).  INMAX: the wave takes its item's row maxima from the
// segment maxima itself (the largest one per head, exact), so the maximum kernel
// is not launched; used when no wave has more than one item.  CS = 2: the value
// columns of an item are split between two waves (columns [0, D/2) and [D/2, D)),
// each running the full chains of its columns (the same order: a chain is one
// column's sum over the positions), for grids that would otherwise hold about one
// wave per SIMD; with D = 128 a lane then owns one column.
template <int G, int D, bool INMAX, int CS>
__global__ void __launch_bounds__(256) attn_partials_wave_kernel(AttnArgs a) {
    static_assert(CS == 1 || CS == 2, "column split");
    constexpr int DH = D / CS;                         // value columns of this wave
    constexpr int RS = 4096 / DH;                      // rows per step (8 KB of bf16)
    constexpr int PPL = DH >= 128 ? DH / 128 : 0;      // value pairs per lane (0: one column)
    constexpr int GP = G <= 4 ? 4 : 8;                 // e row stride (floats)
    constexpr int NVL = RS * DH / 8 / 64;              // 16-byte vectors per lane per step (8)
    constexpr int NTL = (RS * G + 63) / 64;            // scores per lane per step
    constexpr int NC = PPL > 0 ? PPL : 1;              // chain sets per head
    __shared__ __attribute__((aligned(16))) uint16_t vs[4][RS * DH];
    __shared__ __attribute__((aligned(16))) float es[4][RS * GP];
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int items = (int)(a.B * a.Hkv * a.J);
    const int tw = (int)gridDim.x * 4 / CS;            // waves in the grid per column half
    const int gw = ((int)blockIdx.x * 4 + wave) / CS;
    const int half = ((int)blockIdx.x * 4 + wave) % CS;   // 0 for CS = 1
    uint16_t* vw = vs[wave];
    float* ew = es[wave];

    // the wave's items gw, gw + tw, ... that hold positions
    auto next = [&](int it) {
        while (it < items && item_of(a, it).rows <= 0) it += tw;
        return it;
    };
    uint4 vr[NVL];
    float tr[NTL];
    // INMAX: the first 512 of the item's G * Jb segment maxima are loaded with its first
    // step into smv and reduced before its exponentials; lane-local maxima of any further
    // values (sequences longer than 512 / G segments) are taken at once into mr.  When G
    // divides 64, lane l only ever holds values of head l % G, kept in mr[0].
    float smv[INMAX ? 8 : 1];
    float mr[G];
    auto fetch = [&](const Item& w, int s) {
        const int r0 = s * RS;
        const int nrow = min(RS, w.rows - r0);          // >= 1
        const uint16_t* vb = a.v + (((int64_t)w.b * a.Hkv + w.g) * a.Lmax + w.l0 + r0) * D + half * DH;
#pragma unroll
        for (int u = 0; u < NVL; ++u) {
            const int i = lane + 64 * u;                // vector i: row i / (DH / 8), column 8 (i % (DH / 8))
            const int row = i / (DH / 8);
            vr[u] = row < nrow ? ldnt(reinterpret_cast<const uint4*>(vb + (int64_t)row * D + 8 * (i % (DH / 8))))
                               : make_uint4(0u, 0u, 0u, 0u);
        }
        const int64_t tb = ((int64_t)w.b * a.H + (int64_t)w.g * G) * a.Lmax + w.l0 + r0;
#pragma unroll
        for (int u = 0; u < NTL; ++u) {
            const int q = lane + 64 * u;                // (position q / G, head q % G)
            const int l = q / G, h = q - l * G;
            tr[u] = (q < RS * G && l < nrow) ? a.t[tb + (int64_t)h * a.Lmax + l] : 0.0f;
        }
        if (s == 0) {
            if constexpr (INMAX) {
                const int jb = (w.L + kAttnSeg - 1) / kAttnSeg;
                const float* smb = a.segmax + ((int64_t)w.b * a.H + (int64_t)w.g * G) * a.J;   // head h at h * J
                const int snv = G * jb;
#pragma unroll
                for (int u = 0; u < 8; ++u) {
                    const int idx = lane + 64 * u;
                    smv[u] = idx < snv ? smb[(int64_t)(idx % G) * a.J + idx / G] : -__builtin_inff();
                }
#pragma unroll
                for (int h = 0; h < G; ++h) mr[h] = -__builtin_inff();
                for (int base = 512; base < snv; base += 64) {
                    const int idx = base + lane;
                    if (idx < snv) {
                        const float v = smb[(int64_t)(idx % G) * a.J + idx / G];
                        if constexpr (64 % G == 0) {
                            mr[0] = __builtin_fmaxf(mr[0], v);
                        } else {
                            const int h = idx % G;
#pragma unroll
                            for (int i = 0; i < G; ++i) mr[i] = (h == i) ? __builtin_fmaxf(mr[i], v) : mr[i];
                        }
                    }
                }
            } else {
#pragma unroll
                for (int h = 0; h < G; ++h) mr[h] = a.mmax[(int64_t)w.b * a.H + (int64_t)w.g * G + h];
            }
        }
    };

    int it = next(gw);
    if (it >= items) return;
    Item w = item_of(a, it);
    int st = 0;
    fetch(w, 0);
    float n0[NC][G], n1[NC][G], ssum = 0.0f;
    float mcur[G];
    while (it < items) {
        const Item cur = w;
        const int ss = st;
        const int nrow = min(RS, cur.rows - ss * RS);
        // stage this step: value rows and e = EXP1(t - m) for the valid positions (+0 elsewhere)
        if (ss == 0) {
            if constexpr (!INMAX) {
#pragma unroll
                for (int h = 0; h < G; ++h) mcur[h] = mr[h];
            } else if constexpr (64 % G == 0) {
                // reduce over the lanes of each head, then take head h's maximum from lane h
                float ml = mr[0];
#pragma unroll
                for (int u = 0; u < 8; ++u) ml = __builtin_fmaxf(ml, smv[u]);
#pragma unroll
                for (int sh = 32; sh >= G; sh >>= 1) ml = __builtin_fmaxf(ml, __shfl_xor(ml, sh, 64));
#pragma unroll
                for (int h = 0; h < G; ++h)
                    mcur[h] = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(ml), h));
            } else {
                float ml[G];
#pragma unroll
                for (int h = 0; h < G; ++h) ml[h] = mr[h];
#pragma unroll
                for (int u = 0; u < 8; ++u) {
                    const int h = (lane + 64 * u) % G;
#pragma unroll
                    for (int i = 0; i < G; ++i) ml[i] = (h == i) ? __builtin_fmaxf(ml[i], smv[u]) : ml[i];
                }
#pragma unroll
                for (int sh = 32; sh > 0; sh >>= 1)
#pragma unroll
                    for (int h = 0; h < G; ++h) ml[h] = __builtin_fmaxf(ml[h], __shfl_xor(ml[h], sh, 64));
#pragma unroll
                for (int h = 0; h < G; ++h) mcur[h] = ml[h];
            }
        }
#pragma unroll
        for (int u = 0; u < NVL; ++u) *reinterpret_cast<uint4*>(vw + 8 * (lane + 64 * u)) = vr[u];
#pragma unroll
        for (int u = 0; u < NTL; ++u) {
            const int q = lane + 64 * u;
            if (q < RS * G) {
                const int l = q / G, h = q - l * G;
                float mh = mcur[0];
#pragma unroll
                for (int i = 1; i < G; ++i) mh = (h == i) ? mcur[i] : mh;
                ew[l * GP + h] = l < nrow ? exp1(tr[u] - mh) : 0.0f;
            }
        }
        __builtin_amdgcn_wave_barrier();
        // next step (this item's, or the next item's first) in flight during the chains
        if (st + 1 < (cur.rows + RS - 1) / RS) {
            ++st;
        } else {
            st = 0;
            it = next(it + tw);
            if (it < items) w = item_of(a, it);
        }
        if (it < items) fetch(w, st);
        if (ss == 0) {
#pragma unroll
            for (int k = 0; k < NC; ++k)
#pragma unroll
                for (int h = 0; h < G; ++h) n0[k][h] = n1[k][h] = 0.0f;
            ssum = 0.0f;
        }
        const float* es_own = ew + (lane < G ? lane : 0);
#pragma unroll 4
        for (int l = 0; l < nrow; ++l) {
            float ev[G];
#pragma unroll
            for (int h = 0; h < G; ++h) ev[h] = ew[l * GP + h];
            if constexpr (PPL == 0) {
                // one column per lane
                const float v1 = __uint_as_float((uint32_t)vw[l * DH + lane] << 16);
#pragma unroll
                for (int h = 0; h < G; ++h) n0[0][h] = __builtin_fmaf(ev[h], v1, n0[0][h]);
            } else {
#pragma unroll
                for (int k = 0; k < PPL; ++k) {
                    const uint32_t v2 = *reinterpret_cast<const uint32_t*>(vw + l * DH + 128 * k + 2 * lane);
                    const float vlo = __uint_as_float(v2 << 16), vhi = __uint_as_float(v2 & 0xffff0000u);
#pragma unroll
                    for (int h = 0; h < G; ++h) {
                        n0[k][h] = __builtin_fmaf(ev[h], vlo, n0[k][h]);
                        n1[k][h] = __builtin_fmaf(ev[h], vhi, n1[k][h]);
                    }
                }
            }
            ssum = ssum + es_own[l * GP];               // lanes < G: head `lane`'s segment sum
        }
        if (ss == (cur.rows + RS - 1) / RS - 1) {
            const int64_t hb = (int64_t)cur.b * a.H + (int64_t)cur.g * G;
#pragma unroll
            for (int h = 0; h < G; ++h) {
                float* nb = a.npart + ((hb + h) * a.J + cur.j) * D + half * DH;
                if constexpr (PPL == 0) {
                    nb[lane] = n0[0][h];
                } else {
#pragma unroll
                    for (int k = 0; k < PPL; ++k) {
                        nb[128 * k + 2 * lane] = n0[k][h];
                        nb[128 * k + 2 * lane + 1] = n1[k][h];
                    }
                }
            }
            // (both halves sum the same e in the same order; the first writes the sums)
            if (lane < G && half == 0) a.spart[(hb + lane) * a.J + cur.j] = ssum;
        }
        __builtin_amdgcn_wave_barrier();
    }
}

// 4. out = N / S after the ascending folds of the segment partials.  Workgroup (b, h),
// thread d.
__global__ void __launch_bounds__(256) attn_fold_kernel(AttnArgs a) {
    const int64_t bh = blockIdx.x, b = bh / a.H;
    const int L = clamp_len(a.lens, b, a.Lmax);
    const int Jb = (L + kAttnSeg - 1) / kAttnSeg;
    const int D = a.D;
    const float* sp = a.spart + bh * a.J;
    for (int d = threadIdx.x; d < D; d += blockDim.x) {
        const float* np = a.npart + bh * a.J * D + d;
        float S = 0.0f, N = 0.0f;
        int jj = 0;
        for (; jj + 32 <= Jb; jj += 32) {          // loads issued in groups, additions in order
            float sv[32], nv[32];
#pragma unroll
            for (int i = 0; i < 32; ++i) {
                sv[i] = sp[jj + i];
                nv[i] = np[(int64_t)(jj + i) * D];
            }
#pragma unroll
            for (int i = 0; i < 32; ++i) {
                S = (jj + i == 0) ? sv[i] : S + sv[i];
                N = (jj + i == 0) ? nv[i] : N + nv[i];
            }
        }
        for (; jj + 8 <= Jb; jj += 8) {
            float sv[8], nv[8];
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                sv[i] = sp[jj + i];
                nv[i] = np[(int64_t)(jj + i) * D];
            }
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                S = (jj + i == 0) ? sv[i] : S + sv[i];
                N = (jj + i == 0) ? nv[i] : N + nv[i];
            }
        }
        for (; jj < Jb; ++jj) {
            S = (jj == 0) ? sp[0] : S + sp[jj];
            N = (jj == 0) ? np[0] : N + np[(int64_t)jj * D];
        }
        a.out[bh * D + d] = N / S;
    }
}

// Workgroups each kernel keeps resident per CU: LDS-limited (160 KB per CU).
constexpr int64_t kLdsPerCU = 160 * 1024;

// Persistent grids: as many workgroups as the LDS of the device keeps resident.
template <typename K1, typename K3>
hipError_t launch_pair(K1 k1, int64_t lds1, K3 k3, int64_t lds3, const AttnArgs& a, int cus, hipStream_t stream) {
    const int64_t items = a.B * a.Hkv * a.J;
    const int64_t g1 = items < (kLdsPerCU / lds1) * cus ? items : (kLdsPerCU / lds1) * cus;
    const int64_t g3 = items < (kLdsPerCU / lds3) * cus ? items : (kLdsPerCU / lds3) * cus;
    hipLaunchKernelGGL(k1, dim3((unsigned)g1), dim3(256), 0, stream, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(attn_max_kernel, dim3((unsigned)((a.B * a.H + 255) / 256)), dim3(256), 0, stream, a);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k3, dim3((unsigned)g3), dim3(256), 0, stream, a);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(attn_fold_kernel, dim3((unsigned)(a.B * a.H)), dim3(256), 0, stream, a);
    return hipGetLastError();
}

// Fixed head dims (64, 128, 256).  Scores: 64-column key steps (32 KB tiles, four
// workgroups per CU); with eight query heads per kv head the two-positions-per-
// thread kernel (32-column steps, 128 threads, about 20 KB of LDS; measured
// 111 -> 90 us for the scores of a 32 x 64-head, 4096-position batch, and 0-22 %
// slower than the 64-column kernel with six or fewer heads).  Partials: one wave per
// work item for D = 128 and 256 (four 4-wave workgroups per CU, each wave walking
// items gw, gw + waves, ...), two waves per item (value columns split) when there
// are at most four items per CU (one 32K-token sequence: the pass 21.0 -> 20.3 us,
// the call level within its spread); for D = 64 the workgroup-per-item kernel with
// 16384 / D-row value steps (32 KB tiles, four workgroups per CU).  Other D <= DM:
// launch_any.
template <int G, int D>
hipError_t launch_fixed(const AttnArgs& a, int cus, hipStream_t stream) {
    constexpr int RS = 16384 / D;
    const int64_t items = a.B * a.Hkv * a.J;
    if constexpr (G == 8) {
        const int64_t lds1 = (int64_t)kAttnSeg * (32 + 8) * 2 + 8 * G;
        const int64_t g1 = items < (kLdsPerCU / lds1) * cus ? items : (kLdsPerCU / lds1) * cus;
        hipLaunchKernelGGL((attn_scores2_kernel<G, D>), dim3((unsigned)g1), dim3(128), 0, stream, a);
    } else {
        const int64_t lds1 = (int64_t)kAttnSeg * (64 + 8) * 2 + 16 * G;
        const int64_t g1 = items < (kLdsPerCU / lds1) * cus ? items : (kLdsPerCU / lds1) * cus;
        hipLaunchKernelGGL((attn_scores_kernel<G, 64, D / 64, true>), dim3((unsigned)g1), dim3(256), 0, stream, a);
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    // partials of head dims 128 and 256: one wave per item; when no wave has more than one
    // item the waves take the row maxima themselves and the maximum kernel is not launched
    // (measured 1-8 % faster with up to six query heads per kv head, 1 % slower with eight)
    constexpr bool kInmax = (D == 128 || D == 256) && G < 8;
    // at most one item per SIMD (one long sequence, say): each item's value columns are
    // split between two waves
    const int cs = (D == 128 || D == 256) && items <= 4 * (int64_t)cus ? 2 : 1;
    const int64_t gw = (cs * items + 3) / 4 < 4 * (int64_t)cus ? (cs * items + 3) / 4 : 4 * (int64_t)cus;
    const bool inmax = kInmax && cs * items <= 4 * gw;
    if (!inmax) {
        hipLaunchKernelGGL(attn_max_kernel, dim3((unsigned)((a.B * a.H + 255) / 256)), dim3(256), 0, stream, a);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    if constexpr (D == 128 || D == 256) {
        bool launched = false;
        if constexpr (kInmax) {
            if (inmax) {
                if (cs == 2)
                    hipLaunchKernelGGL((attn_partials_wave_kernel<G, D, true, 2>), dim3((unsigned)gw), dim3(256), 0,
                                       stream, a);
                else
                    hipLaunchKernelGGL((attn_partials_wave_kernel<G, D, true, 1>), dim3((unsigned)gw), dim3(256), 0,
                                       stream, a);
                launched = true;
            }
        }
        if (!launched) {
            if (cs == 2)
                hipLaunchKernelGGL((attn_partials_wave_kernel<G, D, false, 2>), dim3((unsigned)gw), dim3(256), 0, stream,
                                   a);
            else
                hipLaunchKernelGGL((attn_partials_wave_kernel<G, D, false, 1>), dim3((unsigned)gw), dim3(256), 0, stream,
                                   a);
        }
    } else {
        const int64_t lds3 = (int64_t)G * kAttnSeg * 4 + (int64_t)RS * (D + 8) * 2;
        const int64_t g3 = items < (kLdsPerCU / lds3) * cus ? items : (kLdsPerCU / lds3) * cus;
        hipLaunchKernelGGL((attn_partials_kernel<G, D, RS, true>), dim3((unsigned)g3), dim3(256), 0, stream, a);
    }
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(attn_fold_kernel, dim3((unsigned)(a.B * a.H)), dim3(256), 0, stream, a);
    return hipGetLastError();
}

template <int G, int DM>
hipError_t launch_any(const AttnArgs& a, int cus, hipStream_t stream) {
    const int64_t lds1 = (int64_t)kAttnSeg * (DM + 8) * 2 + 16 * G;
    const int64_t lds3 = (int64_t)G * kAttnSeg * 4 + (int64_t)kAttnSeg * (DM + 8) * 2;
    return launch_pair(attn_scores_kernel<G, DM, 1, false>, lds1, attn_partials_kernel<G, DM, kAttnSeg, false>, lds3,
                       a, cus, stream);
}

template <int G>
hipError_t launch_dm(const AttnArgs& a, int cus, hipStream_t stream) {
    if (a.D == 64) return launch_fixed<G, 64>(a, cus, stream);
    if (a.D == 128) return launch_fixed<G, 128>(a, cus, stream);
    if (a.D == 256) return launch_fixed<G, 256>(a, cus, stream);
    if (a.D <= 64) return launch_any<G, 64>(a, cus, stream);
    if (a.D <= 128) return launch_any<G, 128>(a, cus, stream);
    return launch_any<G, 256>(a, cus, stream);
}

}  // namespace

hipError_t launch_attn(const AttnArgs& a, int cus, hipStream_t stream) {
    if (cus < 1) cus = 1;
    if (a.D < 8 || a.D > 256 || a.D % 8 != 0 || a.Hkv < 1 || a.H % a.Hkv != 0) return hipErrorInvalidValue;
    switch (a.H / a.Hkv) {
        case 1: return launch_dm<1>(a, cus, stream);
        case 2: return launch_dm<2>(a, cus, stream);
        case 3: return launch_dm<3>(a, cus, stream);
        case 4: return launch_dm<4>(a, cus, stream);
        case 5: return launch_dm<5>(a, cus, stream);
        case 6: return launch_dm<6>(a, cus, stream);
        case 7: return launch_dm<7>(a, cus, stream);
        case 8: return launch_dm<8>(a, cus, stream);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace rg
