// Fused-upcast linear layer kernels for gfx950 (MI355X).
//
// Every kernel here computes y[m][n] = sum_k x[m][k] * up(W[n][k]) (+ b[n]) in the one
// order documented in include/rg.h ("RG-ORDER-1"): 256-wide K segments, each a
// chain of fmaf from +0 in ascending k, segment partials folded left to right
// in ascending segment order (paper: Design, eq. 2 and rules R1-R4).  Kernels
// differ only in how outputs are spread over lanes, waves and workgroups,
// which never changes a bit of any output.
//
// Arithmetic: only v_fma_f32 / v_fmac_f32 (IEEE fused) and v_add_f32, with
// binary32 denormals preserved (the kernel descriptors keep
// float_denorm_mode_32 = 3).  No matrix-core (MFMA) or dot-product
// instructions; the library is built with -ffp-contract=off and packed FP32
// disabled, so the compiler cannot fuse, reassociate or pair operations.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "rg_kernels.h"

namespace rg {

// ---------------------------------------------------------------------------
// helpers
// ---------------------------------------------------------------------------

// Exact bfloat16 -> float32 widening of the low / high half of a packed dword
// (element k at the lower address sits in the low 16 bits).
__device__ __forceinline__ float up_lo(uint32_t v) { return __uint_as_float(v << 16); }
__device__ __forceinline__ float up_hi(uint32_t v) { return __uint_as_float(v & 0xffff0000u); }
__device__ __forceinline__ float up1(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

// Weight element types.  bfloat16 bit patterns are widened exactly (up1 and
// friends); float32 weights (the FP32-weight variant) are used as they are.
// A 16-byte vector load carries E elements.
__device__ __forceinline__ float wval(uint16_t b) { return up1(b); }
__device__ __forceinline__ float wval(float f) { return f; }

template <typename WT>
struct WVec;
template <>
struct WVec<uint16_t> {
    using V = uint4;
    static constexpr int E = 8;
    static __device__ __forceinline__ V zero() { return make_uint4(0u, 0u, 0u, 0u); }
    static __device__ __forceinline__ V neg_zero() {   // every element bf16 -0 (0x8000)
        return make_uint4(0x80008000u, 0x80008000u, 0x80008000u, 0x80008000u);
    }
    static __device__ __forceinline__ float get(const V& v, int h) {
        const uint32_t d[4] = {v.x, v.y, v.z, v.w};
        return (h & 1) ? up_hi(d[h >> 1]) : up_lo(d[h >> 1]);
    }
};
template <>
struct WVec<float> {
    using V = float4;
    static constexpr int E = 4;
    static __device__ __forceinline__ V zero() { return make_float4(0.f, 0.f, 0.f, 0.f); }
    static __device__ __forceinline__ V neg_zero() { return make_float4(-0.f, -0.f, -0.f, -0.f); }
    static __device__ __forceinline__ float get(const V& v, int h) {
        const float d[4] = {v.x, v.y, v.z, v.w};
        return d[h];
    }
};

// A 16-byte load marked non-temporal: for weights that are read once (the caches need
// not keep them, and x, which every workgroup reads, stays resident).
template <typename V>
__device__ __forceinline__ V load_nt(const V* p) {
    static_assert(sizeof(V) == 16, "16-byte vector");
    using E = __attribute__((ext_vector_type(4))) uint32_t;
    const E e = __builtin_nontemporal_load(reinterpret_cast<const E*>(p));
    V v;
    __builtin_memcpy(&v, &e, sizeof v);
    return v;
}

// Broadcast lane E of every quad (4 lanes) to the whole quad (DPP quad_perm).
template <int E>
__device__ __forceinline__ float quad_bcast(float v) {
    constexpr int ctrl = E | (E << 2) | (E << 4) | (E << 6);
    return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), ctrl, 0xf, 0xf, true));
}


// acc = fmaf(x[quad lane E], w[h], acc) for h = 0..7 in order, with the x
// broadcast fused into the FMA (v_fmac_f32_dpp, DPP on the x operand).  The
// leading s_nop covers the two wait states a DPP read needs after a VALU
// write of its source.  Each v_fmac is one IEEE-754 binary32 fused
// multiply-add; the DPP modifier only selects which lane's x is read.
template <int E>
__device__ __forceinline__ void fmac8_bcast(float& acc, const float* x, const float* w) {
    asm("s_nop 1\n\t"
        "v_fmac_f32_dpp %0, %1, %9 quad_perm:[%17,%17,%17,%17] row_mask:0xf bank_mask:0xf bound_ctrl:1\n\t"
        "v_fmac_f32_dpp %0, %2, %10 quad_perm:[%17,%17,%17,%17] row_mask:0xf bank_mask:0xf bound_ctrl:1\n\t"
        "v_fmac_f32_dpp %0, %3, %11 quad_perm:[%17,%17,%17,%17] row_mask:0xf bank_mask:0xf bound_ctrl:1\n\t"
        "v_fmac_f32_dpp %0, %4, %12 quad_perm:[%17,%17,%17,%17] row_mask:0xf bank_mask:0xf bound_ctrl:1\n\t"
        "v_fmac_f32_dpp %0, %5, %13 quad_perm:[%17,%17,%17,%17] row_mask:0xf bank_mask:0xf bound_ctrl:1\n\t"
        "v_fmac_f32_dpp %0, %6, %14 quad_perm:[%17,%17,%17,%17] row_mask:0xf bank_mask:0xf bound_ctrl:1\n\t"
        "v_fmac_f32_dpp %0, %7, %15 quad_perm:[%17,%17,%17,%17] row_mask:0xf bank_mask:0xf bound_ctrl:1\n\t"
        "v_fmac_f32_dpp %0, %8, %16 quad_perm:[%17,%17,%17,%17] row_mask:0xf bank_mask:0xf bound_ctrl:1"
        : "+v"(acc)
        : "v"(x[0]), "v"(x[1]), "v"(x[2]), "v"(x[3]), "v"(x[4]), "v"(x[5]), "v"(x[6]), "v"(x[7]),
          "v"(w[0]), "v"(w[1]), "v"(w[2]), "v"(w[3]), "v"(w[4]), "v"(w[5]), "v"(w[6]), "v"(w[7]), "n"(E));
}

// Four independent chains at once: for h = h0 .. h0+3, for m = 0..3:
// acc[m] = fmaf(x_m[quad lane E][h], w[h], acc[m]).  Interleaving the four
// accumulators keeps consecutive FMAs independent (each chain still sees its
// own FMAs in ascending h), so the VALU does not stall on the previous result.
template <int E>
__device__ __forceinline__ void fmac4x4_bcast(float (&acc)[4], const float* x0, const float* x1, const float* x2,
                                              const float* x3, const float* w) {
#define RG_F(A, X, W) "v_fmac_f32_dpp %" #A ", %" #X ", %" #W " quad_perm:[%24,%24,%24,%24] row_mask:0xf bank_mask:0xf bound_ctrl:1\n\t"
    asm("s_nop 1\n\t"
        RG_F(0, 4, 20) RG_F(1, 8, 20) RG_F(2, 12, 20) RG_F(3, 16, 20)
        RG_F(0, 5, 21) RG_F(1, 9, 21) RG_F(2, 13, 21) RG_F(3, 17, 21)
        RG_F(0, 6, 22) RG_F(1, 10, 22) RG_F(2, 14, 22) RG_F(3, 18, 22)
        RG_F(0, 7, 23) RG_F(1, 11, 23) RG_F(2, 15, 23) RG_F(3, 19, 23)
        : "+v"(acc[0]), "+v"(acc[1]), "+v"(acc[2]), "+v"(acc[3])
        : "v"(x0[0]), "v"(x0[1]), "v"(x0[2]), "v"(x0[3]), "v"(x1[0]), "v"(x1[1]), "v"(x1[2]), "v"(x1[3]),
          "v"(x2[0]), "v"(x2[1]), "v"(x2[2]), "v"(x2[3]), "v"(x3[0]), "v"(x3[1]), "v"(x3[2]), "v"(x3[3]),
          "v"(w[0]), "v"(w[1]), "v"(w[2]), "v"(w[3]), "n"(E));
#undef RG_F
}

__device__ __forceinline__ uint32_t lds_addr(const void* p) {
    return (uint32_t)(uintptr_t)((const __attribute__((address_space(3))) void*)p);
}

// 16-byte global -> LDS DMA.  Lane l writes LDS bytes [lds_base + 16*l, +16).
// Issued through inline asm so the compiler does not add its conservative
// vmcnt(0) before every LDS read; the kernel waits with vmcnt_wait<N>().
// M0 (which holds the LDS address for the DMA and is read when the
// instruction issues) is saved and restored around it.  On this generation an
// LDS DMA must not read M0 in the cycle after a scalar write of M0 (one wait
// state, which the compiler inserts for its own DMA but cannot see inside
// inline asm): the s_nop provides it.  NT: the weight stream, whose bytes are
// read once, is loaded non-temporal (the caches need not keep it, and x, which
// every workgroup reads, stays resident); x itself is loaded normally.
template <bool NT = false>
__device__ __forceinline__ void dma16(const void* sbase, uint32_t voff, uint32_t lds_base) {
    uint32_t saved;
    if constexpr (NT) {
        asm volatile(
            "s_mov_b32 %0, m0\n\t"
            "s_mov_b32 m0, %2\n\t"
            "s_nop 0\n\t"
            "global_load_lds_dwordx4 %1, %3 nt\n\t"
            "s_mov_b32 m0, %0\n\t"
            : "=&s"(saved)
            : "v"(voff), "s"(lds_base), "s"(sbase)
            : "memory");
    } else {
        asm volatile(
            "s_mov_b32 %0, m0\n\t"
            "s_mov_b32 m0, %2\n\t"
            "s_nop 0\n\t"
            "global_load_lds_dwordx4 %1, %3\n\t"
            "s_mov_b32 m0, %0\n\t"
            : "=&s"(saved)
            : "v"(voff), "s"(lds_base), "s"(sbase)
            : "memory");
    }
}

// Eight DMA instructions into LDS [lds_base + 1024 t, + 1024), t = 0..7, from
// sbase + vo[t]: the skinny kernel's step with no clamping (whole row group, whole
// segments), with no vector instruction spent on addresses (vo[] is loop-invariant).
// Same M0 handling as dma16; NT as there.  (The instruction's immediate offset is
// not used: it would move the LDS destination as well.)
template <bool NT>
__device__ __forceinline__ void dma8(const void* sbase, const uint32_t (&vo)[8], uint32_t lds_base) {
#define RG_DMA8(P)                                                                                          \
    asm volatile("s_mov_b32 %0, m0\n\t"                                                                    \
                 "s_mov_b32 m0, %9\n\t"                                                                    \
                 "s_nop 0\n\t"                                                                             \
                 "global_load_lds_dwordx4 %1, %10" P "\n\t"                                                 \
                 "s_add_u32 m0, m0, 0x400\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %2, %10" P "\n\t"         \
                 "s_add_u32 m0, m0, 0x400\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %3, %10" P "\n\t"         \
                 "s_add_u32 m0, m0, 0x400\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %4, %10" P "\n\t"         \
                 "s_add_u32 m0, m0, 0x400\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %5, %10" P "\n\t"         \
                 "s_add_u32 m0, m0, 0x400\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %6, %10" P "\n\t"         \
                 "s_add_u32 m0, m0, 0x400\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %7, %10" P "\n\t"         \
                 "s_add_u32 m0, m0, 0x400\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %8, %10" P "\n\t"         \
                 "s_mov_b32 m0, %0\n\t"                                                                    \
                 : "=&s"(saved)                                                                             \
                 : "v"(vo[0]), "v"(vo[1]), "v"(vo[2]), "v"(vo[3]), "v"(vo[4]), "v"(vo[5]), "v"(vo[6]),     \
                   "v"(vo[7]), "s"(lds_base), "s"(sbase)                                                    \
                 : "memory", "scc")
    uint32_t saved;
    if constexpr (NT) RG_DMA8(" nt");
    else RG_DMA8("");
#undef RG_DMA8
}

// Wait until at most N vector-memory operations of this wave are outstanding.
// Used only while the outstanding operations are all global->LDS DMA loads of
// this wave, which complete in issue order among themselves.
template <int N>
__device__ __forceinline__ void vmcnt_wait() {
    static_assert(N >= 0 && N <= 63, "vmcnt range");
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}


// n / J and n % J for small n (n < 2^16) without a runtime divide: the host
// passes jmagic = ceil(2^32 / J), exact for n < 2^32 / J (J = 1 handled apart).
__device__ __forceinline__ int div_j(int n, int J, uint32_t jmagic) {
    return J == 1 ? n : (int)__umulhi((uint32_t)n, jmagic);
}

// Left fold of one output's J segment partials p[0..J-1] (contiguous floats in
// LDS): ((p0 + p1) + p2) + ...  The reads are issued in groups ahead of the
// additions; the additions stay in ascending order.
__device__ __forceinline__ float fold_partials(const float* p, int J) {
    float y = p[0];
    int j = 1;
    for (; j + 16 <= J; j += 16) {
        float v[16];
#pragma unroll
        for (int u = 0; u < 16; ++u) v[u] = p[j + u];
#pragma unroll
        for (int u = 0; u < 16; ++u) y = y + v[u];
    }
    for (; j < J; ++j) y = y + p[j];
    return y;
}

// ---------------------------------------------------------------------------
// generic kernel: one thread per output, any K, any alignment.
// ---------------------------------------------------------------------------
template <typename WT>
__global__ void __launch_bounds__(256) generic_kernel(const float* __restrict__ x,
                                                      const WT* __restrict__ w,
                                                      const float* __restrict__ bias, float* __restrict__ y, int64_t M, int64_t N,
                                                      int64_t K, int reverse) {
    const int64_t total = M * N;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    const int64_t b = reverse ? (int64_t)(gridDim.x - 1 - blockIdx.x) : (int64_t)blockIdx.x;
    for (int64_t idx = b * blockDim.x + threadIdx.x; idx < total; idx += stride) {
        const int64_t m = idx / N, n = idx % N;
        const float* xr = x + m * K;
        const WT* wr = w + n * K;
        float acc = 0.0f;
        for (int64_t k0 = 0, j = 0; k0 < K; k0 += kChunk, ++j) {
            const int64_t k1 = (k0 + kChunk < K) ? k0 + kChunk : K;
            float p = 0.0f;
            for (int64_t k = k0; k < k1; ++k) p = __builtin_fmaf(xr[k], wval(wr[k]), p);
            acc = (j == 0) ? p : acc + p;
        }
        y[m * N + n] = bias ? acc + bias[n] : acc;   // the bias: one more rounding after the fold
    }
}

// First quad of each round of a workgroup in the decode kernels.  The Q quads
// are split over G workgroups as evenly as possible (qb = Q / G each, one more
// for the first qr = Q % G) and taken RQ at a time.  Contiguous placement:
// each workgroup owns one range of quads.  Round-major placement: the quads
// all workgroups take in round r form one contiguous window [T(r), T(r+1)),
// in workgroup order, where T(r) counts the quads taken in the rounds before
// r, so at any moment the grid streams neighbouring rows of W rather than G
// ranges far apart (measured faster for one or two rows of x, slower for four).
// In round-major placement every round before r_full = qb / RQ is full for
// every workgroup (round r starts at (r G + g) RQ), and a workgroup has at
// most r_full + 1 rounds, so only round r_full needs the general count.
template <bool RM>
struct QuadPlace {
    int64_t base, step;   // rounds r < r_full start at base + r * step (every round when !RM)
    int r_full;
    int64_t last;         // first quad of round r_full (RM)
    __device__ int64_t start(int r) const {
        if constexpr (!RM) return base + (int64_t)r * step;
        else return r < r_full ? base + (int64_t)r * step : last;
    }
};

template <bool RM>
__device__ __forceinline__ QuadPlace<RM> quad_place(int g, int G, int64_t qb, int qr, int RQ) {
    QuadPlace<RM> p;
    if constexpr (!RM) {
        p.base = (int64_t)g * qb + min(g, qr);
        p.step = RQ;
        p.r_full = 0;
        p.last = 0;
    } else {
        p.base = (int64_t)g * RQ;
        p.step = (int64_t)G * RQ;
        p.r_full = (int)(qb / RQ);
        const int64_t done = (int64_t)p.r_full * RQ;                          // quads a workgroup took before
        const int64_t c1 = min((int64_t)RQ, max((int64_t)0, qb + 1 - done));  // taken in round r_full by g < qr
        const int64_t c0 = min((int64_t)RQ, max((int64_t)0, qb - done));      // ... and by the others
        const int64_t before = (int64_t)qr * min(qb + 1, done) + (int64_t)(G - qr) * min(qb, done);
        p.last = before + (int64_t)min(g, qr) * c1 + (int64_t)max(0, g - qr) * c0;
    }
    return p;
}

// Global row of staged result row o (rows of the workgroup in round order).
template <bool RM>
__device__ __forceinline__ int64_t staged_row(const QuadPlace<RM>& p, int o, int RQ) {
    if constexpr (!RM) return 4 * p.base + o;   // one contiguous range
    else {
        const int r = o / (4 * RQ);
        return 4 * p.start(r) + (o - 4 * RQ * r);
    }
}

// ---------------------------------------------------------------------------
// decode kernel (M <= MT <= 4): streaming GEMV / skinny GEMM.
//
// Work split.  Rows of W are grouped in quads (4 rows).  Workgroup g owns a
// balanced share of the quads and all of K for them, so every output is
// finished inside one workgroup (no cross-workgroup traffic, no atomics).
// It walks its quads in rounds of RQ quads, placed contiguously or
// round-major over the grid (quad_place).  In a round every lane owns one
// (row, segment) pair: the 4 lanes of a DPP quad hold 4 consecutive rows and
// one segment j; the lane roles (quad-in-round, j, row-in-quad) are fixed for
// the whole kernel, so each lane keeps x of its segment in registers.
//
// Data path.  A wave streams W in steps of one 64-element slab (128 bytes per
// lane, 8 KB per wave) through a DEPTH-deep ring of LDS buffers with 16-byte
// global->LDS DMA loads: 8 lanes read one 128-byte line, so every load
// instruction is fully coalesced.  The LDS image of lane s's 128 bytes is
// XOR-swizzled by ((s >> 1) & 7) in 16-byte units, so the transposing
// ds_read_b128 of each lane (its own row, ascending k) is conflict-free.
// x values are shared inside a quad with DPP quad broadcasts.
//
// Order.  Each lane runs the 256-FMA chain of its (row, segment) from +0 in
// ascending k; partials go to LDS; after the round one thread per output
// folds them in ascending segment order.  Results are staged in LDS and
// written once the W stream has drained.
// ---------------------------------------------------------------------------

// One 64-element slab of a lane's chain: acc[m] = fmaf(x, up(w), acc[m]) for
// the slab's elements in ascending k.  wp holds the lane's 8 pieces of 8 bf16;
// X[m][S][i] holds x for element 16*e + i of the slab in quad lane e.
// FULL: all 8 pieces present (no per-piece test, so the compiler keeps all
// LDS reads in flight together); otherwise the first npieces pieces.
template <int S, int MT, bool FULL>
__device__ __forceinline__ void fma_slab(const uint4 (&wp)[8], const float (&X)[MT][4][16], float (&acc)[MT],
                                         int npieces) {
    if constexpr (FULL) {
#pragma unroll
        for (int t = 0; t < 8; ++t) {
            const uint32_t d[4] = {wp[t].x, wp[t].y, wp[t].z, wp[t].w};
            float wv[8];
#pragma unroll
            for (int h = 0; h < 8; ++h) wv[h] = (h & 1) ? up_hi(d[h >> 1]) : up_lo(d[h >> 1]);
            if constexpr (MT == 4) {
                // the four rows' chains interleaved, 4 elements at a time
#pragma unroll
                for (int hh = 0; hh < 8; hh += 4) {
                    const int o = 8 * (t & 1) + hh;
                    switch (t >> 1) {
                        case 0: fmac4x4_bcast<0>(acc, &X[0][S][o], &X[1][S][o], &X[2][S][o], &X[3][S][o], &wv[hh]); break;
                        case 1: fmac4x4_bcast<1>(acc, &X[0][S][o], &X[1][S][o], &X[2][S][o], &X[3][S][o], &wv[hh]); break;
                        case 2: fmac4x4_bcast<2>(acc, &X[0][S][o], &X[1][S][o], &X[2][S][o], &X[3][S][o], &wv[hh]); break;
                        default: fmac4x4_bcast<3>(acc, &X[0][S][o], &X[1][S][o], &X[2][S][o], &X[3][S][o], &wv[hh]); break;
                    }
                }
            } else {
#pragma unroll
                for (int m = 0; m < MT; ++m) {
                    const float* xb = &X[m][S][8 * (t & 1)];
                    switch (t >> 1) {
                        case 0: fmac8_bcast<0>(acc[m], xb, wv); break;
                        case 1: fmac8_bcast<1>(acc[m], xb, wv); break;
                        case 2: fmac8_bcast<2>(acc[m], xb, wv); break;
                        default: fmac8_bcast<3>(acc[m], xb, wv); break;
                    }
                }
            }
        }
        return;
    }
#pragma unroll
    for (int t = 0; t < 8; ++t) {
        if (!FULL && t >= npieces) break;   // short last segment only
        const uint32_t d[4] = {wp[t].x, wp[t].y, wp[t].z, wp[t].w};
#pragma unroll
        for (int h = 0; h < 8; ++h) {
            const float wv = (h & 1) ? up_hi(d[h >> 1]) : up_lo(d[h >> 1]);
            const int kl = 8 * t + h;          // element inside the slab
            const int i = kl & 15;             // register inside the x block
#pragma unroll
            for (int m = 0; m < MT; ++m) {
                float xv;
                switch (kl >> 4) {             // lane of the quad holding x
                    case 0: xv = quad_bcast<0>(X[m][S][i]); break;
                    case 1: xv = quad_bcast<1>(X[m][S][i]); break;
                    case 2: xv = quad_bcast<2>(X[m][S][i]); break;
                    default: xv = quad_bcast<3>(X[m][S][i]); break;
                }
                acc[m] = __builtin_fmaf(xv, wv, acc[m]);
            }
        }
    }
}

constexpr int kSlab = 64;                    // elements per lane per step
constexpr int kSlabBytesPerWave = 64 * 128;  // 8 KB

template <int MT, int NW, int DEPTH, bool RM>
__global__ void __launch_bounds__(NW * 64, 1) decode_kernel(DecodeArgs a) {
    static_assert(MT == 1 || MT == 2 || MT == 4, "decode M tile");
    static_assert(DEPTH >= 2 && DEPTH <= 3, "pipeline depth");
    constexpr int kThreads = NW * 64;

    __shared__ __attribute__((aligned(16))) uint8_t wring[NW][DEPTH][kSlabBytesPerWave];
    __shared__ float part[2][kThreads * MT];          // [parity][m][row_local * J + j]
    extern __shared__ float yres[];                   // [row_in_wg][m], dynamic

    const int tid = threadIdx.x;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int lane = tid & 63;
    const int J = a.J;
    const int RQ = a.RQ;
    const int64_t N = a.N, K = a.K;

    // Row groups g (a.groups of them) x row slices of x (MT rows each).  The
    // slices of one row group sit 8 workgroups apart, so they are dispatched
    // to the same XCD at about the same time and share its L2 for W.
    int g, slice;
    {
        const int b = (int)blockIdx.x;
        const int S = a.mslices;
        slice = (b >> 3) % S;
        g = ((b >> 3) / S) * 8 + (b & 7);
        if (g >= a.groups) return;                         // padding workgroup: no work
        if (a.reverse) g = a.groups - 1 - g;
    }
    const float* xg = a.x + (int64_t)slice * MT * K;       // this slice's rows of x
    float* yg = a.y + (int64_t)slice * MT * N;
    const int64_t Ms = a.M - (int64_t)slice * MT;           // rows of x in this slice (>= 1)
    // balanced split of the Q quads over the row groups (the first qrem take one more)
    const int nq = (int)a.qbase + (g < a.qrem ? 1 : 0);
    const QuadPlace<RM> place = quad_place<RM>(g, a.groups, a.qbase, a.qrem, RQ);
    const int rounds = (nq + RQ - 1) / RQ;
    const int nsteps = rounds * (kChunk / kSlab);

    // ---- fixed lane role (consumer) ----
    const int ql = tid >> 2;                 // quad lane in the workgroup
    const int e = tid & 3;                   // row inside the quad
    const bool role = ql < RQ * J;
    const int lq = role ? div_j(ql, J, a.jmagic) : 0;   // quad inside the round
    const int jj = role ? ql - lq * J : 0;              // segment
    const int seg_len = (jj == J - 1) ? (int)(K - (int64_t)(J - 1) * kChunk) : kChunk;

    // ---- x of this lane's segment, resident in registers ----
    // X[m][s][i] = x[m][jj*256 + 64 s + 16 e + i] (0 beyond K or M).  These are
    // ordinary compiler-tracked loads: the compiler waits for them with
    // vmcnt(0) before their first use.  (A partial vmcnt wait must never be
    // relied on for them: loads returning to registers and global->LDS DMA
    // loads are not guaranteed to complete in issue order with each other.)
    float X[MT][4][16];
#pragma unroll
    for (int m = 0; m < MT; ++m)
#pragma unroll
        for (int s = 0; s < 4; ++s) {
            const int64_t kb = (int64_t)jj * kChunk + s * kSlab + 16 * e;
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                // unconditional load from a clamped address, then zero what is outside x
                const bool ok = role && m < Ms && kb + 4 * c + 4 <= K;
                const float4 v = *reinterpret_cast<const float4*>(xg + (ok ? (int64_t)m * K + kb + 4 * c : 0));
                X[m][s][4 * c + 0] = ok ? v.x : 0.0f;
                X[m][s][4 * c + 1] = ok ? v.y : 0.0f;
                X[m][s][4 * c + 2] = ok ? v.z : 0.0f;
                X[m][s][4 * c + 3] = ok ? v.w : 0.0f;
            }
        }

    // ---- DMA role: instruction i of this wave fills consumer lane sigma = 8i + (lane>>3) ----
    // Per round, the 8 byte offsets (relative to the round's first row) are fixed
    // except for row clamping at the end of W; precompute the unclamped parts.
    int dma_row[8];      // row inside the round (0 .. 4*RQ-1), or -1 if that consumer is idle
    uint32_t dma_col[8]; // byte offset inside the row at slab 0: j*512 + 16*t
    int dma_jlen[8];     // element length of that consumer's segment
    int dma_kin[8];      // element offset inside the segment at slab 0: 8*t
    {
        const int p = lane & 7;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int sigma = 8 * i + (lane >> 3);
            const int cql = wave * 16 + (sigma >> 2);
            const int t = p ^ ((sigma >> 1) & 7);
            if (cql < RQ * J) {
                const int cq = div_j(cql, J, a.jmagic), cj = cql - cq * J;
                dma_row[i] = 4 * cq + (sigma & 3);
                dma_col[i] = (uint32_t)cj * (kChunk * 2) + 16u * t;
                dma_jlen[i] = (cj == J - 1) ? (int)(K - (int64_t)(J - 1) * kChunk) : kChunk;
                dma_kin[i] = 8 * t;
            } else {
                dma_row[i] = -1;
                dma_col[i] = 0;
                dma_jlen[i] = kChunk;
                dma_kin[i] = 0;
            }
        }
    }
    const uint32_t ring_base = lds_addr(&wring[wave][0][0]);
    const int64_t row_bytes = K * 2;

    // Issue step st (round r = st/4, slab s = st%4) into ring slot st % DEPTH.
    auto issue = [&](int st) {
        const int r = st >> 2, s = st & 3;
        const int64_t row0 = 4 * place.start(r);              // first row of the round
        const int64_t rmax = N - 1 - row0;                    // clamp rows to W
        const char* base = reinterpret_cast<const char*>(a.w) + row0 * row_bytes;
        const uint32_t slot = ring_base + (uint32_t)((st % DEPTH) * kSlabBytesPerWave);
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            int64_t row = dma_row[i] < 0 ? 0 : dma_row[i];
            if (row > rmax) row = rmax;
            uint32_t col = dma_col[i] + (uint32_t)(s * kSlab * 2);
            if (s * kSlab + dma_kin[i] >= dma_jlen[i]) col = 0;   // past the end of a short last segment
            const uint32_t voff = (uint32_t)(row * row_bytes) + col;
            dma16<true>(base, voff, slot + 1024u * i);
        }
    };

    float acc[MT];
    const int rows_wg = 4 * nq;

    // prologue
#pragma unroll
    for (int st = 0; st < DEPTH - 1; ++st)
        if (st < nsteps) issue(st);

    for (int st = 0; st < nsteps; ++st) {
        const int r = st >> 2, s = st & 3;
        if (st + DEPTH - 1 < nsteps) issue(st + DEPTH - 1);
        const int ahead = min(DEPTH - 1, nsteps - 1 - st);
        if (ahead >= 2) vmcnt_wait<16>();
        else if (ahead == 1) vmcnt_wait<8>();
        else vmcnt_wait<0>();

        const bool active = role && (lq < nq - r * RQ);
        if (s == 0) {
#pragma unroll
            for (int m = 0; m < MT; ++m) acc[m] = 0.0f;
        }
        // ---- consume slab s: 64 elements of this lane's (row, segment) ----
        const int npieces = min(8, max(0, (seg_len - s * kSlab) / 8));
        if (active && npieces > 0) {
            const uint8_t* src = &wring[wave][st % DEPTH][lane * 128];
            const int sw = (lane >> 1) & 7;
            uint4 wp[8];
#pragma unroll
            for (int t = 0; t < 8; ++t) wp[t] = *reinterpret_cast<const uint4*>(src + 16 * (t ^ sw));
            if (npieces == 8) {
                switch (s) {   // static slab index keeps X in registers
                    case 0: fma_slab<0, MT, true>(wp, X, acc, 8); break;
                    case 1: fma_slab<1, MT, true>(wp, X, acc, 8); break;
                    case 2: fma_slab<2, MT, true>(wp, X, acc, 8); break;
                    default: fma_slab<3, MT, true>(wp, X, acc, 8); break;
                }
            } else {
                switch (s) {
                    case 0: fma_slab<0, MT, false>(wp, X, acc, npieces); break;
                    case 1: fma_slab<1, MT, false>(wp, X, acc, npieces); break;
                    case 2: fma_slab<2, MT, false>(wp, X, acc, npieces); break;
                    default: fma_slab<3, MT, false>(wp, X, acc, npieces); break;
                }
            }
        }
        if (s == 3) {
            // segment partials of this round -> LDS, then fold in ascending segment order
            const int par = r & 1;
            if (active) {
#pragma unroll
                for (int m = 0; m < MT; ++m) part[par][m * (kThreads) + (4 * lq + e) * J + jj] = acc[m];
            }
            __syncthreads();
            const int rows_round = 4 * min(RQ, nq - r * RQ);
            for (int o = tid; o < rows_round * MT; o += kThreads) {
                const int rl = o / MT, m = o % MT;
                yres[(r * RQ * 4 + rl) * MT + m] = fold_partials(&part[par][m * kThreads + rl * J], J);
            }
            // The next round writes the other parity; this parity is rewritten
            // only after the next round's barrier, which all folds precede.
        }
    }
    vmcnt_wait<0>();
    __syncthreads();
    // ---- write results ----
    for (int o = tid; o < rows_wg * MT; o += kThreads) {
        const int m = o / rows_wg, rl = o % rows_wg;
        const int64_t n = staged_row(place, rl, RQ);
        if (m < Ms && n < N) {
            const float v = yres[rl * MT + m];
            yg[(int64_t)m * N + n] = a.bias ? v + a.bias[n] : v;
        }
    }
}

// ---------------------------------------------------------------------------
// decode kernel for M == 1 with x streamed beside W.
//
// Same work split, lane roles, order and W data path as decode_kernel, but x
// is not preloaded into registers: with every 64-element W slab, each wave
// also DMAs the matching 64 floats of x for each of its 16 quads (4 KB) into
// a second LDS ring.  All loads in flight are then global->LDS DMA loads of
// one wave, which complete in issue order, so a slab can be consumed as soon
// as its own loads have landed.  Lane e of a quad reads the 16 floats x[16e,
// 16e+16) of the slab; the others reach it through DPP quad broadcasts.  The
// 256-byte x image of a quad is stored with its 16-byte pieces permuted
// (piece c of lane e at slot 4e + (c ^ (quad & 3))) so that the 16 lanes of
// an LDS phase read 16 distinct bank groups.  The segment partials of up to
// 4 rounds are kept in LDS and folded together, one row per thread.
// ---------------------------------------------------------------------------
constexpr int kXSlabBytesPerWave = 16 * 256;  // 4 KB: 16 quads x 64 floats

template <bool FULL>
__device__ __forceinline__ void fma_slab1(const uint4 (&wp)[8], const float (&Xs)[16], float& acc, int npieces) {
    if constexpr (FULL) {
        // 8 pieces of 8 elements; piece t uses the x block of quad lane t/2
#pragma unroll
        for (int t = 0; t < 8; ++t) {
            const uint32_t d[4] = {wp[t].x, wp[t].y, wp[t].z, wp[t].w};
            float wv[8];
#pragma unroll
            for (int h = 0; h < 8; ++h) wv[h] = (h & 1) ? up_hi(d[h >> 1]) : up_lo(d[h >> 1]);
            const float* xb = &Xs[8 * (t & 1)];
            switch (t >> 1) {
                case 0: fmac8_bcast<0>(acc, xb, wv); break;
                case 1: fmac8_bcast<1>(acc, xb, wv); break;
                case 2: fmac8_bcast<2>(acc, xb, wv); break;
                default: fmac8_bcast<3>(acc, xb, wv); break;
            }
        }
        return;
    }
#pragma unroll
    for (int t = 0; t < 8; ++t) {
        if (!FULL && t >= npieces) break;   // short last segment only
        const uint32_t d[4] = {wp[t].x, wp[t].y, wp[t].z, wp[t].w};
#pragma unroll
        for (int h = 0; h < 8; ++h) {
            const float wv = (h & 1) ? up_hi(d[h >> 1]) : up_lo(d[h >> 1]);
            const int kl = 8 * t + h;          // element inside the slab
            const int i = kl & 15;             // register inside the x block
            float xv;
            switch (kl >> 4) {                 // lane of the quad holding x
                case 0: xv = quad_bcast<0>(Xs[i]); break;
                case 1: xv = quad_bcast<1>(Xs[i]); break;
                case 2: xv = quad_bcast<2>(Xs[i]); break;
                default: xv = quad_bcast<3>(Xs[i]); break;
            }
            acc = __builtin_fmaf(xv, wv, acc);
        }
    }
}

template <int NW, int DEPTH, bool RM>
__global__ void __launch_bounds__(NW * 64, 1) decode1_kernel(DecodeArgs a) {
    static_assert(DEPTH >= 2 && DEPTH <= 3, "pipeline depth");
    constexpr int kThreads = NW * 64;
    constexpr int kDmaPerStep = 8 + 4;      // W: 8 KB, x: 4 KB per wave

    __shared__ __attribute__((aligned(16))) uint8_t wring[NW][DEPTH][kSlabBytesPerWave];
    __shared__ __attribute__((aligned(16))) uint8_t xring[NW][DEPTH][kXSlabBytesPerWave];
    constexpr int FR = 4;                             // rounds whose partials are folded together
    __shared__ float part[FR][kThreads];              // [round % FR][row_local * J + j]
    extern __shared__ float yres[];                   // [row_in_wg], dynamic

    const int tid = threadIdx.x;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int lane = tid & 63;
    const int J = a.J;
    const int RQ = a.RQ;
    const int64_t N = a.N, K = a.K;

    // balanced split of the Q quads over the grid (the first qrem workgroups take one more),
    // placed as quad_place says
    const int G = (int)gridDim.x;
    const int g = a.reverse ? G - 1 - (int)blockIdx.x : (int)blockIdx.x;
    const int nq = (int)a.qbase + (g < a.qrem ? 1 : 0);
    const int rounds = (nq + RQ - 1) / RQ;
    const int nsteps = rounds * (kChunk / kSlab);
    const QuadPlace<RM> place = quad_place<RM>(g, G, a.qbase, a.qrem, RQ);

    // ---- fixed lane role (consumer) ----
    const int ql = tid >> 2;
    const int e = tid & 3;
    const bool role = ql < RQ * J;
    const int lq = role ? div_j(ql, J, a.jmagic) : 0;
    const int jj = role ? ql - lq * J : 0;
    const int seg_len = (jj == J - 1) ? (int)(K - (int64_t)(J - 1) * kChunk) : kChunk;
    const int last_len = (int)(K - (int64_t)(J - 1) * kChunk);

    // ---- W DMA role (as in decode_kernel) ----
    int dma_row[8];
    uint32_t dma_col[8];
    int dma_jlen[8];
    int dma_kin[8];
    {
        const int p = lane & 7;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int sigma = 8 * i + (lane >> 3);
            const int cql = wave * 16 + (sigma >> 2);
            const int t = p ^ ((sigma >> 1) & 7);
            if (cql < RQ * J) {
                const int cq = div_j(cql, J, a.jmagic), cj = cql - cq * J;
                dma_row[i] = 4 * cq + (sigma & 3);
                dma_col[i] = (uint32_t)cj * (kChunk * 2) + 16u * t;
                dma_jlen[i] = (cj == J - 1) ? last_len : kChunk;
                dma_kin[i] = 8 * t;
            } else {
                dma_row[i] = -1;
                dma_col[i] = 0;
                dma_jlen[i] = kChunk;
                dma_kin[i] = 0;
            }
        }
    }
    // ---- x DMA role: instruction i fills quads 4i..4i+3 of this wave ----
    // x offsets (elements) of slab 0; the same for every round.
    int xdma_k[4];       // element index inside x at slab 0, or -1 for an idle quad
    int xdma_len[4];     // segment length of that quad
    int xdma_kin[4];     // element offset inside the segment at slab 0
    {
        const int sig = lane & 15;
        const int ee = sig >> 2;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int q = 4 * i + (lane >> 4);
            const int c = (sig & 3) ^ (q & 3);
            const int cql = wave * 16 + q;
            if (cql < RQ * J) {
                const int cj = cql - div_j(cql, J, a.jmagic) * J;
                xdma_kin[i] = 16 * ee + 4 * c;
                xdma_k[i] = cj * kChunk + xdma_kin[i];
                xdma_len[i] = (cj == J - 1) ? last_len : kChunk;
            } else {
                xdma_kin[i] = 0;
                xdma_k[i] = -1;
                xdma_len[i] = kChunk;
            }
        }
    }
    const uint32_t ring_base = lds_addr(&wring[wave][0][0]);
    const uint32_t xring_base = lds_addr(&xring[wave][0][0]);
    const int64_t row_bytes = K * 2;

    auto issue = [&](int st) {
        const int r = st >> 2, s = st & 3;
        const int64_t row0 = 4 * place.start(r);
        const int64_t rmax = N - 1 - row0;
        const char* base = reinterpret_cast<const char*>(a.w) + row0 * row_bytes;
        const uint32_t slot = ring_base + (uint32_t)((st % DEPTH) * kSlabBytesPerWave);
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            int64_t row = dma_row[i] < 0 ? 0 : dma_row[i];
            if (row > rmax) row = rmax;
            uint32_t col = dma_col[i] + (uint32_t)(s * kSlab * 2);
            if (s * kSlab + dma_kin[i] >= dma_jlen[i]) col = 0;
            const uint32_t voff = (uint32_t)(row * row_bytes) + col;
            dma16<true>(base, voff, slot + 1024u * i);
        }
        const uint32_t xslot = xring_base + (uint32_t)((st % DEPTH) * kXSlabBytesPerWave);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            // past the end of a short last segment, or an idle quad: element 0 of x (never used)
            const bool ok = xdma_k[i] >= 0 && s * kSlab + xdma_kin[i] < xdma_len[i];
            const uint32_t voff = ok ? 4u * (uint32_t)(xdma_k[i] + s * kSlab) : 0u;
            dma16(a.x, voff, xslot + 1024u * i);
        }
    };

    float acc = 0.0f;
    const int rows_wg = 4 * nq;
    const int xq = tid >> 2 & 15;          // quad inside the wave

#pragma unroll
    for (int st = 0; st < DEPTH - 1; ++st)
        if (st < nsteps) issue(st);

    for (int st = 0; st < nsteps; ++st) {
        const int r = st >> 2, s = st & 3;
        if (st + DEPTH - 1 < nsteps) issue(st + DEPTH - 1);
        const int ahead = min(DEPTH - 1, nsteps - 1 - st);
        if (ahead >= 2) vmcnt_wait<2 * kDmaPerStep>();
        else if (ahead == 1) vmcnt_wait<kDmaPerStep>();
        else vmcnt_wait<0>();

        const bool active = role && (lq < nq - r * RQ);
        if (s == 0) acc = 0.0f;
        const int npieces = min(8, max(0, (seg_len - s * kSlab) / 8));
        if (active && npieces > 0) {
            const uint8_t* src = &wring[wave][st % DEPTH][lane * 128];
            const int sw = (lane >> 1) & 7;
            uint4 wp[8];
#pragma unroll
            for (int t = 0; t < 8; ++t) wp[t] = *reinterpret_cast<const uint4*>(src + 16 * (t ^ sw));
            const uint8_t* xs = &xring[wave][st % DEPTH][xq * 256];
            float Xs[16];
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                const float4 v = *reinterpret_cast<const float4*>(xs + 16 * (4 * e + (c ^ (xq & 3))));
                Xs[4 * c + 0] = v.x;
                Xs[4 * c + 1] = v.y;
                Xs[4 * c + 2] = v.z;
                Xs[4 * c + 3] = v.w;
            }
            if (npieces == 8) fma_slab1<true>(wp, Xs, acc, 8);
            else fma_slab1<false>(wp, Xs, acc, npieces);
        }
        if (s == 3) {
            // keep the round's partials; every FR rounds (and after the last) fold them all,
            // one row per thread, so the serial fold is waited for once per FR rounds
            const int slot = r % FR;
            if (active) part[slot][(4 * lq + e) * J + jj] = acc;
            if (slot == FR - 1 || r == rounds - 1) {
                __syncthreads();
                const int r0 = r - slot;
                const int rows = 4 * min((slot + 1) * RQ, nq - r0 * RQ);
                for (int o = tid; o < rows; o += kThreads) {
                    const int rr = o / (4 * RQ), ro = o - rr * 4 * RQ;
                    yres[r0 * RQ * 4 + o] = fold_partials(&part[rr][ro * J], J);
                }
                __syncthreads();                      // the next round writes the ring again
            }
        }
    }
    vmcnt_wait<0>();
    __syncthreads();
    for (int o = tid; o < rows_wg; o += kThreads) {
        const int64_t n = staged_row(place, o, RQ);
        if (n < N) a.y[n] = a.bias ? yres[o] + a.bias[n] : yres[o];
    }
}

// ---------------------------------------------------------------------------
// tiled kernel (large M): register-tiled SGEMM-shaped kernel, whole K per
// workgroup, same order.
//
// A 256-thread workgroup owns a BM x BN output tile (16 x 16 threads, each
// holding TM x TN outputs, as two interleaved halves per dimension so that
// LDS reads are conflict free).  K advances in slabs of KT (32 for the 128 x 128
// two-waves-per-SIMD build, 16 otherwise): x[BM][KT] and up(W)[BN][KT] are
// staged transposed in LDS (double buffered, the next slab prefetched into
// registers while the current one is multiplied).  Each output keeps two
// registers: the running chain of the current 256-wide segment (from +0,
// ascending k) and the fold of the finished segments (first segment taken as
// is, later ones added in ascending order).
//
// Every slab runs all KT steps: the missing k of a short last slab are
// staged as +0 in x and -0 in W.  The product +0 * -0 is -0, and -0 + p = p
// for every p (including p = -0, which a chain reaches when a negative
// product underflows), so fmaf(+0, -0, p) = p and the padded steps change no
// bit.  (A +0 weight would not do: fmaf(+0, +0, -0) = +0.)
//
// Limits.  Each thread's 64 independent chains keep the FMA pipeline busy
// (plain FMAs with 16 or more independent chains per wave measure ~69
// TFLOP/s at one wave per SIMD and ~133 at two), so at two waves per SIMD the
// limits are LDS (8 x 8 outputs read 1 byte per FMA, the same order as the
// LDS return rate at the FMA peak) and the per-slab barrier, which the
// 32-wide slab halves.  The 128 x 128 tile comes in two builds: two waves per
// SIMD with the next step's operands read ahead (no spills), and three waves
// per SIMD (at most 168 registers: one operand set per step, a few registers
// spilled outside the FMA loop).  The planner takes the three-wave build only
// where its rounds of 3 workgroups per CU are clearly fuller.
// ---------------------------------------------------------------------------
constexpr int kTK = 16;   // k per slab (the 128 x 128 two-waves-per-SIMD build: 32)

// n consecutive floats from LDS (n = 2, 4 or 8; the address is n*4-byte aligned)
template <int n>
__device__ __forceinline__ void lds_vec(const float* p, float* out) {
    if constexpr (n == 2) {
        const float2 v = *reinterpret_cast<const float2*>(p);
        out[0] = v.x; out[1] = v.y;
    } else {
        static_assert(n % 4 == 0, "vector width");
#pragma unroll
        for (int q = 0; q < n; q += 4) {
            const float4 v = *reinterpret_cast<const float4*>(p + q);
            out[q] = v.x; out[q + 1] = v.y; out[q + 2] = v.z; out[q + 3] = v.w;
        }
    }
}

// KT: k per slab (a divisor of the segment length 256, so a slab never straddles a
// segment); W3: the three-waves-per-SIMD build (one operand set per step).
template <int BM, int BN, int KT, typename WT, bool W3>
__device__ __forceinline__ void tiled_body(const float* __restrict__ x, const WT* __restrict__ w,
                                           const float* __restrict__ bias, float* __restrict__ y, int64_t M,
                                           int64_t N, int64_t K, int reverse) {
    constexpr int TM = BM / 16, TN = BN / 16;        // per-thread outputs per dimension
    constexpr int HM = TM / 2, HN = TN / 2;          // two interleaved halves
    static_assert(TM % 2 == 0 && TN % 2 == 0, "tile");
    constexpr int PADM = BM + 4, PADN = BN + 4;
    static_assert(kChunk % KT == 0, "slabs inside segments");
    __shared__ __attribute__((aligned(16))) float xs[2][KT][PADM];
    __shared__ __attribute__((aligned(16))) float ws[2][KT][PADN];

    const int tid = threadIdx.x;
    const int tn = tid & 15, tm = tid >> 4;
    const int64_t tiles_n = (N + BN - 1) / BN;
    const int64_t b = reverse ? (int64_t)(gridDim.x - 1 - blockIdx.x) : (int64_t)blockIdx.x;
    const int64_t m0 = (b / tiles_n) * BM, n0 = (b % tiles_n) * BN;

    // staging roles: x tile BM x 16 floats, W tile BN x 16 weights (16-byte vectors of WE);
    // k >= K is staged as x = +0, w = -0 (K % 8 == 0 on this path, so a vector is wholly
    // in or out)
    using WV = WVec<WT>;
    constexpr int WE = WV::E, WPR = KT / WE;         // weights per vector, vectors per tile row
    constexpr int XF4 = BM * KT / 4 / 256;           // float4 loads per thread for x
    constexpr int WU4 = (BN * WPR + 255) / 256;      // weight vector loads per thread
    float4 xr[XF4];
    typename WV::V wr[WU4];

    auto load_slab = [&](int64_t k0) {
#pragma unroll
        for (int u = 0; u < XF4; ++u) {
            const int idx = tid + 256 * u;            // over BM rows x KT/4 float4
            const int row = idx / (KT / 4), kq = idx % (KT / 4);
            const int64_t gm = m0 + row, gk = k0 + 4 * kq;
            const bool ok = gm < M && gk + 4 <= K;
            xr[u] = ok ? *reinterpret_cast<const float4*>(x + gm * K + gk) : make_float4(0.f, 0.f, 0.f, 0.f);
        }
#pragma unroll
        for (int u = 0; u < WU4; ++u) {
            const int idx = tid + 256 * u;            // over BN rows x WPR vectors
            const int row = idx / WPR, kh = idx % WPR;
            const int64_t gn = n0 + row, gk = k0 + WE * kh;
            const bool ok = row < BN && gn < N && gk + WE <= K;
            wr[u] = ok ? *reinterpret_cast<const typename WV::V*>(w + gn * K + gk) : WV::neg_zero();
        }
    };
    auto store_slab = [&](int buf) {
#pragma unroll
        for (int u = 0; u < XF4; ++u) {
            const int idx = tid + 256 * u;
            const int row = idx / (KT / 4), kq = idx % (KT / 4);
            xs[buf][4 * kq + 0][row] = xr[u].x;
            xs[buf][4 * kq + 1][row] = xr[u].y;
            xs[buf][4 * kq + 2][row] = xr[u].z;
            xs[buf][4 * kq + 3][row] = xr[u].w;
        }
#pragma unroll
        for (int u = 0; u < WU4; ++u) {
            const int idx = tid + 256 * u;
            const int row = idx / WPR, kh = idx % WPR;
            if (row < BN) {
#pragma unroll
                for (int h = 0; h < WE; ++h) ws[buf][WE * kh + h][row] = WV::get(wr[u], h);
            }
        }
    };

    float acc[TM][TN], tot[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = 0.0f, tot[i][j] = 0.0f;

    const int64_t nslabs = (K + KT - 1) / KT;
    load_slab(0);
    store_slab(0);
    __syncthreads();
    for (int64_t sl = 0; sl < nslabs; ++sl) {
        const int buf = (int)(sl & 1);
        if (sl + 1 < nslabs) load_slab((sl + 1) * KT);
        if constexpr (W3) {
            // one operand set per step; the scheduling barrier keeps later steps' reads from
            // being hoisted into registers (three waves per SIMD hide the LDS latency instead)
#pragma unroll
            for (int kk = 0; kk < KT; ++kk) {
                float xv[TM], wv[TN];
#pragma unroll
                for (int h = 0; h < 2; ++h) {
                    lds_vec<HM>(&xs[buf][kk][h * (BM / 2) + tm * HM], &xv[h * HM]);
                    lds_vec<HN>(&ws[buf][kk][h * (BN / 2) + tn * HN], &wv[h * HN]);
                }
#pragma unroll
                for (int i = 0; i < TM; ++i)
#pragma unroll
                    for (int j = 0; j < TN; ++j) acc[i][j] = __builtin_fmaf(xv[i], wv[j], acc[i][j]);
                __builtin_amdgcn_sched_barrier(0);
            }
        } else {
            // operands of step kk + 1 are read from LDS while step kk's FMAs run
            float xv[2][TM], wv[2][TN];
            auto read_k = [&](int kk, int r) {
#pragma unroll
                for (int h = 0; h < 2; ++h) {
                    lds_vec<HM>(&xs[buf][kk][h * (BM / 2) + tm * HM], &xv[r][h * HM]);
                    lds_vec<HN>(&ws[buf][kk][h * (BN / 2) + tn * HN], &wv[r][h * HN]);
                }
            };
            read_k(0, 0);
#pragma unroll
            for (int kk = 0; kk < KT; ++kk) {
                const int r = kk & 1;
                if (kk + 1 < KT) read_k(kk + 1, r ^ 1);
#pragma unroll
                for (int i = 0; i < TM; ++i)
#pragma unroll
                    for (int j = 0; j < TN; ++j) acc[i][j] = __builtin_fmaf(xv[r][i], wv[r][j], acc[i][j]);
            }
        }
        // end of a 256-wide segment (or of K): fold the segment chain, restart it from +0
        const int64_t kend = min((sl + 1) * KT, K);
        if ((kend % kChunk) == 0 || kend == K) {
            const bool first = kend <= kChunk;
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j) {
                    tot[i][j] = first ? acc[i][j] : tot[i][j] + acc[i][j];
                    acc[i][j] = 0.0f;
                }
        }
        if (sl + 1 < nslabs) {
            store_slab(buf ^ 1);
            __syncthreads();
        }
    }
#pragma unroll
    for (int i = 0; i < TM; ++i) {
        const int64_t gm = m0 + (i < HM ? tm * HM + i : BM / 2 + tm * HM + (i - HM));
        if (gm >= M) continue;
#pragma unroll
        for (int j = 0; j < TN; ++j) {
            const int64_t gn = n0 + (j < HN ? tn * HN + j : BN / 2 + tn * HN + (j - HN));
            if (gn < N) y[gm * N + gn] = bias ? tot[i][j] + bias[gn] : tot[i][j];
        }
    }
}

template <int BM, int BN, typename WT>
__global__ void __launch_bounds__(256) tiled_kernel(const float* __restrict__ x, const WT* __restrict__ w,
                                                    const float* __restrict__ bias, float* __restrict__ y, int64_t M,
                                                    int64_t N, int64_t K, int reverse) {
    // 32 k per slab for the 128 x 128 tile (half the barriers; measured 4-12 % faster), 16 otherwise
    tiled_body<BM, BN, (BM == 128 && BN == 128) ? 32 : kTK, WT, false>(x, w, bias, y, M, N, K, reverse);
}

// The 128 x 128 tile built for three waves per SIMD.
template <typename WT>
__global__ void __launch_bounds__(256, 3) tiled3_kernel(const float* __restrict__ x, const WT* __restrict__ w,
                                                       const float* __restrict__ bias, float* __restrict__ y,
                                                       int64_t M, int64_t N, int64_t K, int reverse) {
    tiled_body<128, 128, kTK, WT, true>(x, w, bias, y, M, N, K, reverse);
}

// ---------------------------------------------------------------------------
// ktile kernel (small M, 4 < M <= 64): register tiles of 4 x 4 outputs with
// the segments of K shared out over groups of threads.
//
// A workgroup of NT threads owns a BM x BN output tile and all of K.  Its
// threads form KS groups of NT / KS; group g runs segments g, g + KS,
// g + 2KS, ... (one segment per group per round), each thread a 4 x 4 tile
// of chains over the segment in ascending k.  x (BM x KT floats) and up(W)
// (BN x KT, widened once when staged) pass through LDS transposed, double
// buffered, KT elements of every group's segment per barrier.  After a round
// the groups' segment partials meet in LDS and group 0 folds them into its
// running totals in ascending segment order (the first partial starts the
// sum).  Splitting K this way gives small-M shapes enough independent work
// for several waves per SIMD while the order stays the documented one.
// ---------------------------------------------------------------------------
template <int BM, int BN, int KS, int NT, typename WT, int CN>
__global__ void __launch_bounds__(NT) ktile_kernel(const float* __restrict__ x, const WT* __restrict__ w,
                                                   const float* __restrict__ bias, float* __restrict__ y, int64_t M, int64_t N, int64_t K,
                                                   int reverse) {
    static_assert(CN == 4 || CN == 8, "W rows per thread");
    static_assert(BM * BN * KS == 4 * CN * NT, "NT threads x 4 CN outputs");
    constexpr int TG = NT / KS;                      // threads per group
    constexpr int KT = KS >= 8 ? 8 : 16;             // elements per slab
    constexpr int NSL = kChunk / KT;                 // slabs per segment
    constexpr int PADM = BM + 4, PADN = BN + 4;
    using WV = WVec<WT>;
    constexpr int WE = WV::E, WPR = KT / WE;         // weights per vector, vectors per slab row
    constexpr int XPT = (BM * KT / 4 + TG - 1) / TG; // float4 x loads per thread
    constexpr int WPT = (BN * WPR + TG - 1) / TG;    // weight vector loads per thread
    __shared__ __attribute__((aligned(16))) float xs[KS][2][KT][PADM];
    __shared__ __attribute__((aligned(16))) float ws[KS][2][KT][PADN];
    __shared__ __attribute__((aligned(16))) float part[KS > 1 ? KS - 1 : 1][TG][4 * CN];

    const int tid = threadIdx.x;
    const int g = tid / TG, tg = tid % TG;
    const int mi = tg % (BM / 4), ni = tg / (BM / 4);
    const int64_t tiles_n = (N + BN - 1) / BN;
    const int64_t b = reverse ? (int64_t)(gridDim.x - 1 - blockIdx.x) : (int64_t)blockIdx.x;
    const int64_t m0 = (b / tiles_n) * BM, n0 = (b % tiles_n) * BN;
    const int J = (int)((K + kChunk - 1) / kChunk);
    const int rounds = (J + KS - 1) / KS;

    float4 xr[XPT];
    typename WV::V wr[WPT];
    // slab sl of this group's segment in round t
    auto load_slab = [&](int t, int sl) {
        const int64_t j = (int64_t)t * KS + g;
        const int64_t k0 = j * kChunk + (int64_t)sl * KT;
#pragma unroll
        for (int u = 0; u < XPT; ++u) {
            const int idx = tg + TG * u;                  // over BM rows x KT/4 float4
            const int row = idx / (KT / 4), kq = idx % (KT / 4);
            const int64_t gm = m0 + row, gk = k0 + 4 * kq;
            const bool ok = idx < BM * KT / 4 && j < J && gm < M && gk + 4 <= K;
            xr[u] = ok ? *reinterpret_cast<const float4*>(x + gm * K + gk) : make_float4(0.f, 0.f, 0.f, 0.f);
        }
#pragma unroll
        for (int u = 0; u < WPT; ++u) {
            const int idx = tg + TG * u;                  // over BN rows x WPR vectors
            const int row = idx / WPR, kh = idx % WPR;
            const int64_t gn = n0 + row, gk = k0 + WE * kh;
            const bool ok = idx < BN * WPR && j < J && gn < N && gk + WE <= K;
            // (a normal load: a slab reads 16 or 32 bytes of each 128-byte line of a row and the
            // next slab the rest, which a non-temporal load would not find in the cache)
            wr[u] = ok ? *reinterpret_cast<const typename WV::V*>(w + gn * K + gk) : WV::zero();
        }
    };
    auto store_slab = [&](int buf) {
#pragma unroll
        for (int u = 0; u < XPT; ++u) {
            const int idx = tg + TG * u;
            if (idx < BM * KT / 4) {
                const int row = idx / (KT / 4), kq = idx % (KT / 4);
                xs[g][buf][4 * kq + 0][row] = xr[u].x;
                xs[g][buf][4 * kq + 1][row] = xr[u].y;
                xs[g][buf][4 * kq + 2][row] = xr[u].z;
                xs[g][buf][4 * kq + 3][row] = xr[u].w;
            }
        }
#pragma unroll
        for (int u = 0; u < WPT; ++u) {
            const int idx = tg + TG * u;
            if (idx < BN * WPR) {
                const int row = idx / WPR, kh = idx % WPR;
#pragma unroll
                for (int h = 0; h < WE; ++h) ws[g][buf][WE * kh + h][row] = WV::get(wr[u], h);
            }
        }
    };

    float acc[4 * CN], tot[4 * CN];
#pragma unroll
    for (int i = 0; i < 4 * CN; ++i) tot[i] = 0.0f;

    load_slab(0, 0);
    store_slab(0);
    __syncthreads();
    int buf = 0;
    for (int t = 0; t < rounds; ++t) {
        const int64_t j = (int64_t)t * KS + g;
        const int len = j < J ? (int)min((int64_t)kChunk, K - j * kChunk) : 0;   // this group's segment length
#pragma unroll
        for (int i = 0; i < 4 * CN; ++i) acc[i] = 0.0f;
        for (int sl = 0; sl < NSL; ++sl) {
            const bool more = sl + 1 < NSL || t + 1 < rounds;
            if (more) load_slab(sl + 1 < NSL ? t : t + 1, sl + 1 < NSL ? sl + 1 : 0);
            const int kvalid = max(0, min(KT, len - sl * KT));
            if (kvalid == KT) {
#pragma unroll
                for (int kk = 0; kk < KT; ++kk) {
                    const float4 xv = *reinterpret_cast<const float4*>(&xs[g][buf][kk][4 * mi]);
                    const float xa[4] = {xv.x, xv.y, xv.z, xv.w};
                    float wa[CN];
#pragma unroll
                    for (int q = 0; q < CN; q += 4) {
                        const float4 wv = *reinterpret_cast<const float4*>(&ws[g][buf][kk][CN * ni + q]);
                        wa[q] = wv.x; wa[q + 1] = wv.y; wa[q + 2] = wv.z; wa[q + 3] = wv.w;
                    }
#pragma unroll
                    for (int r = 0; r < 4; ++r)
#pragma unroll
                        for (int c = 0; c < CN; ++c) acc[CN * r + c] = __builtin_fmaf(xa[r], wa[c], acc[CN * r + c]);
                }
            } else {
                for (int kk = 0; kk < kvalid; ++kk) {
                    const float4 xv = *reinterpret_cast<const float4*>(&xs[g][buf][kk][4 * mi]);
                    const float xa[4] = {xv.x, xv.y, xv.z, xv.w};
                    float wa[CN];
#pragma unroll
                    for (int q = 0; q < CN; q += 4) {
                        const float4 wv = *reinterpret_cast<const float4*>(&ws[g][buf][kk][CN * ni + q]);
                        wa[q] = wv.x; wa[q + 1] = wv.y; wa[q + 2] = wv.z; wa[q + 3] = wv.w;
                    }
#pragma unroll
                    for (int r = 0; r < 4; ++r)
#pragma unroll
                        for (int c = 0; c < CN; ++c) acc[CN * r + c] = __builtin_fmaf(xa[r], wa[c], acc[CN * r + c]);
                }
            }
            if (more) {
                store_slab(buf ^ 1);
                __syncthreads();
                buf ^= 1;
            }
        }
        // the round's segment partials, folded by group 0 in ascending segment order
        if constexpr (KS > 1) {
            if (g > 0) {
#pragma unroll
                for (int i = 0; i < 4 * CN; i += 4)
                    *reinterpret_cast<float4*>(&part[g - 1][tg][i]) = make_float4(acc[i], acc[i + 1], acc[i + 2], acc[i + 3]);
            }
            __syncthreads();
        }
        if (g == 0) {
#pragma unroll
            for (int i = 0; i < 4 * CN; ++i) tot[i] = (t == 0) ? acc[i] : tot[i] + acc[i];
            if constexpr (KS > 1) {
                for (int gg = 1; gg < KS; ++gg) {
                    if ((int64_t)t * KS + gg >= J) break;
#pragma unroll
                    for (int i = 0; i < 4 * CN; i += 4) {
                        const float4 pv = *reinterpret_cast<const float4*>(&part[gg - 1][tg][i]);
                        tot[i] = tot[i] + pv.x;
                        tot[i + 1] = tot[i + 1] + pv.y;
                        tot[i + 2] = tot[i + 2] + pv.z;
                        tot[i + 3] = tot[i + 3] + pv.w;
                    }
                }
            }
        }
        // part[] is written again only after the next round's slab barriers, which group 0
        // reaches after this fold
    }
    if (g == 0) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int64_t gm = m0 + 4 * mi + r;
            if (gm >= M) continue;
#pragma unroll
            for (int c = 0; c < CN; ++c) {
                const int64_t gn = n0 + CN * ni + c;
                if (gn < N) y[gm * N + gn] = bias ? tot[CN * r + c] + bias[gn] : tot[CN * r + c];
            }
        }
    }
}

// ---------------------------------------------------------------------------
// gemv kernel (M == 1, K a multiple of 256 with at least 16 segments):
// dense weight stream.
//
// Work split.  W rows are grouped in quads of 4 consecutive rows.  The grid
// has V waves in all; wave v owns quads v, v + V, v + 2V, ..., so at any
// moment the whole grid reads one compact window of W, and each wave owns
// whole rows: every output is finished inside one wave (no cross-wave or
// cross-workgroup reduction, no atomics, no barriers in the stream).
//
// Data path.  A wave step covers segments 16s .. 16s+15 of the quad's 4 rows
// (4 x 8 KB of W, contiguous within each row).  The wave requests the whole
// step at once with 32 global->LDS DMA instructions (8 lanes per 128-byte
// line) into its own 32 KB LDS slot, so each DRAM page of the window is read
// in one burst.  The DMA image is ordered by quarter: quarter q holds
// elements 64q .. 64q+63 of every segment, so the step is consumed quarter by
// quarter as its DMA instructions land (they complete in issue order) and
// only one quarter's FMAs follow the last byte.  The next step is requested
// as soon as the slot has been read.  Inside a quarter the 128-byte image of
// a lane is XOR-swizzled by ((lane >> 1) & 7) in 16-byte units, so the
// transposing ds_read_b128 are conflict-free.
//
// Lane roles.  Lane c = 4j + r owns segment 16s + j of row r of the quad and
// runs its whole 256-long fmaf chain from +0 inside the step.  The 4 lanes of
// a DPP quad share a segment; lane r holds x for elements 64r .. 64r+63 of it
// and the others read those through quad broadcasts fused into v_fmac_f32.
// x stays in registers when one step covers K (K = 4096).  Otherwise (XP) the
// workgroup stages x one step at a time: the 16 segments of step s (16 KB of
// x) sit in a shared LDS image; at each step every wave reads its 64 values
// into registers, the waves meet at a barrier, each wave DMAs its quarter
// (NW = 4) of the next step's x into the image, and after its FMAs waits for
// that DMA and meets the others at a second barrier.  All waves of a
// workgroup therefore walk the same steps (a wave without a quad at some
// round only moves x), and the 16 KB image leaves room for four 32 KB W
// slots at any K.
//
// Order.  After a step the 16 segment partials of each row go to LDS and
// lane r folds them into row r's running sum in ascending segment order
// (the first partial starts the sum); after the quad's last step lane r
// stores the row.  When one step covers K the partials of up to 8 quads are
// kept and folded together, one row per lane, so the serial fold is paid
// once per 8 quads instead of once per step.
// ---------------------------------------------------------------------------
constexpr int kGemvSlabBytes = 32768;   // 4 rows x 16 segments x 512 bytes of W

template <int NW, bool XP>
__global__ void __launch_bounds__(NW * 64, 1) gemv_kernel(GemvArgs a) {
    static_assert(!XP || 16 % NW == 0, "every wave issues the same number of x DMA instructions");
    constexpr int XN = 16 / NW;   // XP: x DMA instructions per wave per step
    __shared__ __attribute__((aligned(16))) uint8_t wslot[NW][kGemvSlabBytes];
    // partials [row r][segment j] of a step: of the last FB quads when one step covers K
    // (folded FB quads at a time), else of the current step
    constexpr int FB = XP ? 1 : 8;
    __shared__ __attribute__((aligned(16))) float fold[NW][FB][64];
    extern __shared__ __attribute__((aligned(16))) uint8_t ximg[]; // x (J == 16) or a step's part, 16 KB, swizzled

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int J = a.J, S = a.S;
    const int64_t N = a.N, K = a.K;
    const int g = a.reverse ? (int)(gridDim.x - 1 - blockIdx.x) : (int)blockIdx.x;
    const int64_t V = (int64_t)gridDim.x * NW;
    const int64_t v = (int64_t)g * NW + wave;
    const int nq = (int)a.qbase + (v < a.qrem ? 1 : 0);   // quads of this wave
    const int64_t row_bytes = 2 * K;

    // ---- DMA roles: instruction 8q + m, this lane fills consumer lane c = 8m + (lane >> 3),
    // 16-byte slot (lane & 7), which holds piece u = slot ^ ((c >> 1) & 7) of quarter q ----
    uint32_t doff[8];   // byte offset of quarter 0's piece inside the step window, full step
#pragma unroll
    for (int m = 0; m < 8; ++m) {
        const int c = 8 * m + (lane >> 3);
        const int u = (lane & 7) ^ ((c >> 1) & 7);
        doff[m] = (uint32_t)((c & 3) * row_bytes) + 512u * (uint32_t)(c >> 2) + 16u * (uint32_t)u;
    }
    const uint32_t wbase = lds_addr(&wslot[wave][0]);

    // request step (t, s): quad v + t*V, segments 16s .. 16s+15 (32 DMA instructions)
    auto issue = [&](int t, int s) {
        const int64_t row0 = 4 * (v + (int64_t)t * V);
        const char* base = reinterpret_cast<const char*>(a.w) + row0 * row_bytes + (int64_t)s * 8192;
        if (row0 + 4 <= N && 16 * (s + 1) <= J) {
#pragma unroll
            for (int q = 0; q < 4; ++q)
#pragma unroll
                for (int m = 0; m < 8; ++m) dma16<true>(base, doff[m] + 128u * q, wbase + 1024u * (8 * q + m));
        } else {
            // a short last quad or step: absent rows and segments re-read present ones
            // (the same lines as other lanes of the instruction or an earlier one)
            const int rlim = (int)(N - 1 - row0);
            const int jlim = J - 1 - 16 * s;
#pragma unroll
            for (int q = 0; q < 4; ++q)
#pragma unroll
                for (int m = 0; m < 8; ++m) {
                    const int c = 8 * m + (lane >> 3);
                    const int u = (lane & 7) ^ ((c >> 1) & 7);
                    const int r = min(c & 3, rlim), j = min(c >> 2, jlim);
                    const uint32_t voff = (uint32_t)(r * row_bytes) + 512u * (uint32_t)j + 16u * (uint32_t)(8 * q + u);
                    dma16<true>(base, voff, wbase + 1024u * (8 * q + m));
                }
        }
    };

    // ---- x image, fetched by DMA and shared by the waves: 256-byte piece P = x[64P, 64P+64)
    // (of all of x, or of the step's part) at LDS 256P, its 16-byte slot i at slot i ^ (P & 15).
    // Instruction b (1 KB) holds pieces 4b .. 4b+3. ----
    const uint32_t xbase = lds_addr(ximg);
    // XP: part s = x[4096 s, 4096 s + 4096); wave w issues instructions w, w + NW, ... of its 16.
    // Pieces past K (a short last part) copy the part's first piece and are never used.
    auto issue_x = [&](int s) {
        const int P0 = lane >> 4, sl = lane & 15;
#pragma unroll
        for (int i = 0; i < XN; ++i) {
            const int bb = wave + NW * i;
            const int P = 4 * bb + P0;
            const int64_t e0 = 4096 * (int64_t)s + 64 * P;
            const int64_t src = e0 < K ? e0 : 4096 * (int64_t)s;
            dma16(a.x, (uint32_t)(4 * src + 16 * (sl ^ (P & 15))), xbase + 1024u * (uint32_t)bb);
        }
    };
    // XP: every wave of the workgroup walks as many quads as its first wave owns (the most)
    const int nq_wg = XP ? (int)a.qbase + ((int64_t)g * NW < a.qrem ? 1 : 0) : nq;
    if constexpr (XP) {
        if (nq_wg > 0) issue_x(0);
        if (nq > 0) {
            issue(0, 0);
            vmcnt_wait<32>();     // this wave's part of x (issued first) has landed
        } else {
            vmcnt_wait<0>();
        }
    } else {
        const int nxi = (int)(K >> 8);
        const int P0 = lane >> 4, sl = lane & 15;
        for (int b = wave; b < nxi; b += NW) {
            const int P = 4 * b + P0;
            dma16(a.x, (uint32_t)(256 * P + 16 * (sl ^ (P & 15))), xbase + 1024u * (uint32_t)b);
        }
        if (nq > 0) {
            issue(0, 0);
            vmcnt_wait<32>();     // this wave's x instructions (issued first) have landed
        } else {
            vmcnt_wait<0>();
        }
    }
    __syncthreads();          // the x image is in LDS

    // lane c reads x piece P (segment P / 4, part P % 4) into X[0..63]
    float X[64];
    auto load_x = [&](int P) {
        const uint8_t* xp = ximg + 256 * P;
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            const float4 t4 = *reinterpret_cast<const float4*>(xp + 16 * (i ^ (lane & 15)));
            X[4 * i + 0] = t4.x;
            X[4 * i + 1] = t4.y;
            X[4 * i + 2] = t4.z;
            X[4 * i + 3] = t4.w;
        }
    };
    if constexpr (!XP) load_x(lane);   // one step covers K: the same x every step

    const int sw = (lane >> 1) & 7;
    const uint8_t* rd = &wslot[wave][128 * lane];
    float yrun = 0.0f;   // lanes 0..3: running fold of row `lane` of the current quad

    for (int t = 0; t < nq_wg; ++t) {
        for (int s = 0; s < S; ++s) {
            const bool act = t < nq;                              // this wave has a quad at round t
            const bool more = act && ((s + 1 < S) || (t + 1 < nq));
            bool xn = false;                                      // XP: the next step's x was requested
            if constexpr (XP) {
                load_x(lane);                                     // piece `lane` of the step's part
                __syncthreads();                                  // every wave has read the image
                xn = (s + 1 < S) || (t + 1 < nq_wg);
                if (xn) issue_x(s + 1 < S ? s + 1 : 0);
            }
            if (act) {
                float acc = 0.0f;
                auto chain8 = [&](auto qc, const uint4& p, int u) {
                    constexpr int q = decltype(qc)::value;
                    const uint32_t d[4] = {p.x, p.y, p.z, p.w};
                    float wv[8];
#pragma unroll
                    for (int h = 0; h < 8; ++h) wv[h] = (h & 1) ? up_hi(d[h >> 1]) : up_lo(d[h >> 1]);
                    fmac8_bcast<q>(acc, &X[8 * u], wv);
                };
                if (more) {
                    // whole step to registers, request the next one into the freed slot, then the
                    // chains (the step's DMA is everything but the x part issued after it)
                    if (xn) vmcnt_wait<XN>();
                    else vmcnt_wait<0>();
                    uint4 wp[32];
#pragma unroll
                    for (int i = 0; i < 32; ++i)
                        wp[i] = *reinterpret_cast<const uint4*>(rd + 8192 * (i >> 3) + 16 * ((i & 7) ^ sw));
                    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
                    issue(s + 1 < S ? t : t + 1, s + 1 < S ? s + 1 : 0);
#pragma unroll
                    for (int u = 0; u < 8; ++u) chain8(std::integral_constant<int, 0>{}, wp[u], u);
#pragma unroll
                    for (int u = 0; u < 8; ++u) chain8(std::integral_constant<int, 1>{}, wp[8 + u], u);
#pragma unroll
                    for (int u = 0; u < 8; ++u) chain8(std::integral_constant<int, 2>{}, wp[16 + u], u);
#pragma unroll
                    for (int u = 0; u < 8; ++u) chain8(std::integral_constant<int, 3>{}, wp[24 + u], u);
                } else {
                    // this wave's last step: consume each quarter as its 8 DMA instructions land
                    // (at most 8 * (3 - q) of the step's instructions outstanding, plus an x part
                    // issued after them; later operations only add slack)
                    auto quarter = [&](auto qc) {
                        constexpr int q = decltype(qc)::value;
                        if (xn) vmcnt_wait<8 * (3 - q) + (XP ? XN : 0)>();
                        else vmcnt_wait<8 * (3 - q)>();
                        uint4 wp[8];
#pragma unroll
                        for (int u = 0; u < 8; ++u)
                            wp[u] = *reinterpret_cast<const uint4*>(rd + 8192 * q + 16 * (u ^ sw));
#pragma unroll
                        for (int u = 0; u < 8; ++u) chain8(qc, wp[u], u);
                    };
                    quarter(std::integral_constant<int, 0>{});
                    quarter(std::integral_constant<int, 1>{});
                    quarter(std::integral_constant<int, 2>{});
                    quarter(std::integral_constant<int, 3>{});
                }

                if constexpr (!XP) {
                    // one step per quad: keep the quad's 64 partials and fold FB quads at once,
                    // lane 4 qq + r taking row r of the batch's quad qq (16 partials, ascending)
                    const int fq = t % FB;
                    fold[wave][fq][16 * (lane & 3) + (lane >> 2)] = acc;
                    if (fq == FB - 1 || t == nq - 1) {
                        __builtin_amdgcn_wave_barrier();
                        if (lane < 4 * (fq + 1)) {
                            const int qq = lane >> 2, r = lane & 3;
                            float p[16];
#pragma unroll
                            for (int i = 0; i < 4; ++i) {
                                const float4 t4 = *reinterpret_cast<const float4*>(&fold[wave][qq][16 * r + 4 * i]);
                                p[4 * i + 0] = t4.x;
                                p[4 * i + 1] = t4.y;
                                p[4 * i + 2] = t4.z;
                                p[4 * i + 3] = t4.w;
                            }
                            float y = p[0];
#pragma unroll
                            for (int i = 1; i < 16; ++i) y = y + p[i];
                            const int64_t n = 4 * (v + (int64_t)(t - fq + qq) * V) + r;
                            if (n < N) a.y[n] = a.bias ? y + a.bias[n] : y;
                        }
                        __builtin_amdgcn_wave_barrier();
                    }
                } else {
                    // ascending fold of the step's segment partials into each row's running sum
                    fold[wave][0][16 * (lane & 3) + (lane >> 2)] = acc;
                    __builtin_amdgcn_wave_barrier();
                    if (lane < 4) {
                        float p[16];
#pragma unroll
                        for (int i = 0; i < 4; ++i) {
                            const float4 t4 = *reinterpret_cast<const float4*>(&fold[wave][0][16 * lane + 4 * i]);
                            p[4 * i + 0] = t4.x;
                            p[4 * i + 1] = t4.y;
                            p[4 * i + 2] = t4.z;
                            p[4 * i + 3] = t4.w;
                        }
                        const int jn = min(16, J - 16 * s);
                        float y = (s == 0) ? p[0] : yrun + p[0];
                        if (jn == 16) {
#pragma unroll
                            for (int i = 1; i < 16; ++i) y = y + p[i];
                        } else {
#pragma unroll
                            for (int i = 1; i < 16; ++i)
                                if (i < jn) y = y + p[i];
                        }
                        yrun = y;
                        if (s == S - 1) {
                            const int64_t n = 4 * (v + (int64_t)t * V) + lane;
                            if (n < N) a.y[n] = a.bias ? y + a.bias[n] : y;
                        }
                    }
                    __builtin_amdgcn_wave_barrier();
                }
            }
            if constexpr (XP) {
                // this wave's part of the next x has landed (only the next W step, requested
                // after it, may be outstanding), then every wave's has
                if (xn) {
                    if (more) vmcnt_wait<32>();
                    else vmcnt_wait<0>();
                }
                __syncthreads();
            }
        }
    }
}

// ---------------------------------------------------------------------------
// skinny kernel (M >= 1, K % 8 == 0): x shared by the 16 lanes of a DPP row.
//
// Work split.  W rows come in groups of 16 and K in groups of 4 segments.  A
// wave works on one (row group, segment group) pair at a time: lane 16d + i
// runs the chains of row 16 rg + i over segment 4 sg + d for the MT rows of x
// that its workgroup's slice holds.  The 16 lanes of DPP row d share a segment,
// so they share its x: lane i holds x[m][256 j + 16 i .. + 16) for each of the
// MT rows, and the FMA that needs element 16 i + e reads it from lane i with a
// row broadcast (row_newbcast) fused into v_fmac_f32.  x thus costs 16 MT
// registers per segment group, a quarter of what a quad broadcast needs, and
// the kernel runs two waves per SIMD.  Wave w of a workgroup of NW owns the
// segment groups w, w + NW, ... (at most SPW of them, their x loaded once) and
// the workgroup walks row groups g, g + G, ...; every segment group of a row
// group is therefore computed inside one workgroup.
//
// Data path.  A step is 64 weights of each lane's chain: 16 rows x 4 segments
// x 128 bytes = 8 KB, requested with 8 global->LDS DMA instructions (8 lanes
// per 128-byte line) into a ring of DEPTH slots per wave.  The lane's 128-byte
// image is XOR-swizzled by ((lane >> 1) & 7) in 16-byte units so that the
// transposing ds_read_b128 are conflict-free; the step is read to registers,
// the next-but-DEPTH step is requested into the freed slot, and the FMAs run
// with DEPTH steps in flight.  All loads in flight in the stream are DMA loads
// of the wave, which complete in issue order.
//
// Order.  A chain starts at +0 and runs its segment's weights in ascending k
// (a short last segment stops at K).  Its partial goes to LDS; after the row
// group's barrier one thread per (row of x, row of W) folds the J partials in
// ascending segment order, adds b[n] for the bias variant and stores y.
//
// Slices.  With more than MT rows of x the grid holds ceil(M / MT) slices of
// the workgroups; the slices of a row group sit 8 workgroups apart, are
// dispatched to one XCD at about the same time and share its L2 for W.
// ---------------------------------------------------------------------------
constexpr int kSkSlabBytes = 8192;   // one step of a wave: 64 lanes x 128 bytes

// acc[m] = fmaf(x_m[lane L of the row][E0 + h], w[h], acc[m]) for h = 0..3 (outer), m = 0..3
template <int L, int E0>
__device__ __forceinline__ void fmac_nb4(float (&acc)[4], const float (&X)[4][16], const float* w) {
#define RG_G(A, X, W) "v_fmac_f32_dpp %" #A ", %" #X ", %" #W " row_newbcast:%24 row_mask:0xf bank_mask:0xf\n\t"
    asm("s_nop 1\n\t"
        RG_G(0, 4, 20) RG_G(1, 8, 20) RG_G(2, 12, 20) RG_G(3, 16, 20)
        RG_G(0, 5, 21) RG_G(1, 9, 21) RG_G(2, 13, 21) RG_G(3, 17, 21)
        RG_G(0, 6, 22) RG_G(1, 10, 22) RG_G(2, 14, 22) RG_G(3, 18, 22)
        RG_G(0, 7, 23) RG_G(1, 11, 23) RG_G(2, 15, 23) RG_G(3, 19, 23)
        : "+v"(acc[0]), "+v"(acc[1]), "+v"(acc[2]), "+v"(acc[3])
        : "v"(X[0][E0]), "v"(X[0][E0 + 1]), "v"(X[0][E0 + 2]), "v"(X[0][E0 + 3]),
          "v"(X[1][E0]), "v"(X[1][E0 + 1]), "v"(X[1][E0 + 2]), "v"(X[1][E0 + 3]),
          "v"(X[2][E0]), "v"(X[2][E0 + 1]), "v"(X[2][E0 + 2]), "v"(X[2][E0 + 3]),
          "v"(X[3][E0]), "v"(X[3][E0 + 1]), "v"(X[3][E0 + 2]), "v"(X[3][E0 + 3]),
          "v"(w[0]), "v"(w[1]), "v"(w[2]), "v"(w[3]), "n"(L));
#undef RG_G
}

// the same for one row of x and h = 0..7
template <int L, int E0>
__device__ __forceinline__ void fmac_nb1(float (&acc)[1], const float (&X)[1][16], const float* w) {
#define RG_G(X, W) "v_fmac_f32_dpp %0, %" #X ", %" #W " row_newbcast:%17 row_mask:0xf bank_mask:0xf\n\t"
    asm("s_nop 1\n\t"
        RG_G(1, 9) RG_G(2, 10) RG_G(3, 11) RG_G(4, 12) RG_G(5, 13) RG_G(6, 14) RG_G(7, 15) RG_G(8, 16)
        : "+v"(acc[0])
        : "v"(X[0][E0]), "v"(X[0][E0 + 1]), "v"(X[0][E0 + 2]), "v"(X[0][E0 + 3]),
          "v"(X[0][E0 + 4]), "v"(X[0][E0 + 5]), "v"(X[0][E0 + 6]), "v"(X[0][E0 + 7]),
          "v"(w[0]), "v"(w[1]), "v"(w[2]), "v"(w[3]), "v"(w[4]), "v"(w[5]), "v"(w[6]), "v"(w[7]), "n"(L));
#undef RG_G
}

// the same for two rows of x and h = 0..7
template <int L, int E0>
__device__ __forceinline__ void fmac_nb2(float (&acc)[2], const float (&X)[2][16], const float* w) {
#define RG_G(A, X, W) "v_fmac_f32_dpp %" #A ", %" #X ", %" #W " row_newbcast:%26 row_mask:0xf bank_mask:0xf\n\t"
    asm("s_nop 1\n\t"
        RG_G(0, 2, 18) RG_G(1, 10, 18) RG_G(0, 3, 19) RG_G(1, 11, 19)
        RG_G(0, 4, 20) RG_G(1, 12, 20) RG_G(0, 5, 21) RG_G(1, 13, 21)
        RG_G(0, 6, 22) RG_G(1, 14, 22) RG_G(0, 7, 23) RG_G(1, 15, 23)
        RG_G(0, 8, 24) RG_G(1, 16, 24) RG_G(0, 9, 25) RG_G(1, 17, 25)
        : "+v"(acc[0]), "+v"(acc[1])
        : "v"(X[0][E0]), "v"(X[0][E0 + 1]), "v"(X[0][E0 + 2]), "v"(X[0][E0 + 3]),
          "v"(X[0][E0 + 4]), "v"(X[0][E0 + 5]), "v"(X[0][E0 + 6]), "v"(X[0][E0 + 7]),
          "v"(X[1][E0]), "v"(X[1][E0 + 1]), "v"(X[1][E0 + 2]), "v"(X[1][E0 + 3]),
          "v"(X[1][E0 + 4]), "v"(X[1][E0 + 5]), "v"(X[1][E0 + 6]), "v"(X[1][E0 + 7]),
          "v"(w[0]), "v"(w[1]), "v"(w[2]), "v"(w[3]), "v"(w[4]), "v"(w[5]), "v"(w[6]), "v"(w[7]), "n"(L));
#undef RG_G
}

// the same for eight rows of x and h = 0..1
template <int L, int E0>
__device__ __forceinline__ void fmac_nb8(float (&acc)[8], const float (&X)[8][16], const float* w) {
#define RG_G(A, X, W) "v_fmac_f32_dpp %" #A ", %" #X ", %" #W " row_newbcast:%26 row_mask:0xf bank_mask:0xf\n\t"
    asm("s_nop 1\n\t"
        RG_G(0, 8, 24) RG_G(1, 10, 24) RG_G(2, 12, 24) RG_G(3, 14, 24)
        RG_G(4, 16, 24) RG_G(5, 18, 24) RG_G(6, 20, 24) RG_G(7, 22, 24)
        RG_G(0, 9, 25) RG_G(1, 11, 25) RG_G(2, 13, 25) RG_G(3, 15, 25)
        RG_G(4, 17, 25) RG_G(5, 19, 25) RG_G(6, 21, 25) RG_G(7, 23, 25)
        : "+v"(acc[0]), "+v"(acc[1]), "+v"(acc[2]), "+v"(acc[3]), "+v"(acc[4]), "+v"(acc[5]), "+v"(acc[6]),
          "+v"(acc[7])
        : "v"(X[0][E0]), "v"(X[0][E0 + 1]), "v"(X[1][E0]), "v"(X[1][E0 + 1]),
          "v"(X[2][E0]), "v"(X[2][E0 + 1]), "v"(X[3][E0]), "v"(X[3][E0 + 1]),
          "v"(X[4][E0]), "v"(X[4][E0 + 1]), "v"(X[5][E0]), "v"(X[5][E0 + 1]),
          "v"(X[6][E0]), "v"(X[6][E0 + 1]), "v"(X[7][E0]), "v"(X[7][E0 + 1]),
          "v"(w[0]), "v"(w[1]), "n"(L));
#undef RG_G
}

// The FMAs of piece t (weights 8t .. 8t+7 of the lane's 64) of step s of a segment: segment
// element 64 s + 8 t + h, whose x sits in lane 4 s + t / 2 of the row, register 8 (t & 1) + h.
template <int MT, int S, int T>
__device__ __forceinline__ void sk_piece(float (&acc)[MT], const float (&X)[MT][16], const uint4& p) {
    const uint32_t d[4] = {p.x, p.y, p.z, p.w};
    float wv[8];
#pragma unroll
    for (int h = 0; h < 8; ++h) wv[h] = (h & 1) ? up_hi(d[h >> 1]) : up_lo(d[h >> 1]);
    constexpr int L = 4 * S + T / 2, E0 = 8 * (T & 1);
    if constexpr (MT == 1) {
        fmac_nb1<L, E0>(acc, X, wv);
    } else if constexpr (MT == 2) {
        fmac_nb2<L, E0>(acc, X, wv);
    } else if constexpr (MT == 4) {
        fmac_nb4<L, E0>(acc, X, wv);
        fmac_nb4<L, E0 + 4>(acc, X, &wv[4]);
    } else {
        fmac_nb8<L, E0>(acc, X, wv);
        fmac_nb8<L, E0 + 2>(acc, X, &wv[2]);
        fmac_nb8<L, E0 + 4>(acc, X, &wv[4]);
        fmac_nb8<L, E0 + 6>(acc, X, &wv[6]);
    }
}

// One step: the 8 pieces in order; GUARD: only the first np pieces (a short last segment,
// np the same on the 16 lanes of a row, or 0 on a row past the last segment).
template <int MT, int S, bool GUARD>
__device__ __forceinline__ void sk_step(float (&acc)[MT], const float (&X)[MT][16], const uint4 (&wp)[8], int np) {
    if (!GUARD || np > 0) sk_piece<MT, S, 0>(acc, X, wp[0]);
    if (!GUARD || np > 1) sk_piece<MT, S, 1>(acc, X, wp[1]);
    if (!GUARD || np > 2) sk_piece<MT, S, 2>(acc, X, wp[2]);
    if (!GUARD || np > 3) sk_piece<MT, S, 3>(acc, X, wp[3]);
    if (!GUARD || np > 4) sk_piece<MT, S, 4>(acc, X, wp[4]);
    if (!GUARD || np > 5) sk_piece<MT, S, 5>(acc, X, wp[5]);
    if (!GUARD || np > 6) sk_piece<MT, S, 6>(acc, X, wp[6]);
    if (!GUARD || np > 7) sk_piece<MT, S, 7>(acc, X, wp[7]);
}

template <int MT, int SPW, int DEPTH>
__global__ void __launch_bounds__(512) skinny_kernel(SkinnyArgs a) {
    static_assert(MT == 1 || MT == 2 || MT == 4 || MT == 8, "rows of x per slice");
    static_assert(SPW >= 1 && MT * SPW <= 8, "x registers: 16 * MT * SPW <= 128");
    static_assert(DEPTH >= 2 && DEPTH <= 3, "ring depth");
    extern __shared__ __attribute__((aligned(16))) uint8_t sk_lds[];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int NW = (int)(blockDim.x >> 6);
    const int d = lane >> 4, i = lane & 15;
    const int J = a.J, NSG = a.NSG;
    const int64_t N = a.N, K = a.K, RG = a.RG;
    const int64_t row_bytes = 2 * K;

    // workgroup -> (slice, row-group walker g); slices of one g sit 8 workgroups apart
    int64_t g;
    int slice;
    {
        const int64_t b = blockIdx.x;
        const int S = a.mslices;
        slice = (int)((b >> 3) % S);
        g = ((b >> 3) / S) * 8 + (b & 7);
        if (g >= a.groups) return;                        // padding workgroup: no work
    }
    const int64_t G = a.groups;
    const float* xs = a.x + (int64_t)slice * MT * K;
    float* ys = a.y + (int64_t)slice * MT * N;
    const int64_t Ms = a.M - (int64_t)slice * MT;         // rows of x in this slice (>= 1)
    const int nrg = (int)((RG - g + G - 1) / G);          // row groups of this workgroup
    const int nsg = wave < NSG ? min(SPW, (NSG - 1 - wave) / NW + 1) : 0;   // this wave's segment groups
    const int tpr = 4 * nsg;                              // steps per row group
    const int nsteps = nrg * tpr;

    uint8_t* ring = sk_lds + (size_t)wave * DEPTH * kSkSlabBytes;
    // partials [2][MT][16][JP]: an odd row stride JP puts the 16 rows of a write in distinct banks
    float* part = reinterpret_cast<float*>(sk_lds + (size_t)NW * DEPTH * kSkSlabBytes);
    const int JP = a.JP;
    const uint32_t ring_base = lds_addr(ring);
    const int last_len = (int)(K - (int64_t)(J - 1) * kChunk);   // weights of the last segment

    // DMA roles: instruction t fills consumer lanes 8t .. 8t+7 (row 8 (t & 1) + (lane >> 3) of
    // the group, segment 4 sg + t / 2); this lane brings piece u of that consumer's 64 weights
    const int ic0 = lane >> 3, ic1 = 8 + (lane >> 3);
    const int u0 = (lane & 7) ^ (lane >> 4), u1 = (lane & 7) ^ (4 + (lane >> 4));

    auto row_group = [&](int r) -> int64_t {
        const int64_t rgi = g + (int64_t)r * G;
        return a.reverse ? RG - 1 - rgi : rgi;
    };
    // unclamped DMA offsets of this lane past a step's base: instruction t reads row ic,
    // segment t / 2 of the group, piece u
    uint32_t vo[8];
#pragma unroll
    for (int t = 0; t < 8; ++t)
        vo[t] = (uint32_t)(((t & 1) ? ic1 : ic0) * row_bytes) + 512u * (t >> 1) + 16u * ((t & 1) ? u1 : u0);
    // one slice: the weights are read once, non-temporal; several slices read each row group
    // once per slice, the later ones from L2, so it is kept there
    const bool nt = a.mslices == 1;
    auto issue = [&](int st) {
        const int r = st / tpr;
        const int qs = st - r * tpr;
        const int sg = wave + NW * (qs >> 2), s = qs & 3;
        const int64_t n0 = 16 * row_group(r);
        const char* base = reinterpret_cast<const char*>(a.w) + n0 * row_bytes;
        const int rmax = (int)min((int64_t)15, N - 1 - n0);
        const uint32_t slot = ring_base + (uint32_t)((st % DEPTH) * kSkSlabBytes);
        if (rmax == 15 && (4 * sg + 4 < J || (4 * sg + 4 == J && last_len == kChunk))) {
            const char* sb = base + (int64_t)(4 * sg * kChunk + 64 * s) * 2;
            if (nt) dma8<true>(sb, vo, slot);
            else dma8<false>(sb, vo, slot);
            return;
        }
#pragma unroll
        for (int t = 0; t < 8; ++t) {
            const int row = min((t & 1) ? ic1 : ic0, rmax);
            const int j = min(4 * sg + (t >> 1), J - 1);
            const int jlen = (j == J - 1) ? last_len : kChunk;
            int e = 64 * s + 8 * ((t & 1) ? u1 : u0);
            if (e >= jlen) e = 0;                         // past a short last segment: never read
            const uint32_t voff = (uint32_t)(row * row_bytes) + (uint32_t)(j * (2 * kChunk) + 2 * e);
            if (nt) dma16<true>(base, voff, slot + 1024u * t);
            else dma16<false>(base, voff, slot + 1024u * t);
        }
    };

    // prologue: the first DEPTH steps in flight, then x of this wave's segment groups
#pragma unroll
    for (int st = 0; st < DEPTH; ++st)
        if (st < nsteps) issue(st);
    float X[SPW][MT][16];
#pragma unroll
    for (int q = 0; q < SPW; ++q) {
        const int j = 4 * (wave + NW * q) + d;
        const int64_t kb = (int64_t)j * kChunk + 16 * i;
#pragma unroll
        for (int m = 0; m < MT; ++m)
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                // unconditional load from a clamped address, then zero what is outside x
                const bool ok = q < nsg && j < J && m < Ms && kb + 4 * c + 4 <= K;
                const float4 v = *reinterpret_cast<const float4*>(xs + (ok ? (int64_t)m * K + kb + 4 * c : 0));
                X[q][m][4 * c + 0] = ok ? v.x : 0.0f;
                X[q][m][4 * c + 1] = ok ? v.y : 0.0f;
                X[q][m][4 * c + 2] = ok ? v.z : 0.0f;
                X[q][m][4 * c + 3] = ok ? v.w : 0.0f;
            }
    }
    // Everything issued so far has landed: from here on the only loads this wave has in
    // flight in the stream are its DMA steps (the fold's bias loads are waited for at once).
    vmcnt_wait<0>();

    const uint8_t* rd = ring + 128 * lane;
    const int sw = (lane >> 1) & 7;
    int st = 0;
    for (int r = 0; r < nrg; ++r) {
        const int64_t n0 = 16 * row_group(r);
        const int par = r & 1;
        for (int q = 0; q < nsg; ++q) {
            const int sg = wave + NW * q;
            const int j = 4 * sg + d;
            const int len = j < J ? (j == J - 1 ? last_len : kChunk) : 0;
            // every row of the wave has 4 whole segments here: no guards
            const bool whole = 4 * sg + 4 < J || (4 * sg + 4 == J && last_len == kChunk);
            float acc[MT];
#pragma unroll
            for (int m = 0; m < MT; ++m) acc[m] = 0.0f;
            auto step = [&](auto sc) {
                constexpr int s = decltype(sc)::value;
                const int ahead = min(DEPTH - 1, nsteps - 1 - st);
                if (ahead >= 2) vmcnt_wait<16>();
                else if (ahead == 1) vmcnt_wait<8>();
                else vmcnt_wait<0>();
                const uint8_t* src = rd + (st % DEPTH) * kSkSlabBytes;
                uint4 wp[8];
#pragma unroll
                for (int t = 0; t < 8; ++t) wp[t] = *reinterpret_cast<const uint4*>(src + 16 * (t ^ sw));
                asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
                if (st + DEPTH < nsteps) issue(st + DEPTH);
                const int np = min(8, max(0, (len - 64 * s) / 8));
#define RG_SK_STEP(Q)                                                          \
    if (whole) sk_step<MT, s, false>(acc, X[Q], wp, 8);                        \
    else sk_step<MT, s, true>(acc, X[Q], wp, np);
                if constexpr (SPW == 1) {
                    RG_SK_STEP(0)
                } else if constexpr (SPW == 2) {
                    if (q == 0) { RG_SK_STEP(0) } else { RG_SK_STEP(1) }
                } else {
                    switch (q) {
                        case 0: RG_SK_STEP(0) break;
                        case 1: RG_SK_STEP(1) break;
                        case 2: RG_SK_STEP(2) break;
                        default: RG_SK_STEP(3) break;
                    }
                }
#undef RG_SK_STEP
                ++st;
            };
            step(std::integral_constant<int, 0>{});
            step(std::integral_constant<int, 1>{});
            step(std::integral_constant<int, 2>{});
            step(std::integral_constant<int, 3>{});
            if (j < J) {
#pragma unroll
                for (int m = 0; m < MT; ++m) part[((par * MT + m) * 16 + i) * JP + j] = acc[m];
            }
        }
        __syncthreads();
        // fold: one thread per (row of x, row of W); part[par] is written again only after the
        // next row group's barrier, which every thread reaches after this fold
        for (int o = tid; o < 16 * MT; o += 64 * NW) {
            const int m = o >> 4, ii = o & 15;
            const int64_t n = n0 + ii;
            if (m < Ms && n < N) {
                float v = fold_partials(&part[((par * MT + m) * 16 + ii) * JP], J);
                if (a.bias) v = v + a.bias[n];
                ys[(int64_t)m * N + n] = v;
            }
        }
    }
}

// ---------------------------------------------------------------------------
// stream kernel (M <= MT <= 4; FP32 or BF16 weights): streaming GEMV / skinny GEMM.
//
// Work split.  Rows of W come in blocks of 8; workgroup b takes blocks b, b + G,
// b + 2G, ... and all of K for each, so the grid reads one compact window of W
// at a time and every output is finished inside one workgroup (no atomics, no
// cross-workgroup step).  A step covers the next 4 KB of each of the block's 8
// rows: SEGS = 4 (FP32) or 8 (BF16) segments of 256 weights, 32 KB of W.
//
// Data path.  The 256 threads load a step with coalesced 16-byte loads (one
// wave instruction reads 1 KB of one row), one step ahead into registers, and
// move it to LDS between two barriers.  Piece c (row c / SEGS, segment
// c % SEGS) sits in LDS at a stride of 256 weights + 16 bytes, so the lanes
// that walk the pieces in step read different banks.  x for the step's segments
// and the MT rows is staged the same way (one 1 KB piece per row and segment).
//
// Order.  Wave m < MT computes x row m: its lane c < 8 * SEGS runs the fmaf
// chain of piece c from +0 in ascending k; the SEGS lanes of a row fold the
// step's partials into the row's running sum in ascending segment order (the
// first partial of the row starts the sum), and the row is stored, plus b[n]
// for the bias variant, after the block's last step.
// ---------------------------------------------------------------------------
constexpr int kStreamRows = 8;          // W rows per block

template <int MT, typename WT>
__global__ void __launch_bounds__(256) stream_kernel(StreamArgs a) {
    using WV = WVec<WT>;
    constexpr int EPV = WV::E;                          // weights per 16-byte vector
    constexpr int SEGS = 4096 / (kChunk * (int)sizeof(WT));   // segments per 4 KB row step
    constexpr int NP = kStreamRows * SEGS;              // pieces (chains) per step: 32 or 64
    constexpr int WPAD = kChunk + 16 / (int)sizeof(WT); // LDS weights per piece
    constexpr int XPAD = kChunk + 4;                    // LDS floats per x piece
    constexpr int XV = SEGS * 64 / 256;                 // x float4 loads per thread per row
    static_assert(NP <= 64, "one chain per lane");
    __shared__ __attribute__((aligned(16))) WT wsm[NP * WPAD];
    __shared__ __attribute__((aligned(16))) float xsm[MT * SEGS * XPAD];

    const WT* __restrict__ w = reinterpret_cast<const WT*>(a.w);
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int64_t M = a.M, N = a.N, K = a.K;
    const int J = a.J;
    const int nks = (J + SEGS - 1) / SEGS;              // steps per block
    const int64_t G = gridDim.x;
    const int64_t b = a.reverse ? (int64_t)(gridDim.x - 1 - blockIdx.x) : (int64_t)blockIdx.x;
    const int64_t nrb = (N + kStreamRows - 1) / kStreamRows;
    const int64_t myblocks = b < nrb ? (nrb - 1 - b) / G + 1 : 0;
    const int64_t T = myblocks * nks;

    // this thread's W vector of each row: element e0 of the row's 4 KB step window
    const int e0 = wave * (1024 / (int)sizeof(WT)) + lane * EPV;
    const int wl = (e0 / kChunk) * WPAD + e0 % kChunk;  // its LDS offset inside the row's pieces
    typename WV::V wr[kStreamRows];
    float4 xr[MT][XV];
    auto load = [&](int64_t t) {
        const int64_t rb = b + (t / nks) * G;
        const int64_t k0 = (int64_t)(t % nks) * SEGS * kChunk;
#pragma unroll
        for (int r = 0; r < kStreamRows; ++r) {
            const int64_t n = rb * kStreamRows + r;
            wr[r] = (n < N && k0 + e0 < K) ? load_nt(reinterpret_cast<const typename WV::V*>(w + n * K + k0 + e0))
                                           : WV::zero();
        }
#pragma unroll
        for (int m = 0; m < MT; ++m)
#pragma unroll
            for (int u = 0; u < XV; ++u) {
                const int64_t k = k0 + 4 * (tid + 256 * u);
                xr[m][u] = (m < M && k < K) ? *reinterpret_cast<const float4*>(a.x + m * K + k)
                                            : make_float4(0.f, 0.f, 0.f, 0.f);
            }
    };

    float yrun = 0.0f;   // compute lanes: running fold of row (lane / SEGS) for x row `wave`
    float bval = 0.0f;
    if (T > 0) load(0);
    for (int64_t t = 0; t < T; ++t) {
        __syncthreads();                                    // the previous step's chains are done
#pragma unroll
        for (int r = 0; r < kStreamRows; ++r)
            *reinterpret_cast<typename WV::V*>(&wsm[r * SEGS * WPAD + wl]) = wr[r];
#pragma unroll
        for (int m = 0; m < MT; ++m)
#pragma unroll
            for (int u = 0; u < XV; ++u) {
                const int q = tid + 256 * u;                // float4 q of the x window: segment q / 64
                *reinterpret_cast<float4*>(&xsm[(SEGS * m + q / 64) * XPAD + 4 * (q % 64)]) = xr[m][u];
            }
        __syncthreads();
        const int ks = (int)(t % nks);
        const int c = lane, s = c % SEGS;
        const bool computes = wave < MT && c < NP;
        const bool stores = computes && ks == nks - 1 && s == 0;
        const int64_t n = (b + (t / nks) * G) * kStreamRows + c / SEGS;
        if (stores && a.bias && n < N) bval = a.bias[n];   // issued before the next step's loads
        if (t + 1 < T) load(t + 1);                         // in flight during the chains
        if (computes) {
            const int64_t j = (int64_t)ks * SEGS + s;
            const int len = j < J ? (int)(K - j * kChunk < kChunk ? K - j * kChunk : kChunk) : 0;
            const WT* wp = &wsm[c * WPAD];
            const float* xp = &xsm[(SEGS * wave + s) * XPAD];
            float acc = 0.0f;
            auto piece = [&](int e) {                       // EPV weights at element e of the piece
                const typename WV::V wv = *reinterpret_cast<const typename WV::V*>(wp + e);
                float xv[EPV];
#pragma unroll
                for (int i = 0; i < EPV; i += 4) {
                    const float4 x4 = *reinterpret_cast<const float4*>(xp + e + i);
                    xv[i] = x4.x; xv[i + 1] = x4.y; xv[i + 2] = x4.z; xv[i + 3] = x4.w;
                }
#pragma unroll
                for (int i = 0; i < EPV; ++i) acc = __builtin_fmaf(xv[i], WV::get(wv, i), acc);
            };
            if (len == kChunk) {
#pragma unroll 8
                for (int e = 0; e < kChunk; e += EPV) piece(e);
            } else {
                for (int e = 0; e < len; e += EPV) piece(e);
            }
            // the row's SEGS partials (lanes SEGS*r .. SEGS*r + SEGS-1), folded in order
            float p[SEGS];
            if constexpr (SEGS == 4) {
                p[0] = quad_bcast<0>(acc); p[1] = quad_bcast<1>(acc);
                p[2] = quad_bcast<2>(acc); p[3] = quad_bcast<3>(acc);
            } else {
#pragma unroll
                for (int i = 0; i < SEGS; ++i) p[i] = __shfl(acc, (c & ~(SEGS - 1)) + i, 64);
            }
            const int nseg = J - ks * SEGS;                 // >= 1
            float y = (ks == 0) ? p[0] : yrun + p[0];
#pragma unroll
            for (int i = 1; i < SEGS; ++i)
                if (i < nseg) y = y + p[i];
            yrun = y;
            if (stores && n < N && wave < M) a.y[wave * N + n] = a.bias ? y + bval : y;
        }
    }
}

// ---------------------------------------------------------------------------
// cast kernel (comparison point only: the transient FP32 weight copy)
// ---------------------------------------------------------------------------
__global__ void __launch_bounds__(256) cast_kernel(const uint16_t* __restrict__ w, float* __restrict__ o,
                                                   int64_t count) {
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < count; i += stride) o[i] = up1(w[i]);
}

// ---------------------------------------------------------------------------
// argmax per row, lowest index on ties, NaN never wins.  Comparisons are
// exact, so the result does not depend on the reduction tree.
// ---------------------------------------------------------------------------
__device__ __forceinline__ bool better(float v, int64_t i, float bv, int64_t bi) {
    return (v == v) & ((bi < 0) | (bv != bv) | (v > bv) | ((v == bv) & (i < bi)));
}

constexpr int kArgmaxThreads = 1024;
constexpr int kArgmaxBatch = 16;     // independent loads in flight per thread (4 or 16 bytes each)

__global__ void __launch_bounds__(kArgmaxThreads) argmax_kernel(const float* __restrict__ y, int64_t* __restrict__ out,
                                                                int64_t N) {
    __shared__ float sv[kArgmaxThreads];
    __shared__ int64_t si[kArgmaxThreads];
    const int64_t m = blockIdx.x;
    const float* row = y + m * N;
    float bv = 0.0f;
    int64_t bi = -1;
    constexpr int64_t step = (int64_t)kArgmaxThreads * kArgmaxBatch;
    int64_t n0 = threadIdx.x;
    if (N % 4 == 0 && ((uintptr_t)row & 15) == 0) {
        // 16-byte loads: a row of the 128256-entry LM head is two rounds of 16 loads per thread
        const float4* row4 = reinterpret_cast<const float4*>(row);
        const int64_t N4 = N / 4;
        for (int64_t q0 = threadIdx.x; q0 < N4; q0 += step) {
            float4 v[kArgmaxBatch];
#pragma unroll
            for (int u = 0; u < kArgmaxBatch; ++u) {
                const int64_t q = q0 + (int64_t)u * kArgmaxThreads;
                v[u] = q < N4 ? row4[q] : make_float4(0.f, 0.f, 0.f, 0.f);
            }
#pragma unroll
            for (int u = 0; u < kArgmaxBatch; ++u) {
                const int64_t q = q0 + (int64_t)u * kArgmaxThreads;
                if (q >= N4) continue;
                const float e[4] = {v[u].x, v[u].y, v[u].z, v[u].w};
#pragma unroll
                for (int h = 0; h < 4; ++h) {
                    const bool take = better(e[h], 4 * q + h, bv, bi);   // selects, not branches
                    bv = take ? e[h] : bv;
                    bi = take ? 4 * q + h : bi;
                }
            }
        }
        n0 = N;   // nothing left for the scalar loops
    }
    for (; n0 + (kArgmaxBatch - 1) * kArgmaxThreads < N; n0 += step) {
        float v[kArgmaxBatch];
#pragma unroll
        for (int u = 0; u < kArgmaxBatch; ++u) v[u] = row[n0 + (int64_t)u * kArgmaxThreads];
#pragma unroll
        for (int u = 0; u < kArgmaxBatch; ++u) {
            const int64_t n = n0 + (int64_t)u * kArgmaxThreads;
            if (better(v[u], n, bv, bi)) { bv = v[u]; bi = n; }
        }
    }
    for (int64_t n = n0; n < N; n += kArgmaxThreads) {
        const float v = row[n];
        if (better(v, n, bv, bi)) { bv = v; bi = n; }
    }
    sv[threadIdx.x] = bv;
    si[threadIdx.x] = bi;
    __syncthreads();
    for (int h = kArgmaxThreads / 2; h > 0; h >>= 1) {
        if (threadIdx.x < h) {
            const float v = sv[threadIdx.x + h];
            const int64_t i = si[threadIdx.x + h];
            if (i >= 0 && better(v, i, sv[threadIdx.x], si[threadIdx.x])) {
                sv[threadIdx.x] = v;
                si[threadIdx.x] = i;
            }
        }
        __syncthreads();
    }
    if (threadIdx.x == 0) out[m] = si[0];
}

// ---------------------------------------------------------------------------
// host-side launchers
// ---------------------------------------------------------------------------
template <typename WT>
static hipError_t launch_generic_t(const float* x, const WT* w, const float* bias, float* y, int64_t M, int64_t N,
                                   int64_t K, int grid, int reverse, hipStream_t stream) {
    hipLaunchKernelGGL(generic_kernel<WT>, dim3(grid), dim3(256), 0, stream, x, w, bias, y, M, N, K, reverse);
    return hipGetLastError();
}

hipError_t launch_generic(const float* x, const uint16_t* w, const float* bias, float* y, int64_t M, int64_t N,
                          int64_t K, int grid, int reverse, hipStream_t stream) {
    return launch_generic_t(x, w, bias, y, M, N, K, grid, reverse, stream);
}

hipError_t launch_generic(const float* x, const float* w, const float* bias, float* y, int64_t M, int64_t N,
                          int64_t K, int grid, int reverse, hipStream_t stream) {
    return launch_generic_t(x, w, bias, y, M, N, K, grid, reverse, stream);
}

// Round-major placement is built for MT <= 2 only (the host never asks for it with 4 rows).
template <int MT, int NW, int DEPTH>
static hipError_t launch_decode_t(const DecodeArgs& a, int grid, hipStream_t stream) {
    const size_t dyn = (size_t)a.max_rows_wg * MT * sizeof(float);
    if constexpr (MT <= 2) {
        if (a.round_major) {
            hipLaunchKernelGGL((decode_kernel<MT, NW, DEPTH, true>), dim3(grid), dim3(NW * 64), dyn, stream, a);
            return hipGetLastError();
        }
    } else {
        if (a.round_major) return hipErrorInvalidValue;
    }
    hipLaunchKernelGGL((decode_kernel<MT, NW, DEPTH, false>), dim3(grid), dim3(NW * 64), dyn, stream, a);
    return hipGetLastError();
}

// Pipeline depths whose LDS ring (NW * DEPTH * 8 KB) fits next to the
// partials and results: 3 slabs up to 4 waves, 2 above.  (A depth of 4 is
// not built: its first GPU run, together with another change, faulted, and
// the cause has not been shown.)
template <int MT, int NW>
static hipError_t launch_decode_d(const DecodeArgs& a, int grid, int depth, hipStream_t stream) {
    if (depth == 2) return launch_decode_t<MT, NW, 2>(a, grid, stream);
    if constexpr (NW <= 4) {
        if (depth == 3) return launch_decode_t<MT, NW, 3>(a, grid, stream);
    }
    return hipErrorInvalidValue;
}

template <int MT>
static hipError_t launch_decode_w(const DecodeArgs& a, int grid, int nw, int depth, hipStream_t stream) {
    if constexpr (MT == 4) {   // 4 rows of x in registers: one wave per SIMD at most
        if (nw > 4) return hipErrorInvalidValue;
    }
    switch (nw) {
        case 1: return launch_decode_d<MT, 1>(a, grid, depth, stream);
        case 2: return launch_decode_d<MT, 2>(a, grid, depth, stream);
        case 4: return launch_decode_d<MT, 4>(a, grid, depth, stream);
        case 6: if constexpr (MT < 4) return launch_decode_d<MT, 6>(a, grid, depth, stream); else break;
        case 7: if constexpr (MT < 4) return launch_decode_d<MT, 7>(a, grid, depth, stream); else break;
        default: break;
    }
    return hipErrorInvalidValue;
}

template <int NW, int DEPTH>
static hipError_t launch_decode1_t(const DecodeArgs& a, int grid, hipStream_t stream) {
    const size_t dyn = (size_t)a.max_rows_wg * sizeof(float);
    if (a.round_major) hipLaunchKernelGGL((decode1_kernel<NW, DEPTH, true>), dim3(grid), dim3(NW * 64), dyn, stream, a);
    else hipLaunchKernelGGL((decode1_kernel<NW, DEPTH, false>), dim3(grid), dim3(NW * 64), dyn, stream, a);
    return hipGetLastError();
}

// M == 1 with x streamed through LDS.  Rings of NW * DEPTH * 12 KB: depth 3
// up to 4 waves, depth 2 up to 6 waves.
hipError_t launch_decode1(const DecodeArgs& a, int grid, int nw, int depth, hipStream_t stream) {
    switch (nw * 10 + depth) {
        case 12: return launch_decode1_t<1, 2>(a, grid, stream);
        case 13: return launch_decode1_t<1, 3>(a, grid, stream);
        case 22: return launch_decode1_t<2, 2>(a, grid, stream);
        case 23: return launch_decode1_t<2, 3>(a, grid, stream);
        case 42: return launch_decode1_t<4, 2>(a, grid, stream);
        case 43: return launch_decode1_t<4, 3>(a, grid, stream);
        case 62: return launch_decode1_t<6, 2>(a, grid, stream);
        default: return hipErrorInvalidValue;
    }
}

template <int NW, bool XP>
static hipError_t launch_gemv_t(const GemvArgs& a, int grid, hipStream_t stream) {
    const size_t dyn = 4096 * sizeof(float);   // the x image: all of x (K = 4096) or a step's part
    hipLaunchKernelGGL((gemv_kernel<NW, XP>), dim3(grid), dim3(NW * 64), dyn, stream, a);
    return hipGetLastError();
}

// M == 1 dense stream: 1..4 waves of 32 KB slots beside a 16 KB x image; x
// pieces held in registers for the whole kernel when J == 16, else staged a
// step at a time (1, 2 or 4 waves).
hipError_t launch_gemv(const GemvArgs& a, int grid, int nw, hipStream_t stream) {
    if (a.J == 16) {
        switch (nw) {
            case 1: return launch_gemv_t<1, false>(a, grid, stream);
            case 2: return launch_gemv_t<2, false>(a, grid, stream);
            case 3: return launch_gemv_t<3, false>(a, grid, stream);
            case 4: return launch_gemv_t<4, false>(a, grid, stream);
            default: return hipErrorInvalidValue;
        }
    }
    switch (nw) {
        case 1: return launch_gemv_t<1, true>(a, grid, stream);
        case 2: return launch_gemv_t<2, true>(a, grid, stream);
        case 4: return launch_gemv_t<4, true>(a, grid, stream);
        default: return hipErrorInvalidValue;
    }
}

hipError_t launch_decode(const DecodeArgs& a, int mt, int grid, int nw, int depth, hipStream_t stream) {
    switch (mt) {
        case 1: return launch_decode_w<1>(a, grid, nw, depth, stream);
        case 2: return launch_decode_w<2>(a, grid, nw, depth, stream);
        case 4: return launch_decode_w<4>(a, grid, nw, depth, stream);
        default: return hipErrorInvalidValue;
    }
}

template <typename WT>
static hipError_t launch_tiled_t(const float* x, const WT* w, const float* bias, float* y, int64_t M, int64_t N,
                                 int64_t K, int bm, int bn, int occ, int reverse, hipStream_t stream) {
    const int64_t tiles = ((M + bm - 1) / bm) * ((N + bn - 1) / bn);
    if (tiles > 0x7fffffff) return hipErrorInvalidValue;
    const dim3 grid((unsigned)tiles), block(256);
    if (bm == 128 && bn == 128 && occ == 3) hipLaunchKernelGGL((tiled3_kernel<WT>), grid, block, 0, stream, x, w, bias, y, M, N, K, reverse);
    else if (bm == 128 && bn == 128 && occ == 2) hipLaunchKernelGGL((tiled_kernel<128, 128, WT>), grid, block, 0, stream, x, w, bias, y, M, N, K, reverse);
    else if (bm == 64 && bn == 128) hipLaunchKernelGGL((tiled_kernel<64, 128, WT>), grid, block, 0, stream, x, w, bias, y, M, N, K, reverse);
    else if (bm == 64 && bn == 64) hipLaunchKernelGGL((tiled_kernel<64, 64, WT>), grid, block, 0, stream, x, w, bias, y, M, N, K, reverse);
    else return hipErrorInvalidValue;
    return hipGetLastError();
}

hipError_t launch_tiled(const float* x, const uint16_t* w, const float* bias, float* y, int64_t M, int64_t N, int64_t K,
                        int bm, int bn, int occ, int reverse, hipStream_t stream) {
    return launch_tiled_t(x, w, bias, y, M, N, K, bm, bn, occ, reverse, stream);
}

hipError_t launch_tiled(const float* x, const float* w, const float* bias, float* y, int64_t M, int64_t N, int64_t K,
                        int bm, int bn, int occ, int reverse, hipStream_t stream) {
    return launch_tiled_t(x, w, bias, y, M, N, K, bm, bn, occ, reverse, stream);
}

// Small-M tiles (16 outputs per thread, K shared out over KS = 16 * nt / (bm * bn) groups).
template <typename WT>
static hipError_t launch_ktile_t(const float* x, const WT* w, const float* bias, float* y, int64_t M, int64_t N,
                                 int64_t K, int bm, int bn, int nt, int cn, int reverse, hipStream_t stream) {
    const int64_t tiles = ((M + bm - 1) / bm) * ((N + bn - 1) / bn);
    if (tiles > 0x7fffffff) return hipErrorInvalidValue;
    const dim3 grid((unsigned)tiles);
#define RG_KT(BM, BN, NT, CN) \
    if (bm == BM && bn == BN && nt == NT && cn == CN) { \
        hipLaunchKernelGGL((ktile_kernel<BM, BN, 4 * CN * NT / (BM * BN), NT, WT, CN>), grid, dim3(NT), 0, stream, x, w, bias, \
                           y, M, N, K, reverse); \
        return hipGetLastError(); \
    }
    RG_KT(16, 16, 256, 4) RG_KT(16, 32, 256, 4) RG_KT(16, 64, 256, 4) RG_KT(32, 16, 256, 4) RG_KT(32, 32, 256, 4)
    RG_KT(32, 64, 256, 4) RG_KT(64, 16, 256, 4) RG_KT(64, 32, 256, 4) RG_KT(64, 64, 256, 4)
    RG_KT(16, 16, 512, 4) RG_KT(32, 16, 512, 4) RG_KT(64, 16, 512, 4)
    RG_KT(16, 32, 256, 8) RG_KT(16, 64, 256, 8) RG_KT(32, 32, 256, 8) RG_KT(32, 64, 256, 8) RG_KT(64, 32, 256, 8)
    RG_KT(64, 64, 256, 8)
#undef RG_KT
    return hipErrorInvalidValue;
}

hipError_t launch_ktile(const float* x, const uint16_t* w, const float* bias, float* y, int64_t M, int64_t N, int64_t K,
                        int bm, int bn, int nt, int cn, int reverse, hipStream_t stream) {
    return launch_ktile_t(x, w, bias, y, M, N, K, bm, bn, nt, cn, reverse, stream);
}

hipError_t launch_ktile(const float* x, const float* w, const float* bias, float* y, int64_t M, int64_t N, int64_t K,
                        int bm, int bn, int nt, int cn, int reverse, hipStream_t stream) {
    return launch_ktile_t(x, w, bias, y, M, N, K, bm, bn, nt, cn, reverse, stream);
}

template <typename WT>
static hipError_t launch_stream_t(const StreamArgs& a, int mt, int grid, hipStream_t stream) {
    if (mt == 1) hipLaunchKernelGGL((stream_kernel<1, WT>), dim3(grid), dim3(256), 0, stream, a);
    else if (mt == 2) hipLaunchKernelGGL((stream_kernel<2, WT>), dim3(grid), dim3(256), 0, stream, a);
    else if (mt == 4) hipLaunchKernelGGL((stream_kernel<4, WT>), dim3(grid), dim3(256), 0, stream, a);
    else return hipErrorInvalidValue;
    return hipGetLastError();
}

hipError_t launch_stream(const StreamArgs& a, bool f32_weights, int mt, int grid, hipStream_t stream) {
    return f32_weights ? launch_stream_t<float>(a, mt, grid, stream) : launch_stream_t<uint16_t>(a, mt, grid, stream);
}

template <int MT, int SPW, int DEPTH>
static hipError_t launch_skinny_t(const SkinnyArgs& a, int nw, hipStream_t stream) {
    const size_t dyn = skinny_lds_bytes(MT, nw, DEPTH, a.JP);   // up to the CU's 160 KB, no opt-in needed
    const int64_t blocks = (a.groups + 7) / 8 * 8 * a.mslices;
    if (blocks > 0x7fffffff) return hipErrorInvalidValue;
    hipLaunchKernelGGL((skinny_kernel<MT, SPW, DEPTH>), dim3((unsigned)blocks), dim3(nw * 64), dyn, stream, a);
    return hipGetLastError();
}

template <int MT, int SPW>
static hipError_t launch_skinny_d(const SkinnyArgs& a, int nw, int depth, hipStream_t stream) {
    if (depth == 2) return launch_skinny_t<MT, SPW, 2>(a, nw, stream);
    if (depth == 3) return launch_skinny_t<MT, SPW, 3>(a, nw, stream);
    return hipErrorInvalidValue;
}

// Rows of x per slice (2, 4 or 8) and segment groups per wave (x registers: 16 * mt * spw <= 128).
hipError_t launch_skinny(const SkinnyArgs& a, int mt, int spw, int nw, int depth, hipStream_t stream) {
    if (nw < 1 || nw > 8 || a.JP < a.J || skinny_lds_bytes(mt, nw, depth, a.JP) > 160 * 1024) return hipErrorInvalidValue;
    if ((int64_t)nw * spw < a.NSG) return hipErrorInvalidValue;   // every segment group has a wave
    switch (mt * 10 + spw) {
        case 11: return launch_skinny_d<1, 1>(a, nw, depth, stream);
        case 12: return launch_skinny_d<1, 2>(a, nw, depth, stream);
        case 14: return launch_skinny_d<1, 4>(a, nw, depth, stream);
        case 21: return launch_skinny_d<2, 1>(a, nw, depth, stream);
        case 22: return launch_skinny_d<2, 2>(a, nw, depth, stream);
        case 24: return launch_skinny_d<2, 4>(a, nw, depth, stream);
        case 41: return launch_skinny_d<4, 1>(a, nw, depth, stream);
        case 42: return launch_skinny_d<4, 2>(a, nw, depth, stream);
        case 81: return launch_skinny_d<8, 1>(a, nw, depth, stream);
        default: return hipErrorInvalidValue;
    }
}

hipError_t launch_cast(const uint16_t* w, float* o, int64_t count, hipStream_t stream) {
    int64_t blocks = (count + 255) / 256;
    if (blocks > 65536) blocks = 65536;
    if (blocks < 1) blocks = 1;
    hipLaunchKernelGGL(cast_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, w, o, count);
    return hipGetLastError();
}

hipError_t launch_argmax(const float* y, int64_t* out, int64_t M, int64_t N, hipStream_t stream) {
    hipLaunchKernelGGL(argmax_kernel, dim3((unsigned)M), dim3(kArgmaxThreads), 0, stream, y, out, N);
    return hipGetLastError();
}

}  // namespace rg
