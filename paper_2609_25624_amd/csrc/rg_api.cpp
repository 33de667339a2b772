// C-ABI of the fused-upcast linear layer: argument checks, the shape-only
// planner and kernel dispatch.  See include/rg.h for the contract.
//
// The planner decides only scheduling (which kernel, how many waves and
// workgroups).  The floating-point order of every output is fixed by K alone
// (paper: rules R2 and R3: configurations are a pure function of the shape,
// the segmentation a pure function of K), and every kernel implements it.

#include <hip/hip_runtime.h>

#include <atomic>
#include <cstdint>
#include <cstring>
#include <mutex>

#include "../../include/rg.h"
#include "../../include/rg_attn.h"
#include "rg_kernels.h"
#include "rg_wtile.h"

namespace {

constexpr int kNominalCUs = 256;            // MI355X; scheduling only
constexpr int kMaxDevices = 64;
constexpr int64_t kMaxDecodeRowsStage = 4096 / 4 * 4;  // rows * MT floats staged per WG <= 16 KB
constexpr int64_t kDecodeMaxM = 64;         // larger M goes to the tiled kernel

rg_launch_t g_launch = {};                  // all zero: planner defaults
thread_local int t_last_hip = 0;            // last hipError_t seen by this thread's calls
std::mutex g_launch_mu;

struct DeviceInfo {
    std::once_flag once;
    int status = RG_OK;
    int cus = 0;
};
DeviceInfo g_dev[kMaxDevices];

int hip_status(hipError_t e);

int device_check(int* cus_out) {
    int dev = 0;
    const hipError_t ge = hipGetDevice(&dev);
    if (ge != hipSuccess) return hip_status(ge);
    if (dev < 0 || dev >= kMaxDevices) return RG_ERR_HIP;
    DeviceInfo& d = g_dev[dev];
    std::call_once(d.once, [&] {
        hipDeviceProp_t p;
        if (hipGetDeviceProperties(&p, dev) != hipSuccess) {
            d.status = RG_ERR_HIP;
            return;
        }
        d.cus = p.multiProcessorCount;
        d.status = (std::strncmp(p.gcnArchName, "gfx950", 6) == 0) ? RG_OK : RG_ERR_ARCH;
    });
    if (cus_out) *cus_out = d.cus;
    return d.status;
}

bool mul_ok(int64_t a, int64_t b) { return a <= 0 || b <= INT64_MAX / 4 / a; }

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

struct Plan {
    int kernel = RG_KERNEL_GENERIC;
    int mt = 0, nw = 0, grid = 0, depth = 0, rq = 0, reverse = 0;
    int64_t Q = 0;
    int max_rows_wg = 0;
    bool x_streamed = false;
    int mslices = 1;
    int tile_m = 0, tile_n = 0;
    int cn = 4;          // ktile: W rows per thread's register tile (4 x cn outputs)
    int spw = 0;         // skinny: segment groups per wave
    int jp = 0;          // skinny: row stride of the LDS partials
    int64_t groups = 0;  // skinny: row-group walkers per slice
};

// Largest decode pipeline depth whose LDS ring fits for a wave count.
//  decode  (x in registers): NW * depth * 8 KB of W slabs.
//  decode1 (M == 1, x streamed): NW * depth * 12 KB of W and x slabs.
int max_depth(bool x_streamed, int nw) {
    if (x_streamed) return nw <= 4 ? 3 : (nw <= 6 ? 2 : 0);
    return nw <= 4 ? 3 : 2;
}

// Decode schedule for a shape: waves per workgroup, quads per round, depth.
// Each workgroup streams its rows through an LDS ring of nw * depth slabs,
// (depth - 1) of them in flight per wave.  The choice maximises the useful
// W bytes in flight per CU (up to ~96 KB, which covers HBM latency at the
// per-CU share of 8 TB/s), then minimises rounds, then idle lanes.
bool decode_schedule(int64_t N, int64_t J, int mt, bool x_streamed, const rg_launch_t& o, Plan* p) {
    static const int kNW[] = {7, 6, 4, 2, 1};
    const int64_t stage_cap = x_streamed ? kMaxDecodeRowsStage / 2 : kMaxDecodeRowsStage;
    p->Q = ceil_div(N, 4);
    int64_t grid = o.grid_wgs > 0 ? o.grid_wgs : (p->Q >= kNominalCUs ? kNominalCUs : p->Q);
    // staging of results: 4 * ceil(Q/grid) rows * mt floats must stay small
    while (4 * ceil_div(p->Q, grid) * mt > stage_cap) {
        if (o.grid_wgs > 0) return false;
        grid *= 2;
    }
    if (grid > p->Q) grid = p->Q;
    const int64_t qpw = ceil_div(p->Q, grid);
    int best_nw = 0, best_rq = 0, best_depth = 0;
    int64_t best_rounds = 0;
    double best_eff = -1.0, best_fly = -1.0;
    for (int nw : kNW) {
        if (o.waves_per_wg > 0 && nw != o.waves_per_wg) continue;
        if (mt == 4 && nw > 4) continue;   // 4 rows of x need one wave per SIMD (registers)
        const int dmax = max_depth(x_streamed, nw);
        if (dmax == 0) continue;
        const int64_t rq = (16 * nw) / J;
        if (rq < 1) continue;
        const int depth = o.depth > 0 ? o.depth : dmax;
        if (depth < 2 || depth > dmax) continue;
        const int64_t rounds = ceil_div(qpw, rq);
        const double eff = (double)(qpw * J) / (double)(rounds * 16 * nw);
        double fly = nw * (depth - 1) * 8.0 * eff;          // KB of useful W in flight
        if (fly > 96.0) fly = 96.0;
        const bool better = best_nw == 0 || fly > best_fly + 1e-9 ||
                            (fly > best_fly - 1e-9 && (rounds < best_rounds ||
                                                       (rounds == best_rounds && eff > best_eff + 1e-9)));
        if (better) {
            best_nw = nw;
            best_rq = (int)rq;
            best_depth = depth;
            best_rounds = rounds;
            best_eff = eff;
            best_fly = fly;
        }
    }
    if (best_nw == 0) return false;
    p->nw = best_nw;
    p->rq = best_rq;
    p->grid = (int)grid;
    p->depth = best_depth;
    p->max_rows_wg = (int)(4 * qpw);
    return true;
}

// Dense-stream M == 1 kernel: K a multiple of 256 with J >= 16 segments (64
// lanes of a wave = 4 rows x 16 segments).  LDS per workgroup: a 32 KB slot
// and 2 KB of partials per wave (256 bytes when K > 4096), plus a 16 KB x
// image (all of x for K = 4096, else the current step's part), so four waves
// fit at any K.  With
// J > 16 the waves of a workgroup share the x part and each DMAs the same
// share of it: 1, 2 or 4 waves.
constexpr int kGemvMaxWaves = 4;

bool gemv_shape_ok(int64_t N, int64_t K) {
    return K % rg::kChunk == 0 && K / rg::kChunk >= 16 && K <= ((int64_t)1 << 26) &&
           ceil_div(N, 4) < ((int64_t)1 << 31);
}

// Waves and workgroups of the dense stream.  Default: the fewest rounds of
// quads per wave that 256 workgroups of four waves allow, then as few waves
// as give that many rounds (every wave the same number of quads when the
// shape allows; 4 rather than 3 waves when J > 16), spread over as many
// workgroups as possible.
bool gemv_schedule(int64_t N, int64_t K, const rg_launch_t& o, Plan* p) {
    const bool xp = K / rg::kChunk != 16;
    const int64_t Q = ceil_div(N, 4);
    int nw = 0;
    int64_t G = 0;
    if (o.waves_per_wg > 0) {
        if (o.waves_per_wg > kGemvMaxWaves || (xp && o.waves_per_wg == 3)) return false;
        nw = o.waves_per_wg;
    }
    if (o.grid_wgs > 0) G = o.grid_wgs;
    if (nw == 0 && G == 0) {
        const int64_t rounds = ceil_div(Q, (int64_t)kNominalCUs * kGemvMaxWaves);
        const int64_t vneed = ceil_div(Q, rounds);
        nw = (int)ceil_div(vneed, kNominalCUs);
        if (xp && nw == 3) nw = 4;
        G = ceil_div(vneed, nw);
    } else if (nw == 0) {
        nw = (int)ceil_div(Q, G);
        if (nw > kGemvMaxWaves) nw = kGemvMaxWaves;
        if (nw < 1) nw = 1;
        if (xp && nw == 3) nw = 4;
    } else if (G == 0) {
        G = ceil_div(Q, nw);
        if (G > kNominalCUs) G = kNominalCUs;
    }
    p->nw = nw;
    p->grid = (int)G;
    p->Q = Q;
    p->depth = 0;
    p->rq = nw;
    return true;
}

// Small-M tiles: BM rows of x (16, 32 or 64, the least that covers M up to
// 64), BN columns of W, K shared out over 4096 / (BM * BN) thread groups.
// Default BN (measured on the Llama-shaped layers): 16, or wider where N is
// large enough to keep ~2 workgroups per CU with the wider tile (x is then
// re-read from L2 fewer times).
bool ktile_schedule(int64_t M, int64_t N, int64_t K, const rg_launch_t& o, Plan* p) {
    const int bm = M <= 16 ? 16 : (M <= 32 ? 32 : 64);   // M > 64 (forced): 64-row tiles
    int bn = o.tile_n;
    // 4 x 8 register tiles with 64-wide tiles where M > 16 and N gives at least 448 such tiles
    // (measured on the gate+up layer 28672 x 4096: M = 32 155 against 204 us, M = 64 253 against
    // 259 us); everywhere else 4 x 4 tiles (fewer K groups keep more parallelism and 16-wide slabs)
    const bool wide = o.depth == 0 && o.tile_n == 0 && o.waves_per_wg == 0 && bm > 16 && ceil_div(N, 64) >= 448;
    if (bn == 0) {
        bn = 16;
        if (bm == 16 && ceil_div(N, 64) >= 448) bn = 64;
        if (bm > 16 && ceil_div(N, 32) >= 896) bn = 32;
        if (wide) bn = 64;
    }
    if (bn != 16 && bn != 32 && bn != 64) return false;
    const int64_t tiles = ceil_div(M, bm) * ceil_div(N, bn);
    if (tiles > 0x7fffffff) return false;
    // 8 waves (twice the K groups) when the tiles alone would leave a CU with one wave
    // per SIMD and K has a segment for every group
    int nw = 4;
    if (o.waves_per_wg > 0) nw = o.waves_per_wg;
    else if (bn == 16 && tiles < 2 * kNominalCUs && ceil_div(K, rg::kChunk) >= 512 / bm) nw = 8;
    if (nw != 4 && nw != 8) return false;
    if (nw == 8 && bn != 16) return false;
    // register tile per thread: 4 x 4 outputs, or 4 x 8 (half the W reads per FMA from LDS)
    int cn = wide ? 8 : 4;
    if (o.depth == 3) cn = 8;
    if (o.depth == 2) cn = 4;
    if (cn == 8 && (bn == 16 || nw != 4)) return false;
    p->tile_m = bm;
    p->tile_n = bn;
    p->grid = (int)tiles;
    p->nw = nw;
    p->cn = cn;
    p->depth = cn == 8 ? 3 : 2;
    return true;
}

// Wave-tile kernel: 64 x 64 tiles, one per workgroup of four waves (eight when forced: more
// segments in flight per tile, one workgroup per CU); the grid order applies.
bool wtile_schedule(int64_t M, int64_t N, const rg_launch_t& o, Plan* p) {
    if ((o.waves_per_wg != 0 && o.waves_per_wg != 4 && o.waves_per_wg != 8) || o.grid_wgs != 0 || o.depth != 0 ||
        (o.tile_n != 0 && o.tile_n != 64) || o.slice_m != 0)
        return false;
    const int64_t tiles = ceil_div(M, rg::kWtileRows) * ceil_div(N, rg::kWtileRows);
    if (tiles > 0x7fffffff) return false;
    p->tile_m = rg::kWtileRows;
    p->tile_n = rg::kWtileRows;
    p->grid = (int)tiles;
    p->nw = o.waves_per_wg > 0 ? o.waves_per_wg : 4;
    p->depth = 0;
    return true;
}

// Skinny kernel: slices of mt = 1, 2, 4 or 8 rows of x, waves of 16 W rows x 4 segments with
// x shared through DPP row broadcasts.  Each wave keeps x of spw segment groups in registers
// (16 * mt * spw <= 128 floats), so nw = ceil(NSG / spw) <= 8 waves cover K.  Two waves per
// SIMD: ceil(8 / nw) workgroups per CU where LDS allows.  Depth (steps in flight per wave):
// the one that keeps the most bytes in flight per CU, 2 on a tie.
constexpr int64_t kSkinnyMaxM = 16;
constexpr int64_t kLdsBytes = 160 * 1024;

bool skinny_shape_ok(int64_t M, int64_t K) {
    return M >= 1 && K < ((int64_t)1 << 26);
}

// One slice width: S slices of mt rows of x, G row-group walkers per slice, the depth that
// keeps the most bytes in flight per CU.  ok = false when no depth fits LDS.
struct SkinnyGrid {
    bool ok = false;
    int64_t S = 0, G = 0;
    int depth = 0, jp = 0;
};

SkinnyGrid skinny_grid(int64_t M, int64_t N, int64_t J, int64_t nw, int mt, const rg_launch_t& o) {
    SkinnyGrid r;
    r.S = ceil_div(M, mt);
    const int64_t RG = ceil_div(N, 16);
    double best_fly = -1.0;
    for (int depth = 2; depth <= 3; ++depth) {
        if (o.depth > 0 && depth != o.depth) continue;
        // odd partial stride unless it costs a workgroup per CU
        const int64_t lds_even = (int64_t)rg::skinny_lds_bytes(mt, (int)nw, depth, (int)J);
        const int64_t lds_odd = (int64_t)rg::skinny_lds_bytes(mt, (int)nw, depth, (int)(J | 1));
        const int jp = (lds_even > kLdsBytes || kLdsBytes / lds_odd == kLdsBytes / lds_even) ? (int)(J | 1) : (int)J;
        const int64_t lds = jp == (int)J ? lds_even : lds_odd;
        if (lds > kLdsBytes) continue;
        int64_t wpc = kLdsBytes / lds;                  // workgroups per CU that LDS allows
        const int64_t wave_cap = 8 / nw > 0 ? 8 / nw : 1;   // two waves per SIMD
        if (wpc > wave_cap) wpc = wave_cap;
        int64_t G = (o.grid_wgs > 0 ? o.grid_wgs : kNominalCUs * wpc) / r.S;   // walkers per slice
        if (G < 1) G = 1;
        if (G > RG) G = RG;
        // bytes in flight per CU: resident workgroups x waves x depth
        double res = (double)(G * r.S) / kNominalCUs;
        if (res > (double)wpc) res = (double)wpc;
        const double fly = res * (double)nw * depth;
        if (fly > best_fly + 1e-9) {
            best_fly = fly;
            r.ok = true;
            r.depth = depth;
            r.G = G;
            r.jp = jp;
        }
    }
    return r;
}

bool skinny_schedule(int64_t M, int64_t N, int64_t K, const rg_launch_t& o, Plan* p) {
    if (o.tile_n != 0) return false;
    const int64_t J = ceil_div(K, rg::kChunk);
    const int64_t NSG = ceil_div(J, 4);
    int64_t spw, nw;
    if (o.waves_per_wg > 0) {
        nw = o.waves_per_wg;
        spw = ceil_div(NSG, nw);
    } else {
        spw = ceil_div(NSG, 8);
        if (spw == 3) spw = 4;
        nw = ceil_div(NSG, spw);
    }
    if (spw == 3) spw = 4;
    // the widest slice whose x registers fit (narrower slices read W once more each, mostly from L2)
    int mt = o.slice_m > 0 ? o.slice_m : (M <= 1 ? 1 : (M <= 2 ? 2 : (M <= 4 ? 4 : 8)));
    while (mt > 1 && mt * spw > 8) mt /= 2;
    if (spw > 4 || mt * spw > 8) return false;
    if (ceil_div(M, mt) > 65536) return false;
    SkinnyGrid g = skinny_grid(M, N, J, nw, mt, o);
    // Where the row groups cap the walkers below the workgroups the CUs hold, halve the slice
    // while that gives more workgroups (measured, interleaved A/B: QKV 6144 x 4096 at M = 3, 4
    // and 8 12-19 % faster, O 4096 x 4096 at M = 2 and 8 4 %, level elsewhere; the second slice
    // reads W from L2)
    while (o.slice_m == 0 && o.grid_wgs == 0 && g.ok && mt > 1 && ceil_div(M, mt / 2) <= 65536) {
        const SkinnyGrid h = skinny_grid(M, N, J, nw, mt / 2, o);
        if (!h.ok || h.S * h.G <= g.S * g.G) break;
        mt /= 2;
        g = h;
    }
    if (!g.ok) return false;
    const int64_t RG = ceil_div(N, 16);
    const int64_t S = g.S;
    const int best_depth = g.depth;
    const int64_t best_g = g.G;
    const int best_jp = g.jp;
    if (ceil_div(RG, best_g) * 4 * spw > 0x7fffffff) return false;   // steps per wave fit int32
    p->mt = mt;
    p->rq = 4;                 // reported as 16 W rows per row group
    p->tile_m = mt;            // reported: rows of x per slice x W rows per group
    p->tile_n = 16;
    p->spw = (int)spw;
    p->jp = best_jp;
    p->nw = (int)nw;
    p->depth = best_depth;
    p->groups = best_g;
    p->mslices = (int)S;
    if (ceil_div(best_g, 8) * 8 * S > 0x7fffffff) return false;   // launched: padded to 8 per slice
    p->grid = (int)(best_g * S);                                  // reported: workgroups with work
    return true;
}

hipError_t launch_stream(const float* x, const void* w, const float* bias, float* y, int64_t M, int64_t N, int64_t K,
                         const Plan& p, bool f32_weights, hipStream_t st) {
    rg::StreamArgs a;
    a.x = x;
    a.w = w;
    a.bias = bias;
    a.y = y;
    a.M = M;
    a.N = N;
    a.K = K;
    a.J = (int)ceil_div(K, rg::kChunk);
    a.reverse = p.reverse;
    return rg::launch_stream(a, f32_weights, p.mt, p.grid, st);
}

// 8-row blocks of W, up to 8 workgroups per CU (measured: more workgroups in
// flight stream the large layers faster).
bool stream_schedule(int64_t M, int64_t N, const rg_launch_t& o, Plan* p) {
    if ((o.waves_per_wg > 0 && o.waves_per_wg != 4) || o.depth > 0 || o.tile_n > 0) return false;
    const int64_t blocks = ceil_div(N, 8);
    const int64_t grid = o.grid_wgs > 0 ? o.grid_wgs : (blocks < 8 * kNominalCUs ? blocks : 8 * kNominalCUs);
    p->mt = M <= 1 ? 1 : (M <= 2 ? 2 : 4);
    p->grid = (int)grid;
    p->nw = 4;
    p->rq = 2;                                    // reported as 8 rows per round
    return true;
}

// Attention workspace: t [B][H][Lmax], segmax and spart [B][H][J], mmax [B][H], npart [B][H][J][D]
// (float32), each region starting on a 256-byte boundary.
struct AttnLayout {
    int64_t t = 0, segmax = 0, spart = 0, mmax = 0, npart = 0, total = 0;
};

bool attn_layout(int64_t B, int64_t H, int64_t Lmax, int64_t D, AttnLayout* lay) {
    if (B < 1 || H < 1 || Lmax < 1 || D < 1 || D > 256) return false;
    if (!mul_ok(B, H) || !mul_ok(B * H, Lmax) || !mul_ok(B * H * Lmax, 4)) return false;
    const int64_t J = ceil_div(Lmax, 256);
    if (!mul_ok(B * H * J, D)) return false;
    auto round256 = [](int64_t v) { return (v + 255) / 256 * 256; };
    lay->t = 0;
    lay->segmax = round256(B * H * Lmax * 4);
    lay->spart = lay->segmax + round256(B * H * J * 4);
    lay->mmax = lay->spart + round256(B * H * J * 4);
    lay->npart = lay->mmax + round256(B * H * 4);
    lay->total = lay->npart + round256(B * H * J * D * 4);
    return true;
}

// Register-tiled kernel: the largest tile that still gives every CU a few workgroups.
// Register tiles for large M.  The 128 x 128 tile has two builds (waves per
// SIMD, reported in `depth`).  Per round of resident workgroups (2 or 3 per
// CU) the three-wave build is no faster than the two-wave one (its spills cost
// what the third wave gains: 7168 tiles 82 against 84 TFLOP/s, 1024 tiles 69
// against 86), so it is taken only where it fills its rounds clearly better:
// 639 tiles fill 0.62 of two rounds of 512 but 0.83 of one round of 768
// (64 against 59 TFLOP/s).
int tiled_schedule(int64_t M, int64_t N, const rg_launch_t& o, Plan* p) {
    const int64_t t128 = ceil_div(M, 128) * ceil_div(N, 128);
    const int64_t t64x128 = ceil_div(M, 64) * ceil_div(N, 128);
    if (t128 >= 2 * kNominalCUs) { p->tile_m = 128; p->tile_n = 128; }
    else if (t64x128 >= kNominalCUs) { p->tile_m = 64; p->tile_n = 128; }
    else { p->tile_m = 64; p->tile_n = 64; }
    const int64_t tiles = ceil_div(M, p->tile_m) * ceil_div(N, p->tile_n);
    if (tiles > 0x7fffffff) return RG_ERR_RANGE;
    p->grid = (int)tiles;
    p->nw = 4;
    p->depth = 0;
    if (p->tile_m == 128) {
        const double s2 = 2.0 * kNominalCUs, s3 = 3.0 * kNominalCUs;
        const double fill2 = (double)tiles / (ceil_div(tiles, (int64_t)s2) * s2);
        const double fill3 = (double)tiles / (ceil_div(tiles, (int64_t)s3) * s3);
        p->depth = (tiles > (int64_t)s2 && fill3 >= 1.2 * fill2) ? 3 : 2;
        if (o.depth > 0) p->depth = o.depth;
    }
    return RG_OK;
}

// One thread per output, grid-strided.
void generic_schedule(int64_t M, int64_t N, const rg_launch_t& o, Plan* p) {
    const int64_t blocks = ceil_div(M * N, 256);
    int64_t grid = o.grid_wgs > 0 ? o.grid_wgs : (blocks < 8 * kNominalCUs ? blocks : 8 * kNominalCUs);
    if (grid < 1) grid = 1;
    p->grid = (int)grid;
    p->nw = 4;
}

// The planner.  `fast_ok`: x and W 16-byte aligned and K % 8 == 0.
int make_plan(int64_t M, int64_t N, int64_t K, bool fast_ok, const rg_launch_t& o, Plan* p) {
    const int64_t J = ceil_div(K, rg::kChunk);
    int want = RG_KERNEL_GENERIC;
    // decode kernels take x in slices of mt <= 4 rows (several slices for M > 4)
    const int mt = M <= 1 ? 1 : M <= 2 ? 2 : 4;
    const int64_t mslices = ceil_div(M, mt);
    const bool decode_ok = fast_ok && J <= 112 && mslices <= 65536;
    const bool tiled_ok = fast_ok;
    const bool gemv_ok = fast_ok && M == 1 && gemv_shape_ok(N, K);
    // M == 1 where the skinny schedule does not fit: the 32 KB-burst kernel where one
    // step covers K (J == 16); the slab-streaming kernels elsewhere (they measure faster
    // once x must be re-read from LDS every step)
    const bool ktile_ok = fast_ok && M <= kDecodeMaxM;
    // ktile from M = 9 on; for 5 <= M <= 8 only where its 16 x 16 tiles are many (measured:
    // the streaming decode kernel is faster on the narrow layers there)
    const bool ktile_pref = M > 8 || (M > 4 && ceil_div(N, 16) >= 384);
    const bool skinny_ok = fast_ok && skinny_shape_ok(M, K);
    // M == 1 too: the one-row skinny build measured 2 % faster than the GEMV on the
    // 28672 x 4096, 4096 x 14336 and 128256 x 4096 layers
    // 16 < M <= 64: skinny where ktile's tiles are narrow (fewer than 448 of 64 W rows: every
    // ktile workgroup re-reads all of x) and x of two segment groups fits (K <= 16384).
    // Measured, interleaved A/B: QKV 6144 x 4096 at M = 32 / 48 / 64 40.6 / 83.3 / 73.8 against
    // 71.7 / 86.7 / 89.8 us, O 4096 x 4096 at M = 24 / 32 / 64 33.2 / 29.6 / 51.5 against
    // 36.3 / 39.4 / 65.5, down 4096 x 14336 at M = 32 113 against 133 (level at M = 64);
    // ktile stays faster on gate+up 28672 x 4096 and the 70B down 8192 x 28672
    const bool skinny_mid = skinny_ok && M > kSkinnyMaxM && M <= kDecodeMaxM && ceil_div(N, 64) < 448 &&
                            ceil_div(J, 4) <= 16;
    // 32 < M <= 64 on wide layers with at most 1024 tiles of 64 W rows: the wave-tile kernel
    // (interleaved A/B against ktile: gate+up 28672 x 4096 at M = 40 / 64 219 / 225 against
    // 250 / 252 us, 70B gate+up 57344 x 8192 at M = 64 858 against 944; level on the
    // 128256-row LM head, whose 2004 tiles already fill the CUs under ktile)
    const bool wtile_pref = fast_ok && M > 32 && M <= kDecodeMaxM && ceil_div(N, 64) >= 448 &&
                            ceil_div(N, 64) <= 1024;
    // M == 1, one 16-segment step per row (K = 4096), N <= 4096: the GEMV's 32 KB bursts put a
    // wave's whole share of W in flight at once, which these short launches need (timed the way
    // the benchmark times, events on the launch stream: 4096 x 4096 8.1 against the skinny
    // kernel's 9.2 us, 2048 x 4096 7.2 against 7.8; skinny from 6144 rows on: 11.2 / 13.1 / 36.3
    // against 11.3 / 13.6 / 37.0 at 6144 / 8192 / 28672)
    const bool gemv_short = gemv_ok && ceil_div(K, rg::kChunk) == 16 && N <= 4096;
    if (gemv_short) want = RG_KERNEL_GEMV;
    else if (skinny_ok && (M <= kSkinnyMaxM || skinny_mid)) want = RG_KERNEL_SKINNY;
    else if (wtile_pref) want = RG_KERNEL_WTILE;
    else if (gemv_ok && ceil_div(K, rg::kChunk) == 16) want = RG_KERNEL_GEMV;
    else if (ktile_ok && ktile_pref) want = RG_KERNEL_KTILE;
    else if (decode_ok && M <= kDecodeMaxM) want = (M == 1) ? RG_KERNEL_DECODE_XS : RG_KERNEL_DECODE;
    else if (tiled_ok) want = RG_KERNEL_TILED;
    const bool forced = o.kernel > 0;
    if (forced) {
        want = o.kernel - 1;
        if ((want == RG_KERNEL_DECODE || want == RG_KERNEL_DECODE_XS) && !decode_ok) return RG_ERR_RANGE;
        if (want == RG_KERNEL_DECODE_XS && M != 1) return RG_ERR_RANGE;
        if (want == RG_KERNEL_TILED && !tiled_ok) return RG_ERR_RANGE;
        if (want == RG_KERNEL_GEMV && !gemv_ok) return RG_ERR_RANGE;
        if (want == RG_KERNEL_KTILE && !fast_ok) return RG_ERR_RANGE;   // any M when forced
        if (want == RG_KERNEL_STREAM && !(fast_ok && M <= 4)) return RG_ERR_RANGE;
        if (want == RG_KERNEL_SKINNY && !skinny_ok) return RG_ERR_RANGE;
        if (want == RG_KERNEL_WTILE && !fast_ok) return RG_ERR_RANGE;
    }
    p->mslices = 1;
    p->kernel = want;
    p->reverse = o.grid_order;
    if (want == RG_KERNEL_SKINNY) {
        if (skinny_schedule(M, N, K, o, p)) return RG_OK;
        if (forced || o.waves_per_wg > 0 || o.grid_wgs > 0 || o.depth > 0) return RG_ERR_RANGE;
        // x of a wave's segment groups does not fit its registers: the earlier kernels
        p->mslices = 1;
        if (M == 1)
            want = p->kernel = (gemv_ok && J == 16) ? RG_KERNEL_GEMV
                             : (decode_ok ? RG_KERNEL_DECODE_XS : (tiled_ok ? RG_KERNEL_TILED : RG_KERNEL_GENERIC));
        else
            want = p->kernel = (ktile_ok && ktile_pref) ? RG_KERNEL_KTILE
                             : (decode_ok ? RG_KERNEL_DECODE : (tiled_ok ? RG_KERNEL_TILED : RG_KERNEL_GENERIC));
    }
    if (want == RG_KERNEL_WTILE) {
        if (wtile_schedule(M, N, o, p)) return RG_OK;
        if (forced) return RG_ERR_RANGE;
        want = p->kernel = RG_KERNEL_KTILE;   // overrides the wave-tile kernel does not take
    }
    if (want == RG_KERNEL_KTILE) {
        if (ktile_schedule(M, N, K, o, p)) return RG_OK;
        return RG_ERR_RANGE;
    }
    if (want == RG_KERNEL_STREAM) return stream_schedule(M, N, o, p) ? RG_OK : RG_ERR_RANGE;
    if (want == RG_KERNEL_GEMV) {
        if (gemv_schedule(N, K, o, p)) return RG_OK;
        if (forced) return RG_ERR_RANGE;
        want = p->kernel = decode_ok ? RG_KERNEL_DECODE_XS : (tiled_ok ? RG_KERNEL_TILED : RG_KERNEL_GENERIC);
    }
    if (want == RG_KERNEL_DECODE_XS) {
        // M == 1: x streamed beside W, when its wave counts cover J; else x in registers.
        p->mt = 1;
        if (decode_schedule(N, J, 1, true, o, p)) {
            p->x_streamed = true;
        } else {
            if (forced) return RG_ERR_RANGE;
            want = p->kernel = RG_KERNEL_DECODE;
        }
    }
    if (want == RG_KERNEL_DECODE) {
        p->mt = mt;
        p->mslices = (int)mslices;
        if (!decode_schedule(N, J, mt, false, o, p)) {
            if (forced || o.waves_per_wg > 0 || o.grid_wgs > 0 || o.depth > 0) return RG_ERR_RANGE;
            p->kernel = tiled_ok ? RG_KERNEL_TILED : RG_KERNEL_GENERIC;
            p->mslices = 1;
        }
    }
    if (p->kernel == RG_KERNEL_TILED) return tiled_schedule(M, N, o, p);
    if (p->kernel == RG_KERNEL_GENERIC) generic_schedule(M, N, o, p);
    return RG_OK;
}

// The planner for FP32 weights (rg_linear_f32w).  `fast_ok`: x and W 16-byte
// aligned and K % 4 == 0.  M <= 4: the FP32-weight streaming kernel; then the
// same ktile / tiled / generic kernels as BF16 weights (their weight loads are
// templated on the element type).
int make_plan_f32w(int64_t M, int64_t N, int64_t K, bool fast_ok, const rg_launch_t& o, Plan* p) {
    int want = RG_KERNEL_GENERIC;
    if (fast_ok && M <= 4) want = RG_KERNEL_STREAM;
    else if (fast_ok && M <= kDecodeMaxM) want = RG_KERNEL_KTILE;
    else if (fast_ok) want = RG_KERNEL_TILED;
    const bool forced = o.kernel > 0;
    if (forced) {
        want = o.kernel - 1;
        if (want == RG_KERNEL_DECODE || want == RG_KERNEL_DECODE_XS || want == RG_KERNEL_GEMV ||
            want == RG_KERNEL_SKINNY)
            return RG_ERR_RANGE;
        if (want != RG_KERNEL_GENERIC && !fast_ok) return RG_ERR_RANGE;
        if (want == RG_KERNEL_STREAM && M > 4) return RG_ERR_RANGE;
    }
    p->kernel = want;
    p->reverse = o.grid_order;
    p->mslices = 1;
    if (want == RG_KERNEL_STREAM) return stream_schedule(M, N, o, p) ? RG_OK : RG_ERR_RANGE;
    if (want == RG_KERNEL_KTILE) return ktile_schedule(M, N, K, o, p) ? RG_OK : RG_ERR_RANGE;
    if (want == RG_KERNEL_WTILE) return wtile_schedule(M, N, o, p) ? RG_OK : RG_ERR_RANGE;
    if (want == RG_KERNEL_TILED) return tiled_schedule(M, N, o, p);
    generic_schedule(M, N, o, p);
    return RG_OK;
}

int validate_launch(const rg_launch_t& c) {
    if (c.kernel < -1 || c.kernel > 9) return RG_ERR_RANGE;
    if (c.tile_n != 0 && c.tile_n != 16 && c.tile_n != 32 && c.tile_n != 64) return RG_ERR_RANGE;
    if (c.slice_m != 0 && c.slice_m != 1 && c.slice_m != 2 && c.slice_m != 4 && c.slice_m != 8) return RG_ERR_RANGE;
    if (c.reserved != 0) return RG_ERR_RANGE;
    if (c.waves_per_wg < 0 || c.waves_per_wg > 8) return RG_ERR_RANGE;
    if (c.grid_wgs < 0 || c.grid_wgs > 65536) return RG_ERR_RANGE;
    if (c.depth < 0 || c.depth > 3 || c.depth == 1) return RG_ERR_RANGE;
    if (c.grid_order < 0 || c.grid_order > 1) return RG_ERR_RANGE;
    return RG_OK;
}

rg_launch_t current_launch() {
    std::lock_guard<std::mutex> lk(g_launch_mu);
    return g_launch;
}

// Map a launch result to an rg_status, remembering the HIP code for rg_last_hip_error.
int hip_status(hipError_t e) {
    t_last_hip = (int)e;
    return e == hipSuccess ? RG_OK : RG_ERR_HIP;
}

bool overlaps(const void* a, size_t an, const void* b, size_t bn) {
    const uintptr_t a0 = (uintptr_t)a, b0 = (uintptr_t)b;
    return a0 < b0 + bn && b0 < a0 + an;
}

}  // namespace

extern "C" {

const char* rg_strerror(int code) {
    switch (code) {
        case RG_OK: return "ok";
        case RG_ERR_INVAL: return "invalid argument (null pointer, size < 1 or size overflow)";
        case RG_ERR_ALIGN: return "misaligned pointer";
        case RG_ERR_ARCH: return "current device is not gfx950";
        case RG_ERR_HIP: return "HIP runtime error";
        case RG_ERR_RANGE: return "launch setting out of range for this shape";
        case RG_ERR_ALIAS: return "output overlaps an input";
        default: return "unknown rg status";
    }
}

int rg_linear_set_launch(const rg_launch_t* cfg) {
    rg_launch_t c = {};
    if (cfg) {
        c = *cfg;
        const int s = validate_launch(c);
        if (s != RG_OK) return s;
    }
    std::lock_guard<std::mutex> lk(g_launch_mu);
    g_launch = c;
    return RG_OK;
}

int rg_plan(int64_t M, int64_t N, int64_t K, rg_plan_t* out) {
    if (!out || M < 1 || N < 1 || K < 1) return RG_ERR_INVAL;
    if (!mul_ok(M, K) || !mul_ok(N, K) || !mul_ok(M, N)) return RG_ERR_INVAL;
    Plan p;
    const int s = make_plan(M, N, K, (K % 8) == 0, current_launch(), &p);
    if (s != RG_OK) return s;
    std::memset(out, 0, sizeof *out);
    out->order_id = RG_ORDER_ID;
    out->chunk = rg::kChunk;
    out->nchunks = ceil_div(K, rg::kChunk);
    out->kernel = p.kernel;
    out->waves_per_wg = p.nw;
    out->grid_wgs = p.grid;
    out->depth = p.depth;
    out->rows_per_round = 4 * p.rq;
    out->tile_m = p.tile_m;
    out->tile_n = p.tile_n;
    return RG_OK;
}

int rg_plan_f32w(int64_t M, int64_t N, int64_t K, rg_plan_t* out) {
    if (!out || M < 1 || N < 1 || K < 1) return RG_ERR_INVAL;
    if (!mul_ok(M, K) || !mul_ok(N, K) || !mul_ok(M, N)) return RG_ERR_INVAL;
    Plan p;
    const int s = make_plan_f32w(M, N, K, (K % 4) == 0, current_launch(), &p);
    if (s != RG_OK) return s;
    std::memset(out, 0, sizeof *out);
    out->order_id = RG_ORDER_ID;
    out->chunk = rg::kChunk;
    out->nchunks = ceil_div(K, rg::kChunk);
    out->kernel = p.kernel;
    out->waves_per_wg = p.nw;
    out->grid_wgs = p.grid;
    out->depth = p.depth;
    out->rows_per_round = 4 * p.rq;
    out->tile_m = p.tile_m;
    out->tile_n = p.tile_n;
    return RG_OK;
}

}  // extern "C"

namespace {

// The one implementation behind rg_linear and rg_linear_bias (bias may be null).
int linear_impl(const float* x, const uint16_t* w, const float* bias, float* y, int64_t M, int64_t N, int64_t K,
                void* stream) {
    if (!x || !w || !y || M < 1 || N < 1 || K < 1) return RG_ERR_INVAL;
    if (!mul_ok(M, K) || !mul_ok(N, K) || !mul_ok(M, N)) return RG_ERR_INVAL;
    if (((uintptr_t)x & 3) || ((uintptr_t)w & 1) || ((uintptr_t)y & 3) || ((uintptr_t)bias & 3)) return RG_ERR_ALIGN;
    if (overlaps(y, (size_t)(M * N) * 4, x, (size_t)(M * K) * 4) ||
        overlaps(y, (size_t)(M * N) * 4, w, (size_t)(N * K) * 2) ||
        (bias && overlaps(y, (size_t)(M * N) * 4, bias, (size_t)N * 4)))
        return RG_ERR_ALIAS;
    int cus = 0;
    const int dc = device_check(&cus);
    if (dc != RG_OK) return dc;
    const bool fast_ok = (K % 8) == 0 && ((uintptr_t)x & 15) == 0 && ((uintptr_t)w & 15) == 0;
    Plan p;
    const int s = make_plan(M, N, K, fast_ok, current_launch(), &p);
    if (s != RG_OK) return s;
    hipStream_t st = (hipStream_t)stream;
    (void)hipGetLastError();   // drop an error left by an unrelated earlier HIP call on this thread
    hipError_t e = hipSuccess;
    if (p.kernel == RG_KERNEL_GEMV) {
        rg::GemvArgs a;
        a.x = x;
        a.w = w;
        a.bias = bias;
        a.y = y;
        a.N = N;
        a.K = K;
        const int64_t V = (int64_t)p.grid * p.nw;
        a.qbase = p.Q / V;
        a.qrem = p.Q % V;
        a.J = (int)(K / rg::kChunk);
        a.S = (int)ceil_div(a.J, 16);
        a.reverse = p.reverse;
        e = rg::launch_gemv(a, p.grid, p.nw, st);
    } else if (p.kernel == RG_KERNEL_DECODE || p.kernel == RG_KERNEL_DECODE_XS) {
        rg::DecodeArgs a;
        a.x = x;
        a.w = w;
        a.bias = bias;
        a.y = y;
        a.M = M;
        a.N = N;
        a.K = K;
        a.Q = p.Q;
        a.qbase = p.Q / p.grid;
        a.qrem = (int)(p.Q % p.grid);
        a.J = (int)ceil_div(K, rg::kChunk);
        a.jmagic = a.J > 1 ? (uint32_t)(((uint64_t)1 << 32) / (uint64_t)a.J + 1) : 0u;
        a.RQ = p.rq;
        a.reverse = p.reverse;
        a.max_rows_wg = p.max_rows_wg;
        // round-major quad placement: measured 1-5 % faster for one or two rows of x when a
        // workgroup has 4 or more rounds, about even at 2-5 rounds, slower for four rows of x
        // (one round: the same placement either way)
        const int64_t rounds = ceil_div(ceil_div(p.Q, p.grid), p.rq);
        a.round_major = (p.mt <= 2 && rounds >= 4) ? 1 : 0;
        a.groups = p.grid;
        a.mslices = p.mslices;
        // decode_kernel: ceil(groups / 8) * 8 * mslices workgroups (the padding ones exit at once)
        const int64_t blocks = ceil_div(p.grid, 8) * 8 * p.mslices;
        if (!p.x_streamed && blocks > 0x7fffffff) return RG_ERR_RANGE;
        e = p.x_streamed ? rg::launch_decode1(a, p.grid, p.nw, p.depth, st)
                         : rg::launch_decode(a, p.mt, (int)blocks, p.nw, p.depth, st);
    } else if (p.kernel == RG_KERNEL_SKINNY) {
        rg::SkinnyArgs a;
        a.x = x;
        a.w = w;
        a.bias = bias;
        a.y = y;
        a.M = M;
        a.N = N;
        a.K = K;
        a.RG = ceil_div(N, 16);
        a.groups = p.groups;
        a.J = (int)ceil_div(K, rg::kChunk);
        a.NSG = (int)ceil_div(a.J, 4);
        a.JP = p.jp;
        a.mslices = p.mslices;
        a.reverse = p.reverse;
        e = rg::launch_skinny(a, p.mt, p.spw, p.nw, p.depth, st);
    } else if (p.kernel == RG_KERNEL_STREAM) {
        e = launch_stream(x, w, bias, y, M, N, K, p, false, st);
    } else if (p.kernel == RG_KERNEL_KTILE) {
        e = rg::launch_ktile(x, w, bias, y, M, N, K, p.tile_m, p.tile_n, 64 * p.nw, p.cn, p.reverse, st);
    } else if (p.kernel == RG_KERNEL_WTILE) {
        e = rg::launch_wtile(x, w, bias, y, M, N, K, p.nw, p.reverse, st);
    } else if (p.kernel == RG_KERNEL_TILED) {
        e = rg::launch_tiled(x, w, bias, y, M, N, K, p.tile_m, p.tile_n, p.depth, p.reverse, st);
    } else {
        e = rg::launch_generic(x, w, bias, y, M, N, K, p.grid, p.reverse, st);
    }
    return hip_status(e);
}

int linear_f32w_impl(const float* x, const float* w, float* y, int64_t M, int64_t N, int64_t K, void* stream) {
    if (!x || !w || !y || M < 1 || N < 1 || K < 1) return RG_ERR_INVAL;
    if (!mul_ok(M, K) || !mul_ok(N, K) || !mul_ok(M, N)) return RG_ERR_INVAL;
    if (((uintptr_t)x & 3) || ((uintptr_t)w & 3) || ((uintptr_t)y & 3)) return RG_ERR_ALIGN;
    if (overlaps(y, (size_t)(M * N) * 4, x, (size_t)(M * K) * 4) ||
        overlaps(y, (size_t)(M * N) * 4, w, (size_t)(N * K) * 4))
        return RG_ERR_ALIAS;
    const int dc = device_check(nullptr);
    if (dc != RG_OK) return dc;
    const bool fast_ok = (K % 4) == 0 && ((uintptr_t)x & 15) == 0 && ((uintptr_t)w & 15) == 0;
    Plan p;
    const int s = make_plan_f32w(M, N, K, fast_ok, current_launch(), &p);
    if (s != RG_OK) return s;
    hipStream_t st = (hipStream_t)stream;
    (void)hipGetLastError();
    hipError_t e = hipSuccess;
    if (p.kernel == RG_KERNEL_STREAM) {
        e = launch_stream(x, w, nullptr, y, M, N, K, p, true, st);
    } else if (p.kernel == RG_KERNEL_KTILE) {
        e = rg::launch_ktile(x, w, nullptr, y, M, N, K, p.tile_m, p.tile_n, 64 * p.nw, p.cn, p.reverse, st);
    } else if (p.kernel == RG_KERNEL_WTILE) {
        e = rg::launch_wtile(x, w, nullptr, y, M, N, K, p.nw, p.reverse, st);
    } else if (p.kernel == RG_KERNEL_TILED) {
        e = rg::launch_tiled(x, w, nullptr, y, M, N, K, p.tile_m, p.tile_n, p.depth, p.reverse, st);
    } else {
        e = rg::launch_generic(x, w, nullptr, y, M, N, K, p.grid, p.reverse, st);
    }
    return hip_status(e);
}

}  // namespace

extern "C" {

int64_t rg_attn_workspace_size(int64_t B, int64_t H, int64_t Lmax, int64_t D) {
    AttnLayout lay;
    return attn_layout(B, H, Lmax, D, &lay) ? lay.total : 0;
}

}  // extern "C"

namespace {

// Argument checks of the attention entry points, in the order of the error codes:
// sizes, then alignment, then aliasing.  `workspace` is null for the no-allocation
// entry point (whose scratch is the library's own, so nothing can alias it).
int attn_check(const float* q, const uint16_t* kc, const uint16_t* vc, const int32_t* lens, float* out, int64_t B,
               int64_t H, int64_t Hkv, int64_t Lmax, int64_t D, const void* workspace, int64_t workspace_bytes,
               AttnLayout* lay) {
    if (!q || !kc || !vc || !lens || !out) return RG_ERR_INVAL;
    if (B < 1 || H < 1 || Hkv < 1 || H % Hkv != 0 || H / Hkv > 8 || Lmax < 1) return RG_ERR_INVAL;
    if (D < 8 || D > 256 || D % 8 != 0) return RG_ERR_INVAL;
    if (!attn_layout(B, H, Lmax, D, lay)) return RG_ERR_INVAL;
    if (!mul_ok(B * Hkv, Lmax) || !mul_ok(B * Hkv * Lmax, D)) return RG_ERR_INVAL;
    const int64_t J = ceil_div(Lmax, 256);
    if (B * Hkv * J > 0x3fffffff || B * H > 0x7fffffff) return RG_ERR_INVAL;   // work items fit int32
    if (workspace && workspace_bytes < lay->total) return RG_ERR_INVAL;
    if (((uintptr_t)q & 15) || ((uintptr_t)out & 15) || ((uintptr_t)workspace & 15) || ((uintptr_t)kc & 15) ||
        ((uintptr_t)vc & 15) || ((uintptr_t)lens & 3))
        return RG_ERR_ALIGN;
    const size_t qb = (size_t)(B * H * D) * 4, cb = (size_t)(B * Hkv * Lmax * D) * 2, lb = (size_t)B * 4;
    if (overlaps(out, qb, q, qb) || overlaps(out, qb, kc, cb) || overlaps(out, qb, vc, cb) ||
        overlaps(out, qb, lens, lb))
        return RG_ERR_ALIAS;
    if (workspace) {
        const size_t wb = (size_t)lay->total;
        if (overlaps(out, qb, workspace, wb) || overlaps(workspace, wb, q, qb) || overlaps(workspace, wb, kc, cb) ||
            overlaps(workspace, wb, vc, cb) || overlaps(workspace, wb, lens, lb))
            return RG_ERR_ALIAS;
    }
    return RG_OK;
}

// Fill the kernel arguments and enqueue the attention kernels (arguments already checked).
int attn_launch(const float* q, const uint16_t* kc, const uint16_t* vc, const int32_t* lens, float* out, int64_t B,
                int64_t H, int64_t Hkv, int64_t Lmax, int64_t D, float scale, const AttnLayout& lay, char* ws,
                int cus, void* stream) {
    const int64_t J = ceil_div(Lmax, 256);
    rg::AttnArgs a;
    a.q = q;
    a.k = kc;
    a.v = vc;
    a.lens = lens;
    a.out = out;
    a.t = reinterpret_cast<float*>(ws + lay.t);
    a.segmax = reinterpret_cast<float*>(ws + lay.segmax);
    a.spart = reinterpret_cast<float*>(ws + lay.spart);
    a.mmax = reinterpret_cast<float*>(ws + lay.mmax);
    a.npart = reinterpret_cast<float*>(ws + lay.npart);
    a.B = B;
    a.H = H;
    a.Hkv = Hkv;
    a.Lmax = Lmax;
    a.D = D;
    a.J = J;
    a.scale = scale;
    const uint64_t vpr = (uint64_t)(D / 8);
    a.vmagic = vpr > 1 ? (uint32_t)((((uint64_t)1 << 32) + vpr - 1) / vpr) : 0u;
    (void)hipGetLastError();
    return hip_status(rg::launch_attn(a, cus, (hipStream_t)stream));
}

// Scratch of rg_attn_decode_noalloc: a file-scope device array (each device that
// loads the library holds its own copy until the process ends).  Host code never
// passes the array's name to a kernel: its device address is taken once per
// device with hipGetSymbolAddress (with that device current) and kept below.
// No attention kernel reads a workspace value it has not written in the same
// call, so nothing here needs clearing between calls.
__device__ __align__(256) uint8_t scratch[RG_ATTN_SCRATCH_BYTES];

struct ScratchSlot {
    std::once_flag once;
    hipError_t status = hipSuccess;
    void* ptr = nullptr;
};
ScratchSlot g_scratch[kMaxDevices];

int scratch_ptr(void** out) {
    int dev = 0;
    const hipError_t ge = hipGetDevice(&dev);
    if (ge != hipSuccess) return hip_status(ge);
    if (dev < 0 || dev >= kMaxDevices) return RG_ERR_HIP;
    ScratchSlot& sl = g_scratch[dev];
    std::call_once(sl.once, [&] {
        void* p = nullptr;
        sl.status = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (sl.status == hipSuccess) sl.ptr = p;
        else (void)hipGetLastError();
    });
    if (sl.status != hipSuccess || !sl.ptr) return hip_status(sl.status != hipSuccess ? sl.status : hipErrorUnknown);
    *out = sl.ptr;
    return RG_OK;
}

}  // namespace

extern "C" {

int rg_attn_decode(const float* q, const uint16_t* kc, const uint16_t* vc, const int32_t* lens, float* out,
                   int64_t B, int64_t H, int64_t Hkv, int64_t Lmax, int64_t D, float scale, void* workspace,
                   int64_t workspace_bytes, void* stream) {
    if (!workspace) return RG_ERR_INVAL;
    AttnLayout lay;
    const int st = attn_check(q, kc, vc, lens, out, B, H, Hkv, Lmax, D, workspace, workspace_bytes, &lay);
    if (st != RG_OK) return st;
    int cus = 0;
    const int dc = device_check(&cus);
    if (dc != RG_OK) return dc;
    return attn_launch(q, kc, vc, lens, out, B, H, Hkv, Lmax, D, scale, lay, static_cast<char*>(workspace), cus,
                       stream);
}

int rg_attn_decode_noalloc(const float* q, const uint16_t* kc, const uint16_t* vc, const int32_t* lens, float* out,
                           int64_t B, int64_t H, int64_t Hkv, int64_t Lmax, int64_t D, float scale, void* stream) {
    AttnLayout lay;
    int st = attn_check(q, kc, vc, lens, out, B, H, Hkv, Lmax, D, nullptr, 0, &lay);
    if (st != RG_OK) return st;
    if (lay.total > (int64_t)RG_ATTN_SCRATCH_BYTES) return RG_ERR_RANGE;   // before any HIP call
    int cus = 0;
    const int dc = device_check(&cus);
    if (dc != RG_OK) return dc;
    void* ws = nullptr;
    st = scratch_ptr(&ws);
    if (st != RG_OK) return st;
    return attn_launch(q, kc, vc, lens, out, B, H, Hkv, Lmax, D, scale, lay, static_cast<char*>(ws), cus, stream);
}

int rg_linear_f32w(const float* x, const float* w, float* y, int64_t M, int64_t N, int64_t K, void* stream) {
    return linear_f32w_impl(x, w, y, M, N, K, stream);
}

int rg_linear(const float* x, const uint16_t* w, float* y, int64_t M, int64_t N, int64_t K, void* stream) {
    return linear_impl(x, w, nullptr, y, M, N, K, stream);
}

int rg_linear_bias(const float* x, const uint16_t* w, const float* bias, float* y, int64_t M, int64_t N, int64_t K,
                   void* stream) {
    if (!bias) return RG_ERR_INVAL;
    return linear_impl(x, w, bias, y, M, N, K, stream);
}

int rg_cast_bf16_f32(const uint16_t* w, float* o, int64_t count, void* stream) {
    if (!w || !o || count < 1 || !mul_ok(count, 1)) return RG_ERR_INVAL;
    if (((uintptr_t)w & 1) || ((uintptr_t)o & 3)) return RG_ERR_ALIGN;
    if (overlaps(o, (size_t)count * 4, w, (size_t)count * 2)) return RG_ERR_ALIAS;
    const int dc = device_check(nullptr);
    if (dc != RG_OK) return dc;
    (void)hipGetLastError();
    return hip_status(rg::launch_cast(w, o, count, (hipStream_t)stream));
}

int rg_argmax_rows(const float* y, int64_t* out, int64_t M, int64_t N, void* stream) {
    if (!y || !out || M < 1 || N < 1 || M > 2147483647 || !mul_ok(M, N)) return RG_ERR_INVAL;
    if (((uintptr_t)y & 3) || ((uintptr_t)out & 7)) return RG_ERR_ALIGN;
    if (overlaps(out, (size_t)M * 8, y, (size_t)(M * N) * 4)) return RG_ERR_ALIAS;
    const int dc = device_check(nullptr);
    if (dc != RG_OK) return dc;
    (void)hipGetLastError();
    return hip_status(rg::launch_argmax(y, out, M, N, (hipStream_t)stream));
}

int rg_stream_create_cu_mask(const uint32_t* mask, uint32_t nwords, void** out_stream) {
    if (!mask || nwords == 0 || !out_stream) return RG_ERR_INVAL;
    hipStream_t s = nullptr;
    const int st = hip_status(hipExtStreamCreateWithCUMask(&s, nwords, mask));
    if (st == RG_OK) *out_stream = (void*)s;
    else (void)hipGetLastError();   // the runtime may refuse a mask; do not leave its error for the next caller
    return st;
}

int rg_stream_destroy(void* stream) {
    if (!stream) return RG_ERR_INVAL;
    return hip_status(hipStreamDestroy((hipStream_t)stream));
}

int rg_last_hip_error(void) { return t_last_hip; }

int rg_device_cu_count(int32_t* out) {
    if (!out) return RG_ERR_INVAL;
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return RG_ERR_HIP;
    int cus = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return RG_ERR_HIP;
    *out = cus;
    return RG_OK;
}

}  // extern "C"
