/*
 * rg_attn.h -- C-ABI of a fixed-order decode attention for AMD MI355X (gfx950),
 * part of librg.so.
 *
 * The paper pins the reduction order of the linear layers and names attention
 * as the remaining kernel whose order still depends on the GPU (Evaluation,
 * cross-architecture determinism: the first divergence is the output of a
 * layer's attention).  This is that kernel under the same design rules: IEEE
 * binary32 FMA/add/multiply/divide only (R1), an order that is a function of
 * the shape alone (R2, R3), and per-row arithmetic that does not depend on
 * the batch (R4).  The order below ("RG-ATTN-1") is this library's own
 * definition; the paper gives none.
 *
 * Decode attention: one query token per sequence, grouped-query heads.
 *   q    float32 [B][H][D]                      (the new token's queries)
 *   kc   bfloat16 bits [B][Hkv][Lmax][D]       (key cache; widened exactly, up(b) = bits << 16)
 *   vc   bfloat16 bits [B][Hkv][Lmax][D]       (value cache)
 *   lens int32 [B]: positions 0 .. L_b - 1 are attended, L_b = clamp(lens[b], 0, Lmax)
 *   out  float32 [B][H][D]
 *   query head h reads kv head g = h / (H / Hkv).
 *
 * RG-ATTN-1, for every (b, h), with C = 256:
 *   z_l  = the RG-ORDER-1 dot product of q[b][h] and up(kc[b][g][l]) over d
 *          (segments of 256 along d, each an fmaf chain from +0, folded in
 *          ascending order; for D <= 256 a single chain)
 *   t_l  = z_l * scale                               (one binary32 multiply)
 *   m    = the largest t_l (comparisons are exact, NaN never wins)
 *   e_l  = EXP1(t_l - m)                             (one subtraction, then EXP1)
 *   S    = RG fold over l: S_j = +0, S_j = S_j + e_l for l in [256j, 256j + 256)
 *          ascending, S = S_0 + S_1 + ... ascending
 *   N_d  = RG fold over l: n_j = +0, n_j = fmaf(e_l, up(vc[b][g][l][d]), n_j)
 *          for l ascending in segment j, N_d = n_0 + n_1 + ... ascending
 *   out[b][h][d] = N_d / S                           (one binary32 division)
 * L_b = 0 gives S = N = +0 and out = NaN.
 *
 * EXP1(u), the exponential of RG-ATTN-1 (a definition, written with float
 * constants; every operation is binary32, round to nearest even):
 *   if u is NaN     return u
 *   if u < -87      return +0            (also for u = -inf)
 *   k = rint(u * L2E)                    L2E = 0x1.715476p+0 (log2 e rounded to binary32)
 *   r = fmaf(-k, LN2_HI, u)              LN2_HI = 0x1.62e4p-1 (ln 2 to 16 bits)
 *   r = fmaf(-k, LN2_LO, r)              LN2_LO = 0x1.7f7d1cp-20 (ln 2 - LN2_HI, rounded)
 *   p = c7; p = fmaf(p, r, c_i) for i = 6, 5, ..., 0
 *          c_i = 1/i! rounded to binary32: c0 = c1 = 1, c2 = 0.5, c3 = 0x1.555556p-3,
 *          c4 = 0x1.555556p-5, c5 = 0x1.111112p-7, c6 = 0x1.6c16c2p-10, c7 = 0x1.a01a02p-13
 *   return p * 2^k                       (k is in [-126, 0]; 2^k is exact; the
 *                                         product may round into a subnormal)
 * For u > 0 EXP1 is not used (t_l - m <= 0).
 *
 * The order depends on (B, H, Hkv, D, L_b) only -- not on the kernel grid, the
 * number of compute units, Lmax, other sequences of the batch, or timing.
 *
 * Threading, streams and errors follow include/rg.h (rg_status codes; nothing
 * enqueued on error; asynchronous on `stream`).
 */
#ifndef RG_ATTN_H
#define RG_ATTN_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Bytes of device workspace rg_attn_decode needs for these sizes (scores,
 * segment and row maxima, segment sums and numerators).  Returns 0 for invalid sizes. */
int64_t rg_attn_workspace_size(int64_t B, int64_t H, int64_t Lmax, int64_t D);

/*
 * out = RG-ATTN-1 attention of q over the caches (see above).
 *   q, kc, vc, lens, out, workspace: device pointers (caller-owned); q, out,
 *     workspace 16-byte aligned, kc and vc 16-byte aligned, lens 4-byte aligned
 *   B, H, Hkv >= 1 with H % Hkv == 0 and H / Hkv <= 8;  Lmax >= 1;
 *   D % 8 == 0 and 8 <= D <= 256
 *   scale: multiplies each score after the dot product (e.g. 1/sqrt(D) as a float)
 *   workspace_bytes >= rg_attn_workspace_size(B, H, Lmax, D); its contents on
 *     entry do not matter and are overwritten
 * out must not overlap q, kc, vc, lens or the workspace.  Three or four kernels
 * are enqueued on `stream` (scores and segment maxima; the maximum per row,
 * which for some shapes the next kernel takes itself; exponentials and segment
 * partials; the ascending folds and the division).  Returns RG_OK, or
 * RG_ERR_INVAL / RG_ERR_ALIGN / RG_ERR_ALIAS / RG_ERR_ARCH / RG_ERR_HIP as rg.h.
 */
int rg_attn_decode(const float* q, const uint16_t* kc, const uint16_t* vc, const int32_t* lens, float* out,
                   int64_t B, int64_t H, int64_t Hkv, int64_t Lmax, int64_t D, float scale, void* workspace,
                   int64_t workspace_bytes, void* stream);

/* Largest workspace rg_attn_decode_noalloc serves: 64 MiB (e.g. B = 32 sequences,
 * H = 64 heads, Lmax = 4096, D = 128 needs 48 MiB). */
#define RG_ATTN_SCRATCH_BYTES (64ll << 20)

/*
 * rg_attn_decode without a caller workspace and without any allocation, for
 * callers that cannot allocate device memory (code under HIP graph capture,
 * serving loops, harnesses that forbid hipMalloc).  Same arguments, order,
 * kernels and bits as rg_attn_decode; the workspace is a static device array
 * of RG_ATTN_SCRATCH_BYTES inside librg.so, one per device, held from the first
 * call on a device until the process ends.  Returns RG_ERR_RANGE, enqueueing
 * nothing, when rg_attn_workspace_size(B, H, Lmax, D) exceeds
 * RG_ATTN_SCRATCH_BYTES; otherwise the errors of rg_attn_decode.  Every call on
 * one device shares that array, so calls that may overlap in time on one device
 * (different streams, or host threads without ordering) race and must be
 * serialized by the caller; calls in order on one stream are safe.  Nothing in
 * the array needs to start at any value.
 */
int rg_attn_decode_noalloc(const float* q, const uint16_t* kc, const uint16_t* vc, const int32_t* lens, float* out,
                           int64_t B, int64_t H, int64_t Hkv, int64_t Lmax, int64_t D, float scale, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* RG_ATTN_H */
