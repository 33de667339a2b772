/*
 * CPU ORACLE for the fixed-order decode attention (RG-ATTN-1).  TEST
 * INFRASTRUCTURE ONLY: only the tests, the smoke check and the CPU-baseline leg
 * of the benchmark may load this library.  It shares no code with the GPU path.
 *
 * The paper leaves attention unpinned and names it the remaining source of
 * cross-GPU differences (Evaluation, cross-architecture determinism); this is
 * the order the library defines for it under the paper's rules R1-R4, written
 * out literally for one (batch, query head) at a time:
 *
 *   z_l  = dot(q, up(k_l)) in RG-ORDER-1 (256-wide segments of d, fmaf chains
 *          from +0, ascending left fold of the segment partials)
 *   t_l  = z_l * scale
 *   m    = max_l t_l                      (NaN never wins)
 *   e_l  = rg_exp1(t_l - m)
 *   S    = segments of 256 positions: S_j = +0; S_j = S_j + e_l ascending;
 *          S = S_0 + S_1 + ... ascending
 *   N_d  = the same segments: n_j = +0; n_j = fmaf(e_l, up(v_l[d]), n_j);
 *          N_d = n_0 + n_1 + ... ascending
 *   out_d = N_d / S
 *
 * rg_exp1 is the exponential that order uses: Cody-Waite reduction by ln 2
 * (split in a 16-bit high part and a rounded low part), the Taylor polynomial
 * of degree 7 with coefficients 1/i! rounded to binary32, in Horner form with
 * fmaf, then a multiply by 2^k.  Binary32 round to nearest even throughout,
 * gradual underflow kept (built with -ffp-contract=off, no fast-math).
 */
#include <math.h>
#include <stdint.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define ATT_CHUNK 256

static float attn_up(uint16_t b) {
    const uint32_t u = (uint32_t)b << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return f;
}

static float pow2i(int k) {            /* 2^k for -126 <= k <= 127 */
    const uint32_t u = (uint32_t)(k + 127) << 23;
    float f;
    memcpy(&f, &u, sizeof f);
    return f;
}

float rg_exp1(float u) {
    if (u != u) return u;
    if (u < -87.0f) return 0.0f;
    const float L2E = 0x1.715476p+0f;      /* log2(e) rounded to binary32 */
    const float LN2_HI = 0x1.62e4p-1f;     /* ln 2 to 16 significant bits */
    const float LN2_LO = 0x1.7f7d1cp-20f;  /* ln 2 - LN2_HI rounded to binary32 */
    const float c[8] = {1.0f, 1.0f, 0.5f, 0x1.555556p-3f, 0x1.555556p-5f, 0x1.111112p-7f, 0x1.6c16c2p-10f,
                        0x1.a01a02p-13f}; /* 1/i! rounded to binary32 */
    const float k = rintf(u * L2E);
    float r = fmaf(-k, LN2_HI, u);
    r = fmaf(-k, LN2_LO, r);
    float p = c[7];
    for (int i = 6; i >= 0; --i) p = fmaf(p, r, c[i]);
    return p * pow2i((int)k);
}

/* out[i] = rg_exp1(u[i]) for i < n. */
void rg_exp1_array(const float* u, float* out, int64_t n) {
    for (int64_t i = 0; i < n; ++i) out[i] = rg_exp1(u[i]);
}

/* One (b, h).  q: D floats; k, v: the kv head's [Lmax][D] cache; e: L floats of scratch. */
static void attn_one(const float* q, const uint16_t* k, const uint16_t* v, int64_t L, int64_t D, float scale,
                     float* e, float* out) {
    float m = -INFINITY;
    for (int64_t l = 0; l < L; ++l) {
        float z = 0.0f;
        int64_t j = 0;
        for (int64_t d0 = 0; d0 < D; d0 += ATT_CHUNK, ++j) {
            const int64_t d1 = (d0 + ATT_CHUNK < D) ? d0 + ATT_CHUNK : D;
            float p = +0.0f;
            for (int64_t d = d0; d < d1; ++d) p = fmaf(q[d], attn_up(k[l * D + d]), p);
            z = (j == 0) ? p : z + p;
        }
        e[l] = z * scale;
        if (e[l] > m) m = e[l];
    }
    for (int64_t l = 0; l < L; ++l) e[l] = rg_exp1(e[l] - m);
    float S = 0.0f;
    for (int64_t l0 = 0, j = 0; l0 < L; l0 += ATT_CHUNK, ++j) {
        const int64_t l1 = (l0 + ATT_CHUNK < L) ? l0 + ATT_CHUNK : L;
        float s = +0.0f;
        for (int64_t l = l0; l < l1; ++l) s = s + e[l];
        S = (j == 0) ? s : S + s;
    }
    for (int64_t d = 0; d < D; ++d) {
        float N = 0.0f;
        for (int64_t l0 = 0, j = 0; l0 < L; l0 += ATT_CHUNK, ++j) {
            const int64_t l1 = (l0 + ATT_CHUNK < L) ? l0 + ATT_CHUNK : L;
            float n = +0.0f;
            for (int64_t l = l0; l < l1; ++l) n = fmaf(e[l], attn_up(v[l * D + d]), n);
            N = (j == 0) ? n : N + n;
        }
        out[d] = N / S;
    }
}

/* out[B][H][D]; scratch: nthreads * Lmax floats provided by the caller.
 * Returns 0, or -1 on invalid sizes. */
int rg_attn_oracle(const float* q, const uint16_t* kc, const uint16_t* vc, const int32_t* lens, float* out,
                   int64_t B, int64_t H, int64_t Hkv, int64_t Lmax, int64_t D, float scale, float* scratch,
                   int nthreads) {
    if (B < 1 || H < 1 || Hkv < 1 || H % Hkv != 0 || Lmax < 1 || D < 1) return -1;
    const int64_t group = H / Hkv;
    const int nt = nthreads > 0 ? nthreads : 1;
#pragma omp parallel for schedule(dynamic, 1) num_threads(nt)
    for (int64_t i = 0; i < B * H; ++i) {
        const int64_t b = i / H, h = i % H, g = h / group;
        int64_t L = lens[b];
        if (L < 0) L = 0;
        if (L > Lmax) L = Lmax;
        int tid = 0;
#ifdef _OPENMP
        tid = omp_get_thread_num();
#endif
        const uint16_t* k = kc + (b * Hkv + g) * Lmax * D;
        const uint16_t* v = vc + (b * Hkv + g) * Lmax * D;
        attn_one(q + (b * H + h) * D, k, v, L, D, scale, scratch + (int64_t)tid * Lmax, out + (b * H + h) * D);
    }
    return 0;
}
