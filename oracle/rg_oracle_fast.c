/*
 * SAME-ORDER VECTORISED CPU ORACLE.  TEST INFRASTRUCTURE ONLY: only the tests
 * (and the script that writes stored digests) load it.  It shares no code
 * with the GPU path.
 *
 * It computes exactly what rg_oracle.c's rg_oracle_linear computes -- the
 * documented order of the paper's method (Design, eq. 2 and rules R1-R4):
 *   p_j = +0, p_j = fma(x[m,k], up(W[n,k]), p_j) for k ascending in segment j
 *   (256-long segments), y = p_0 + p_1 + ... folded left to right --
 * with the same operation sequence for every output element; it only runs
 * sixteen independent outputs (sixteen rows of W) side by side in the lanes
 * of two 8-lane AVX2 registers.  Each lane's operations are binary32 fused
 * multiply-adds (vfmadd: one rounding, IEEE-754 fusedMultiplyAdd) and
 * additions in round-to-nearest-even with subnormals kept (MXCSR FTZ and DAZ
 * are cleared in every thread), in the order above.  Nothing is reordered
 * within an output; outputs differ only in which lane and thread run them.
 *
 * It exists so that the largest workloads (2048-row prefill layers, about
 * 1e12 multiply-adds) can be checked output for output in seconds; the tests
 * pin it bit for bit against the definitional oracle on many shapes.
 *
 * Built with -mavx2 -mfma -ffp-contract=off; rg_oracle_fast_supported()
 * reports whether the host CPU runs it (AVX2 and FMA).
 */
#include <immintrin.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define SEG 256      /* segment length of the documented order */
#define NB 16        /* outputs (rows of W) per block: two 8-lane registers */
#define MB 4         /* rows of x per inner block */
#define MC 128       /* rows of x per task */

int rg_oracle_fast_supported(void) {
    __builtin_cpu_init();
    return __builtin_cpu_supports("avx2") && __builtin_cpu_supports("fma");
}

/* Sixteen rows n0 .. n0+15 of W, widened from bfloat16 and stored k-major:
 * wt[k][i] = up(W[n0 + i][k]); rows past N are zero (their outputs are not stored). */
static void widen_block(const uint16_t* w, float* wt, int64_t n0, int64_t N, int64_t K) {
    for (int i = 0; i < NB; ++i) {
        const int64_t n = n0 + i;
        if (n < N) {
            const uint16_t* wr = w + n * K;
            for (int64_t k = 0; k < K; ++k) {
                const uint32_t u = (uint32_t)wr[k] << 16;
                memcpy(&wt[k * NB + i], &u, 4);
            }
        } else {
            for (int64_t k = 0; k < K; ++k) wt[k * NB + i] = 0.0f;
        }
    }
}

/* Rows m0 .. m0+mb-1 of x (mb <= MB = 4) against the widened block: y[m][n0 .. n0+nv-1].
 * The eight chains (4 rows x 2 registers) are written out so that they stay in registers. */
static void block_rows(const float* x, const float* wt, float* y, int64_t m0, int mb, int64_t n0, int nv,
                       int64_t N, int64_t K) {
    const float* x0 = x + m0 * K;                              /* extra rows repeat row m0 */
    const float* x1 = x + (m0 + (mb > 1 ? 1 : 0)) * K;
    const float* x2 = x + (m0 + (mb > 2 ? 2 : 0)) * K;
    const float* x3 = x + (m0 + (mb > 3 ? 3 : 0)) * K;
    __m256 t00 = _mm256_setzero_ps(), t01 = t00, t10 = t00, t11 = t00, t20 = t00, t21 = t00, t30 = t00, t31 = t00;
    for (int64_t k0 = 0, j = 0; k0 < K; k0 += SEG, ++j) {
        const int64_t k1 = (k0 + SEG < K) ? k0 + SEG : K;
        __m256 p00 = _mm256_setzero_ps(), p01 = p00, p10 = p00, p11 = p00;   /* each chain from +0 */
        __m256 p20 = p00, p21 = p00, p30 = p00, p31 = p00;
        for (int64_t k = k0; k < k1; ++k) {
            const __m256 w0 = _mm256_load_ps(wt + k * NB), w1 = _mm256_load_ps(wt + k * NB + 8);
            const __m256 b0 = _mm256_broadcast_ss(x0 + k), b1 = _mm256_broadcast_ss(x1 + k);
            const __m256 b2 = _mm256_broadcast_ss(x2 + k), b3 = _mm256_broadcast_ss(x3 + k);
            p00 = _mm256_fmadd_ps(b0, w0, p00);
            p01 = _mm256_fmadd_ps(b0, w1, p01);
            p10 = _mm256_fmadd_ps(b1, w0, p10);
            p11 = _mm256_fmadd_ps(b1, w1, p11);
            p20 = _mm256_fmadd_ps(b2, w0, p20);
            p21 = _mm256_fmadd_ps(b2, w1, p21);
            p30 = _mm256_fmadd_ps(b3, w0, p30);
            p31 = _mm256_fmadd_ps(b3, w1, p31);
        }
        if (j == 0) {                                          /* the first partial as it is */
            t00 = p00; t01 = p01; t10 = p10; t11 = p11; t20 = p20; t21 = p21; t30 = p30; t31 = p31;
        } else {                                               /* then ascending, one addition each */
            t00 = _mm256_add_ps(t00, p00); t01 = _mm256_add_ps(t01, p01);
            t10 = _mm256_add_ps(t10, p10); t11 = _mm256_add_ps(t11, p11);
            t20 = _mm256_add_ps(t20, p20); t21 = _mm256_add_ps(t21, p21);
            t30 = _mm256_add_ps(t30, p30); t31 = _mm256_add_ps(t31, p31);
        }
    }
    float out[MB][NB];
    _mm256_storeu_ps(out[0], t00); _mm256_storeu_ps(out[0] + 8, t01);
    _mm256_storeu_ps(out[1], t10); _mm256_storeu_ps(out[1] + 8, t11);
    _mm256_storeu_ps(out[2], t20); _mm256_storeu_ps(out[2] + 8, t21);
    _mm256_storeu_ps(out[3], t30); _mm256_storeu_ps(out[3] + 8, t31);
    for (int r = 0; r < mb; ++r) memcpy(y + (m0 + r) * N + n0, out[r], (size_t)nv * 4);
}

/* y[M][N] for x[M][K] (f32) and W[N][K] (bf16 bits), row-major, on nthreads threads.
 * Returns 0; -1 on an invalid argument; -2 if the CPU lacks AVX2/FMA; -3 if out of memory. */
int rg_oracle_fast_linear(const float* x, const uint16_t* w, float* y, int64_t M, int64_t N, int64_t K,
                          int nthreads) {
    if (M < 0 || N < 0 || K < 1) return -1;
    if (!rg_oracle_fast_supported()) return -2;
    if (M == 0 || N == 0) return 0;
    const int64_t nblocks = (N + NB - 1) / NB, mchunks = (M + MC - 1) / MC, tasks = nblocks * mchunks;
    int fail = 0;
#pragma omp parallel num_threads(nthreads > 0 ? nthreads : 1)
    {
        const unsigned csr = _mm_getcsr();
        _mm_setcsr(csr & ~(0x8000u | 0x0040u | 0x6000u));   /* FTZ, DAZ off; round to nearest */
        float* wt = (float*)aligned_alloc(32, (size_t)((K * NB * 4 + 31) / 32 * 32));
        if (!wt) {
#pragma omp atomic write
            fail = 1;
        }
        int64_t have = -1;                                   /* block currently widened in wt */
#pragma omp for schedule(dynamic, 1)
        for (int64_t t = 0; t < tasks; ++t) {
            if (!wt) continue;
            const int64_t nb = t / mchunks, mc = t % mchunks;
            const int64_t n0 = nb * NB;
            const int nv = (int)((N - n0) < NB ? (N - n0) : NB);
            if (have != nb) {
                widen_block(w, wt, n0, N, K);
                have = nb;
            }
            const int64_t m1 = (mc + 1) * MC < M ? (mc + 1) * MC : M;
            for (int64_t m0 = mc * MC; m0 < m1; m0 += MB) {
                const int mb = (int)((m1 - m0) < MB ? (m1 - m0) : MB);
                block_rows(x, wt, y, m0, mb, n0, nv, N, K);
            }
        }
        free(wt);
        _mm_setcsr(csr);
    }
    return fail ? -3 : 0;
}
