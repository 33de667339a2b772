/*
 * CPU ORACLE for the fused-upcast linear layer.  TEST INFRASTRUCTURE ONLY:
 * only the tests, the smoke check and the CPU-baseline leg of the benchmark
 * may load this library.  It shares no code with the GPU path.
 *
 * What it computes (paper: Design, eq. 2 and rules R1-R4; Supplement C):
 *   y[m,n] = sum_k x[m,k] * up(W[n,k])      (no bias; see the readings below)
 * in ONE fixed floating-point order, written out literally:
 *
 *   up(b)  = the float whose bits are (uint32)b << 16        (exact widening
 *            of a bfloat16 pattern, done in registers: Design, eq. 2)
 *   C      = 256,  J = ceil(K / C)                          (segments are a
 *            pure function of K, rule R3; the segment length is a reading,
 *            the paper never prints its pinned value)
 *   p_j    = +0.0f, then for k = jC .. min(jC+C, K)-1 ascending:
 *               p_j = fmaf(x[m,k], up(W[n,k]), p_j)         (IEEE-754 FMA only,
 *            rule R1; each segment accumulated sequentially in ascending k,
 *            rule R3 and Supplement C on R2)
 *   y      = p_0, then for j = 1 .. J-1 ascending:  y = y + p_j
 *            (partials combined in fixed ascending segment order, rule R3)
 *
 * With a bias (rg_oracle_linear_bias): y[m,n] = (the fold above) + b[n], one
 * binary32 addition after the last segment (Design, eq. 2's "+ b"; the bias
 * never enters a segment chain).
 *
 * With FP32 weights (rg_oracle_linear_f32w; the paper probes BF16 and FP32
 * weights alike, Supplement C): the same segments, chains and fold, with the
 * weight read as the float it is in place of up(W[n,k]).
 *
 * Nothing depends on m, n or M (batch invariance by construction, rule R4).
 * Arithmetic is IEEE-754 binary32, round to nearest even, gradual underflow:
 * this file is compiled with -ffp-contract=off and without fast-math, and
 * fmaf is the C library's correctly rounded fused multiply-add.
 *
 * The FP64 reference (rg_ref_fp64) is NOT the oracle: it is the exact-order-
 * free quantity the oracle is checked against within the standard inner
 * product error bound gamma_n = n*u/(1-n*u), u = 2^-24, n = min(C,K) + J - 1.
 */
#include <math.h>
#include <stdint.h>
#include <string.h>

#define RG_ORACLE_CHUNK 256

static float up_bf16(uint16_t b) {
    const uint32_t u = (uint32_t)b << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return f;
}

/* One output element: x and w are one row each, length K. */
float rg_oracle_dot(const float* x, const uint16_t* w, int64_t K) {
    float y = 0.0f;
    int64_t j = 0;
    for (int64_t k0 = 0; k0 < K; k0 += RG_ORACLE_CHUNK, ++j) {
        const int64_t k1 = (k0 + RG_ORACLE_CHUNK < K) ? k0 + RG_ORACLE_CHUNK : K;
        float p = +0.0f;
        for (int64_t k = k0; k < k1; ++k) p = fmaf(x[k], up_bf16(w[k]), p);
        if (j == 0)
            y = p;
        else
            y = y + p;
    }
    return y;
}

/* y[M][N] for x[M][K] (f32) and W[N][K] (bf16 bits), all row-major.
 * Outputs are independent, so they are spread over nthreads threads; the
 * operation sequence of each output is rg_oracle_dot's.  Returns 0, or -1 on
 * an invalid argument (K < 1, M or N < 0). */
int rg_oracle_linear(const float* x, const uint16_t* w, float* y, int64_t M, int64_t N, int64_t K,
                     int nthreads) {
    if (M < 0 || N < 0 || K < 1) return -1;
    const int64_t total = M * N;
#pragma omp parallel for schedule(dynamic, 64) num_threads(nthreads > 0 ? nthreads : 1)
    for (int64_t i = 0; i < total; ++i) {
        const int64_t m = i / N, n = i % N;
        y[i] = rg_oracle_dot(x + m * K, w + n * K, K);
    }
    return 0;
}

/* y[m][n] = rg_oracle_dot(x_m, w_n) + b[n]: the fold, then one addition. */
int rg_oracle_linear_bias(const float* x, const uint16_t* w, const float* b, float* y, int64_t M, int64_t N,
                          int64_t K, int nthreads) {
    if (M < 0 || N < 0 || K < 1 || !b) return -1;
    const int64_t total = M * N;
#pragma omp parallel for schedule(dynamic, 64) num_threads(nthreads > 0 ? nthreads : 1)
    for (int64_t i = 0; i < total; ++i) {
        const int64_t m = i / N, n = i % N;
        const float d = rg_oracle_dot(x + m * K, w + n * K, K);
        y[i] = d + b[n];
    }
    return 0;
}

/* One output with FP32 weights: rg_oracle_dot's order, w[k] used as it is. */
float rg_oracle_dot_f32w(const float* x, const float* w, int64_t K) {
    float y = 0.0f;
    int64_t j = 0;
    for (int64_t k0 = 0; k0 < K; k0 += RG_ORACLE_CHUNK, ++j) {
        const int64_t k1 = (k0 + RG_ORACLE_CHUNK < K) ? k0 + RG_ORACLE_CHUNK : K;
        float p = +0.0f;
        for (int64_t k = k0; k < k1; ++k) p = fmaf(x[k], w[k], p);
        if (j == 0)
            y = p;
        else
            y = y + p;
    }
    return y;
}

/* y[M][N] for x[M][K] and W[N][K], both float32, row-major. */
int rg_oracle_linear_f32w(const float* x, const float* w, float* y, int64_t M, int64_t N, int64_t K,
                          int nthreads) {
    if (M < 0 || N < 0 || K < 1) return -1;
    const int64_t total = M * N;
#pragma omp parallel for schedule(dynamic, 64) num_threads(nthreads > 0 ? nthreads : 1)
    for (int64_t i = 0; i < total; ++i) {
        const int64_t m = i / N, n = i % N;
        y[i] = rg_oracle_dot_f32w(x + m * K, w + n * K, K);
    }
    return 0;
}

/* FP64 reference with FP32 weights: y64 = sum_k (double)x*(double)w, s = sum_k |x*w|. */
int rg_ref_fp64_f32w(const float* x, const float* w, double* y64, double* abs_sum, int64_t M, int64_t N,
                     int64_t K, int nthreads) {
    if (M < 0 || N < 0 || K < 1) return -1;
    const int64_t total = M * N;
#pragma omp parallel for schedule(dynamic, 64) num_threads(nthreads > 0 ? nthreads : 1)
    for (int64_t i = 0; i < total; ++i) {
        const int64_t m = i / N, n = i % N;
        double acc = 0.0, s = 0.0;
        for (int64_t k = 0; k < K; ++k) {
            const double t = (double)x[m * K + k] * (double)w[n * K + k];
            acc += t;
            s += fabs(t);
        }
        y64[i] = acc;
        abs_sum[i] = s;
    }
    return 0;
}

/* Sampled outputs: out[s] = y[rows[s], cols[s]] for s < count. */
int rg_oracle_linear_sampled(const float* x, const uint16_t* w, int64_t K, const int64_t* rows,
                             const int64_t* cols, int64_t count, float* out, int nthreads) {
    if (K < 1 || count < 0) return -1;
#pragma omp parallel for schedule(dynamic, 16) num_threads(nthreads > 0 ? nthreads : 1)
    for (int64_t s = 0; s < count; ++s) out[s] = rg_oracle_dot(x + rows[s] * K, w + cols[s] * K, K);
    return 0;
}

/* FP64 reference: y64[m][n] = sum_k x*up(w) accumulated in double, and
 * abs_sum[m][n] = sum_k |x*up(w)|.  Each product of a binary32 and a bfloat16
 * value is exact in binary64 (24 + 8 significand bits). */
int rg_ref_fp64(const float* x, const uint16_t* w, double* y64, double* abs_sum, int64_t M, int64_t N,
                int64_t K, int nthreads) {
    if (M < 0 || N < 0 || K < 1) return -1;
    const int64_t total = M * N;
#pragma omp parallel for schedule(dynamic, 64) num_threads(nthreads > 0 ? nthreads : 1)
    for (int64_t i = 0; i < total; ++i) {
        const int64_t m = i / N, n = i % N;
        double s = 0.0, a = 0.0;
        for (int64_t k = 0; k < K; ++k) {
            const double t = (double)x[m * K + k] * (double)up_bf16(w[n * K + k]);
            s += t;
            a += fabs(t);
        }
        y64[i] = s;
        abs_sum[i] = a;
    }
    return 0;
}

/* Greedy decision over one row of logits: the index of the largest value,
 * the lower index on ties (the paper's tie-break: argmax returns the lower
 * token id, Evaluation, end-to-end determinism).  NaN entries never win. */
int64_t rg_oracle_argmax(const float* v, int64_t n) {
    int64_t best = -1;
    for (int64_t i = 0; i < n; ++i) {
        if (v[i] != v[i]) continue;
        if (best < 0 || v[i] > v[best]) best = i;
    }
    return best;
}
