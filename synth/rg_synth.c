/*
 * Seeded synthetic inputs for the fused-upcast linear layer.
 *
 * This module only MAKES inputs.  It holds none of the layer's arithmetic
 * (no upcast, no multiply-accumulate, no reduction): both the CPU oracle and
 * the GPU path consume the bits it writes, exactly as the paper's probes
 * generate inputs on the CPU from a fixed seed and copy them to every device
 * (Evaluation, cross-architecture determinism; Supplement C, method).
 *
 * Generator (counter based, so any element can be produced independently and
 * a tensor with more rows has the smaller tensor as its prefix):
 *   key     = splitmix64(seed ^ (tensor_id * 0x9E3779B97F4A7C15))
 *   r_i     = splitmix64(key + 2*idx + i),  i in {0,1},  idx = row*cols + col
 *   u1      = ((r_0 >> 11) + 1) * 2^-53          in (0, 1]
 *   u2      =  (r_1 >> 11)      * 2^-53          in [0, 1)
 *   z       = sqrt(-2 ln u1) * cos(2 pi u2)      (Box-Muller, in double)
 *   value   = mean + std * z, rounded once to the target format:
 *             float  : C cast (round to nearest even)
 *             bf16   : float bits rounded to nearest even on the top 16 bits
 * splitmix64 is Vigna's published mixer (the SplitMix64 output function).
 */
#include <math.h>
#include <stdint.h>
#include <string.h>

static inline uint64_t splitmix64(uint64_t z) {
    z += 0x9E3779B97F4A7C15ULL;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
    return z ^ (z >> 31);
}

static inline uint64_t stream_key(uint64_t seed, uint64_t tensor_id) {
    return splitmix64(seed ^ (tensor_id * 0x9E3779B97F4A7C15ULL));
}

static inline double normal_at(uint64_t key, uint64_t idx) {
    const uint64_t r0 = splitmix64(key + 2 * idx);
    const uint64_t r1 = splitmix64(key + 2 * idx + 1);
    const double u1 = ((double)((r0 >> 11) + 1)) * 0x1p-53;
    const double u2 = ((double)(r1 >> 11)) * 0x1p-53;
    return sqrt(-2.0 * log(u1)) * cos(6.283185307179586476925286766559 * u2);
}

static inline uint16_t f32_to_bf16_rne(float f) {
    uint32_t u;
    memcpy(&u, &f, 4);
    u += 0x7FFFu + ((u >> 16) & 1u);   /* finite inputs only (Box-Muller never gives inf/nan) */
    return (uint16_t)(u >> 16);
}

/* Raw splitmix64 draws, exposed so a test can pin the generator to its published definition. */
void rg_synth_splitmix64(uint64_t start, int64_t n, uint64_t* out) {
    for (int64_t i = 0; i < n; ++i) out[i] = splitmix64(start + (uint64_t)i);
}

/* out[r*cols + c] = float(mean + std * z(seed, tensor_id, r*cols + c)) for r < rows, c < cols. */
void rg_synth_normal_f32(float* out, int64_t rows, int64_t cols, uint64_t seed,
                         uint64_t tensor_id, double mean, double std) {
    const uint64_t key = stream_key(seed, tensor_id);
    const int64_t n = rows * cols;
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) out[i] = (float)(mean + std * normal_at(key, (uint64_t)i));
}

/* Same stream as rg_synth_normal_f32, then rounded to bfloat16 bits. */
void rg_synth_normal_bf16(uint16_t* out, int64_t rows, int64_t cols, uint64_t seed,
                          uint64_t tensor_id, double mean, double std) {
    const uint64_t key = stream_key(seed, tensor_id);
    const int64_t n = rows * cols;
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i)
        out[i] = f32_to_bf16_rne((float)(mean + std * normal_at(key, (uint64_t)i)));
}
