/*
 * rg.h -- C-ABI of a bit-reproducible fused-upcast linear layer for AMD MI355X (gfx950).
 *
 * The operation (paper: Design, eq. 2; rg_linear_bias adds its bias term):
 *
 *     y[m][n] = sum over k of  x[m][k] * up(W[n][k])
 *
 *   x : float32  [M][K] row-major (activations; the paper's FP32 compute path)
 *   W : bfloat16 [N][K] row-major, passed as uint16_t bit patterns
 *       (the nn.Linear [out][in] layout; weights stay resident in BF16)
 *   y : float32  [M][N] row-major, fully overwritten (never read)
 *
 * up(b) widens a bfloat16 pattern to float32 exactly: the float whose bits are
 * (uint32_t)b << 16.  It happens in registers; no FP32 copy of W is ever
 * written to memory (Design, eq. 2 and the dataflow figure).
 *
 * THE REDUCTION ORDER ("RG-ORDER-1").  For every output element, with C = 256
 * and J = ceil(K / C):
 *
 *   p_j = +0.0f;  for k = j*C .. min(j*C + C, K) - 1 in ascending order:
 *                      p_j = fmaf(x[m][k], up(W[n][k]), p_j)
 *   y   = p_0;    for j = 1 .. J-1 in ascending order:  y = y + p_j
 *
 * - Every multiply-add is one IEEE-754 binary32 fused multiply-add and every
 *   combine one binary32 addition, round to nearest even, subnormals kept on
 *   input and output (rule R1: IEEE FMA only; no matrix cores are used).
 * - K is cut into fixed 256-wide segments (a pure function of K, rule R3);
 *   each segment is one sequential chain in ascending k; the segment partials
 *   are combined in fixed ascending segment order with no atomics (rule R3).
 * - The order depends on K alone: not on M, N, the row m or n, the kernel
 *   chosen, the grid, the block, the number of compute units, CU masks, the
 *   stream or timing (rules R2 and R4).  A row of y is therefore bitwise the
 *   same at every batch size M (batch invariance, rule R4, here for all M).
 *
 * Results are bitwise equal to the plain C CPU implementation of this order.
 *
 * Threading and streams.  Calls are asynchronous and stream ordered on the
 * given stream (a hipStream_t passed as void*; NULL = the null stream).  The
 * library never synchronizes and allocates no device memory in rg_linear.
 * Concurrent calls from several threads, on the same or different streams,
 * are safe.  rg_linear_set_launch changes one process-wide setting (a test
 * knob, updated under a lock) that every later call of every thread uses;
 * since launch settings never change the arithmetic, a call racing with it
 * still returns the same bits, or RG_ERR_RANGE if the setting it read does
 * not fit its shape.
 *
 * Errors.  Every entry point returns an rg_status code; none aborts or prints.
 */
#ifndef RG_H
#define RG_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define RG_CHUNK 256     /* segment length C of RG-ORDER-1 */
#define RG_ORDER_ID 1    /* identifies RG-ORDER-1 in rg_plan_t.order_id */

typedef enum {
    RG_OK = 0,
    RG_ERR_INVAL = 1,    /* null pointer, M/N/K < 1, or M*K, N*K, M*N overflow int64 */
    RG_ERR_ALIGN = 2,    /* x, W or y not 4-byte aligned (BF16 W: 2-byte) */
    RG_ERR_ARCH = 3,     /* current device is not gfx950 */
    RG_ERR_HIP = 4,      /* a HIP runtime call failed (launch or query) */
    RG_ERR_RANGE = 5,    /* an rg_launch_t field is out of its documented range */
    RG_ERR_ALIAS = 6     /* y overlaps x or W */
} rg_status;

/* Kernel ids reported by rg_plan (scheduling only; the order is the same). */
typedef enum {
    RG_KERNEL_GENERIC = 0,   /* one thread per output; any K, any alignment */
    RG_KERNEL_DECODE = 1,    /* M <= 4 (or K < 4096 up to M = 64): streaming skinny GEMM, x in registers */
    RG_KERNEL_TILED = 2,     /* larger M: register-tiled kernel, whole K per workgroup */
    RG_KERNEL_DECODE_XS = 3, /* M == 1 (when forced, or where the skinny kernel's x does not fit its
                                registers): streaming GEMV with x streamed through LDS beside W */
    RG_KERNEL_GEMV = 4,      /* M == 1, K % 256 == 0, K >= 4096 (the default for K == 4096 with
                                N <= 4096; elsewhere when forced, or where the skinny kernel's x
                                does not fit): 32 KB W bursts, whole rows per wave */
    RG_KERNEL_STREAM = 5,    /* M <= 4: 8-row blocks of W streamed through LDS, one chain per lane
                                (FP32 weights by default; BF16 weights when forced) */
    RG_KERNEL_KTILE = 6,     /* 16 < M <= 64 (any M when forced): 4 x 4 register tiles, K segments
                                shared out over thread groups */
    RG_KERNEL_SKINNY = 7,    /* M <= 16, and narrow layers to M = 64: waves of 16 W rows x 4
                                segments, x of a segment shared by 16 lanes through DPP row
                                broadcasts, slices of 1, 2, 4 or 8 rows of x */
    RG_KERNEL_WTILE = 8      /* 32 < M <= 64 on wide layers: 64 x 64 output tiles, each wave the
                                whole tile for one segment at a time (8 x 8 chains per lane),
                                its own LDS slabs, the partials added wave by wave in segment
                                order */
} rg_kernel_id;

/* Scheduling overrides for the determinism tests.  0 in a field = planner
 * default.  None of these can change a result bit; they only move work
 * between workgroups, waves and compute units.
 *   kernel        : -1/0 = planner's choice, else 1 + rg_kernel_id to force one
 *                   (a kernel that cannot handle the shape is not forced; the
 *                    call returns RG_ERR_RANGE)
 *   waves_per_wg  : 1..8  waves (64 threads each) per workgroup (gemv: 1..4, and 1, 2
 *                   or 4 when K > 4096; ktile: 4, or 8 with tile_n 16; skinny: any count
 *                   whose ceil(J / 4 / waves) segment groups per wave fit its registers;
 *                   wtile: 4 or 8)
 *   grid_wgs      : 1..65536 workgroups (work is spread over them evenly)
 *   depth         : 2..3  decode pipeline depth in 128-byte-per-row slabs (unused by gemv);
 *                   tiled kernel with 128 x 128 tiles: the build for 2 or 3 waves per SIMD;
 *                   ktile: 2 = 4 x 4, 3 = 4 x 8 outputs per thread (tile_n 32 or 64 only);
 *                   skinny: 8 KB steps in flight per wave
 *   grid_order    : 0 = forward, 1 = reversed workgroup-to-rows mapping
 *   tile_n        : 0 = planner default, else 16, 32 or 64: ktile's W rows per tile
 *   slice_m       : 0 = planner default, else 1, 2, 4 or 8: skinny's rows of x per slice
 *                   (M > slice_m runs ceil(M / slice_m) slices, each streaming all of W;
 *                    capped at what the kernel's x registers hold)
 *   reserved      : must be 0
 */
typedef struct {
    int32_t kernel;
    int32_t waves_per_wg;
    int32_t grid_wgs;
    int32_t depth;
    int32_t grid_order;
    int32_t tile_n;
    int32_t slice_m;
    int32_t reserved;
} rg_launch_t;

/* What rg_linear will do for a shape (on a 256-CU MI355X with default launch). */
typedef struct {
    int32_t order_id;      /* RG_ORDER_ID */
    int32_t chunk;         /* C = 256 */
    int64_t nchunks;       /* J = ceil(K / 256) */
    int32_t kernel;        /* rg_kernel_id */
    int32_t waves_per_wg;
    int32_t grid_wgs;
    int32_t depth;         /* decode: pipeline depth; tiled 128 x 128: waves per SIMD (2 or 3);
                              ktile: 2 = 4 x 4, 3 = 4 x 8 outputs per thread */
    int32_t rows_per_round;/* decode: W rows per workgroup round; skinny: 16 */
    int32_t tile_m, tile_n;/* tiled, ktile, wtile: output tile; skinny: rows of x per slice, 16 W rows */
} rg_plan_t;

/*
 * y = x * up(W)^T in RG-ORDER-1 (Design, eq. 2; rules R1-R4).
 *   x      device pointer, float32 [M][K], 4-byte aligned
 *   w_bf16 device pointer, bfloat16 bits [N][K], 2-byte aligned
 *   y      device pointer, float32 [M][N], 4-byte aligned, must not overlap x or W
 *   M,N,K  >= 1
 *   stream hipStream_t or NULL
 * The caller owns all buffers.  Fast paths need 16-byte aligned x and W and
 * K % 8 == 0; other shapes take a slower kernel with the same order and bits.
 * Returns RG_OK once the kernel is enqueued, or an rg_status error (nothing
 * is enqueued on error).  Launch-time HIP errors are returned as RG_ERR_HIP.
 */
int rg_linear(const float* x, const uint16_t* w_bf16, float* y, int64_t M, int64_t N, int64_t K,
              void* stream);

/*
 * y = x * up(W)^T + b: the product of rg_linear in RG-ORDER-1, then one
 * binary32 round-to-nearest-even addition of b[n] per output (Design, eq. 2
 * with its bias term; the bias is added after the fold, never into a chain).
 *   bias   device pointer, float32 [N], 4-byte aligned, not NULL, must not
 *          overlap y (it may alias x or W, which are only read)
 * Everything else as rg_linear (same kernels, same scheduling, same errors;
 * RG_ERR_INVAL for a NULL bias).
 */
int rg_linear_bias(const float* x, const uint16_t* w_bf16, const float* bias, float* y, int64_t M, int64_t N,
                   int64_t K, void* stream);

/*
 * y = x * W^T with FP32 weights, in RG-ORDER-1 with the weight used as it is in
 * place of up(W) (paper: Supplement C probes BF16 and FP32 weights alike; the
 * same segments, chains and ascending fold, so FP32 weights that hold widened
 * BF16 values give rg_linear's bits exactly).
 *   x      device pointer, float32 [M][K], 4-byte aligned
 *   w_f32  device pointer, float32 [N][K], 4-byte aligned
 *   y      device pointer, float32 [M][N], 4-byte aligned, must not overlap x or W
 * Kernels: RG_KERNEL_STREAM for M <= 4, then ktile (M <= 64) and tiled
 * (wtile when forced), all needing 16-byte aligned x and W and K % 4 == 0;
 * other shapes take the generic kernel.  Errors, streams and ownership as rg_linear; the same
 * rg_linear_set_launch overrides apply (decode, decode_xs and gemv cannot be
 * forced here: RG_ERR_RANGE).
 */
int rg_linear_f32w(const float* x, const float* w_f32, float* y, int64_t M, int64_t N, int64_t K, void* stream);

/* Set (cfg != NULL) or reset (cfg == NULL) the scheduling overrides used by
 * later rg_linear, rg_linear_bias and rg_linear_f32w calls.  RG_ERR_RANGE if a
 * field is out of range.  They exist to show rules R2-R3 hold (Design, R2-R3;
 * Supplement C, the schedule ablations): moving work between workgroups,
 * waves and compute units changes no bit. */
int rg_linear_set_launch(const rg_launch_t* cfg);

/* Fill *out with the plan for (M, N, K) under the current overrides.  A pure
 * function of its arguments and the overrides; queries no device.  CPU safe.
 * Rule R2 (Design): the configuration, and with it every bit of the result,
 * is a function of the shape alone; the segment length C and count J that fix
 * the order depend on K alone (Design, R3). */
int rg_plan(int64_t M, int64_t N, int64_t K, rg_plan_t* out);

/* The same for rg_linear_f32w (FP32 weights). */
int rg_plan_f32w(int64_t M, int64_t N, int64_t K, rg_plan_t* out);

/* Comparison point only (the scheme the paper improves on, Design, eq. 1):
 * w_f32[n][k] = up(W[n][k]) written to a caller-provided FP32 buffer of N*K
 * floats (the transient copy the fused kernel never makes).  Any FP32 GEMM
 * can then consume it.  Stream ordered, asynchronous.  RG_ERR_INVAL for a
 * null pointer or count < 1 (or count * 4 bytes overflowing), RG_ERR_ALIGN for
 * a misaligned pointer, RG_ERR_ALIAS if the two buffers overlap. */
int rg_cast_bf16_f32(const uint16_t* w_bf16, float* w_f32, int64_t count, void* stream);

/* Greedy decision over logits (Evaluation, end-to-end determinism: argmax
 * returns the lower token id on a tie): out_idx[m] = the lowest n with
 * y[m][n] maximal, NaN never wins (all-NaN rows give -1).  y: device float32
 * [M][N]; out_idx: device int64 [M], 8-byte aligned, must not overlap y
 * (RG_ERR_ALIAS).  M <= 2^31 - 1.  Deterministic; no atomics. */
int rg_argmax_rows(const float* y, int64_t* out_idx, int64_t M, int64_t N, void* stream);

/* Test helpers: a stream restricted to the compute units set in `mask`
 * (bit i of word i/32 = CU i), and its destruction. */
int rg_stream_create_cu_mask(const uint32_t* mask, uint32_t nwords, void** out_stream);
int rg_stream_destroy(void* stream);

/* Number of compute units of the current device (RG_ERR_HIP if none). */
int rg_device_cu_count(int32_t* out);

/* The hipError_t code of the last HIP call this thread made inside the
 * library (0 = hipSuccess); explains an RG_ERR_HIP return. */
int rg_last_hip_error(void);

/* Static description of an rg_status code (never NULL). */
const char* rg_strerror(int code);

#ifdef __cplusplus
}
#endif

#endif /* RG_H */
