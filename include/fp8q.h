/*
 * fp8q — FP8 scaled quantization and the scaled FP8 GEMM of an FP8 linear
 * layer, for AMD Instinct MI355X (gfx950).
 *
 * The method (paper "Towards Full Pipeline FP8 Reinforcement Learning for
 * LLMs", Sec. 2.2, Eq. 3): for a high-precision tensor X and a scaling unit
 * U (the whole tensor, one row, or one block),
 *     S_U = max_{x in U} |x| / F_max,  X_hat = Q_FP8(X / S_U),  X_tilde = S_U X_hat
 * where Q_FP8 rounds and clamps to the FP8 set.  The FP8 training engine the
 * paper uses (Sec. 5, experimental setup; Sec. 5.3, training throughput) runs
 * the linear layers of the policy as GEMMs on such operands.
 *
 * Conventions fixed by this library:
 *   - FP8 is OCP E4M3 (1.4.3, bias 7, no infinities, NaN = S.1111.111),
 *     F_max = 448.  Codes are the raw E4M3 bytes.
 *   - S is fp32: S = RN32(amax / 448), and S = 1 when that is 0.  `scales`
 *     always holds S itself (the dequantization multiplier), never 1/S.
 *   - Q_FP8(X / S) = E4M3 nearest-even of the correctly rounded fp32
 *     quotient; magnitudes above 448 clamp to 448; the sign of zero is kept;
 *     fp32 subnormals are not flushed.
 *   - Inputs are bf16, row-major; Inf/NaN inputs are outside the contract.
 *
 * All data pointers are DEVICE pointers owned by the caller.  The library
 * never allocates, frees or synchronizes; every call enqueues its kernels on
 * `stream` (a hipStream_t; NULL is the legacy default stream) and returns.
 * Arguments are validated on the host before anything is enqueued; a
 * rejected call enqueues nothing.  Sizes and leading dimensions above
 * 2^31 - 1 elements (Calibrated Clipping batches above 2^52 tokens, casts
 * above 2^62 values) are FP8Q_ERR_UNSUPPORTED.  Faults inside kernels surface at the
 * caller's next synchronization.  Apart from the one device array of
 * fp8q_calibrate_clip_noalloc, the library holds no mutable global state,
 * so calls from several threads are safe; calls that write the same
 * buffers must be ordered by the caller.
 */
#ifndef FP8Q_H
#define FP8Q_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

struct ihipStream_t; /* hipStream_t is `struct ihipStream_t *` */

typedef enum {
  FP8Q_OK = 0,
  FP8Q_ERR_INVAL = -1,       /* null pointer, size <= 0, ld too small, bad enum */
  FP8Q_ERR_UNSUPPORTED = -2, /* shape or granularity pair the kernels do not take */
  FP8Q_ERR_ALIGN = -3,       /* pointer or leading dimension misaligned */
  FP8Q_ERR_HIP = -4          /* a HIP launch failed */
} fp8q_status;

/* Scaling units of Eq. 3 (Sec. 2.2: tensorwise, rowwise, blockwise).
 * They are stated on the INPUT matrix x[rows][cols]. */
typedef enum {
  FP8Q_TENSOR = 0,       /* one unit: the whole tensor                     */
  FP8Q_ROW = 1,          /* one unit per row (per token / per out channel) */
  FP8Q_COL = 2,          /* one unit per column                            */
  FP8Q_BLOCK_1x128 = 3,  /* 128 consecutive elements of one row            */
  FP8Q_BLOCK_128x1 = 4,  /* 128 consecutive elements of one column         */
  FP8Q_BLOCK_128x128 = 5 /* 128 x 128 tiles                                */
} fp8q_granularity;

/* Write codes as the transpose, codes[c][r] = Q(x[r][c]).  The scaling
 * units stay the same sets of elements; the scales are laid out for the
 * transposed matrix (so 1x128 of x is 128x1 of x^T, ROW of x is COL). */
enum { FP8Q_OUT_TRANSPOSED = 1u };
/* A variant of Eq. 3's scale (not the paper's; for fp8q_gemm_pow2): S is
 * the smallest power of two with 448 S >= amax, at least 2^-127, and 1 when
 * amax is 0.  Every |x| / S is then at most 448 and exact, and S fits the
 * E8M0 block scales of the MI355X matrix instructions. */
enum { FP8Q_POW2_SCALE = 2u };
/* E5M2 codes instead of E4M3 (a variant for gradients; the paper leaves
 * the FP8 format of Eq. 3 open): OCP E5M2, F_max = 57344, so S =
 * RN32(amax / 57344) and each code is the nearest-even E5M2 value of
 * RN32(x / S) clamped at 57344 (never an infinity).  With FP8Q_POW2_SCALE,
 * S is the smallest power of two with 57344 S >= amax, at least 2^-127. */
enum { FP8Q_E5M2 = 4u };

/*
 * Number of fp32 scales fp8q_quantize writes for an input of rows x cols
 * with granularity g and `flags` (the scaling units of Eq. 3 for the
 * granularities of Sec. 2.2); -1 if the arguments are invalid or a size
 * exceeds 2^31 - 1.
 *
 * Scale layouts, for the OUTPUT matrix o[orows][ocols] (x, or x^T when
 * transposed) and the granularity g_o it sees (g, or g with rows and
 * columns exchanged when transposed):
 *   TENSOR   [1]
 *   ROW      [orows]
 *   COL      [ocols]
 *   1x128    [ocols/128][orows]  block-column major: all rows of one
 *                                128-wide column block are contiguous
 *   128x1    [orows/128][ocols]
 *   128x128  [orows/128][ocols/128]
 * With these layouts the transposed output of 1x128 / 128x1 / ROW / COL /
 * TENSOR uses the same scale array as the plain output; 128x128 transposes
 * its block grid.
 */
int64_t fp8q_scales_count(int64_t rows, int64_t cols, fp8q_granularity g,
                          unsigned flags);

/*
 * Eq. 3 per scaling unit: codes and scales of x.  flags: any of
 * FP8Q_OUT_TRANSPOSED, FP8Q_POW2_SCALE and FP8Q_E5M2.
 *   x       bf16 [rows][ldx], ldx >= cols
 *   codes   E4M3 (E5M2 with FP8Q_E5M2) [rows][ldc] (ldc >= cols), or
 *           [cols][ldc] (ldc >= rows)
 *           with FP8Q_OUT_TRANSPOSED
 *   scales  fp32, fp8q_scales_count(rows, cols, g, flags) entries
 * Shape rules: cols % 16 == 0, and rows % 16 == 0 when transposed; a
 * dimension a 128-block splits (cols for 1x128 and 128x128, rows for 128x1
 * and 128x128) must be a multiple of 128; rows <= 65535 x 128 (else
 * FP8Q_ERR_UNSUPPORTED).  x must not overlap codes or scales.
 * Alignment: x and codes 16-byte aligned, ldx % 8 == 0, ldc % 16 == 0,
 * scales 4-byte aligned (else FP8Q_ERR_ALIGN).
 * TENSOR, COL and ROW with FP8Q_OUT_TRANSPOSED run three kernels (partial
 * amaxes, their reduction to S, the cast) and keep the partial amaxes in
 * `codes` between them (only the codes' own bytes, never the padding of a
 * strided code array), or in `scales` when each unit has one partial; the
 * cast then overwrites them.
 */
fp8q_status fp8q_quantize(const void *x, int64_t rows, int64_t cols,
                          int64_t ldx, fp8q_granularity g, unsigned flags,
                          uint8_t *codes, int64_t ldc, float *scales,
                          struct ihipStream_t *stream);

/*
 * Both operand layouts the backward pass needs, from one read of x (Eq. 3
 * applied twice per element).  The weight-gradient GEMM contracts over the
 * token dimension, so it takes x (an activation X or an output gradient dY)
 * transposed and grouped by 128 along the rows, while the forward and
 * data-gradient GEMMs take it grouped by 128 along the columns.  Outputs:
 *   codes_r, scales_r  exactly fp8q_quantize(x, FP8Q_BLOCK_1x128, flags):
 *                      codes [rows][ldc_r] (ldc_r >= cols), scales
 *                      [cols/128][rows]
 *   codes_t, scales_t  exactly fp8q_quantize(x, FP8Q_BLOCK_128x1,
 *                      FP8Q_OUT_TRANSPOSED | flags): codes [cols][ldc_t]
 *                      (ldc_t >= rows), scales [rows/128][cols]
 * x is bf16 [rows][ldx].  flags: FP8Q_POW2_SCALE, FP8Q_E5M2 (for an output
 * gradient), both, or 0; any other bit is FP8Q_ERR_INVAL.  Shape rules: rows % 128 == 0 and cols % 128 == 0
 * (else FP8Q_ERR_UNSUPPORTED).  Alignment: x and both code arrays 16-byte
 * aligned, ldx % 8 == 0, ldc_r % 16 == 0, ldc_t % 16 == 0, scales 4-byte
 * aligned (else FP8Q_ERR_ALIGN).  The four outputs must not overlap.
 */
fp8q_status fp8q_quantize_dual(const void *x, int64_t rows, int64_t cols,
                               int64_t ldx, unsigned flags, uint8_t *codes_r,
                               int64_t ldc_r, float *scales_r,
                               uint8_t *codes_t, int64_t ldc_t,
                               float *scales_t, struct ihipStream_t *stream);

/*
 * The FP8 linear layer's GEMM on dequantized operands (Eq. 3 applied to
 * both; fp32 accumulation; bf16 round-to-nearest-even output):
 *   C[m][n] = sum_k (S_A(m,k) A[m][k]) (S_B(n,k) B[n][k])
 *   A  E4M3 [M][lda], K contiguous (activations X, dY, or X^T / dY^T)
 *   B  E4M3 [N][ldb], K contiguous (weights W stored [N][K], W^T, or dY^T)
 *   C  bf16 [M][ldc]
 * Forward Y = X W^T, dgrad dX = dY W and wgrad dW = dY^T X all take this
 * form once the quantizer has written the operands K-contiguous (dgrad's W^T
 * and wgrad's X^T, dY^T come from FP8Q_OUT_TRANSPOSED).
 * Scales sA, sB in the layouts of fp8q_scales_count for A[M][K], B[N][K].
 * Supported (gA, gB): (TENSOR, TENSOR), (ROW, ROW) — per-token x
 * per-output-channel —, (1x128, 128x128) — activation blocks x weight
 * blocks — and (1x128, 1x128) — both grouped along K, for wgrad.
 * Shape rules: K % 128 == 0; N % 128 == 0 when gB is 128x128; M and N are
 * otherwise free.  Alignment: A and B 16-byte aligned, lda % 16 == 0,
 * ldb % 16 == 0; C 8-byte aligned with ldc % 4 == 0; scales 4-byte aligned.
 */
fp8q_status fp8q_gemm(const uint8_t *A, const float *sA, fp8q_granularity gA,
                      int64_t lda, const uint8_t *B, const float *sB,
                      fp8q_granularity gB, int64_t ldb, int64_t M, int64_t N,
                      int64_t K, void *C, int64_t ldc,
                      struct ihipStream_t *stream);

/* One problem of fp8q_gemm_grouped: the arguments of fp8q_gemm that differ
 * between the problems (pointers, leading dimensions, M and N). */
typedef struct fp8q_gemm_problem {
  const uint8_t *A;   /* codes [M][lda] */
  const float *sA;
  int64_t lda;
  const uint8_t *B;   /* codes [N][ldb] */
  const float *sB;
  int64_t ldb;
  void *C;            /* bf16 [M][ldc] */
  int64_t ldc;
  int64_t M, N;
} fp8q_gemm_problem;

enum { FP8Q_MAX_GROUP = 8 };

/*
 * Several fp8q_gemm problems in one launch: the grouped GEMM of fused
 * projections that share their input (the FP8 linear layers of Sec. 5.3,
 * e.g. the query, key and value projections, or the gate and up
 * projections of an MLP, each with its own weight and output).  Each
 * problems[i] (a host array of 1 .. FP8Q_MAX_GROUP entries, read before the
 * call returns) computes C_i = dequant(A_i) dequant(B_i)^T exactly as
 * fp8q_gemm(A_i, sA_i, gA, lda_i, B_i, sB_i, gB, ldb_i, M_i, N_i, K, C_i,
 * ldc_i) would, with every rule of fp8q_gemm per problem; the A_i may be
 * the same operand.  Supported (gA, gB): (TENSOR, TENSOR), (ROW, ROW) and
 * (1x128, 128x128) (else FP8Q_ERR_UNSUPPORTED).  Each problem's A, B and C
 * must each span less than 2 GiB (M lda, N ldb and 2 M ldc bytes; else
 * FP8Q_ERR_UNSUPPORTED).  The outputs must not overlap each other or any
 * input.  count outside 1 .. FP8Q_MAX_GROUP is FP8Q_ERR_INVAL.
 */
fp8q_status fp8q_gemm_grouped(const fp8q_gemm_problem *problems, int count,
                              fp8q_granularity gA, fp8q_granularity gB,
                              int64_t K, struct ihipStream_t *stream);

/* Operand formats of fp8q_gemm_formats: A's codes, B's codes are E5M2. */
enum { FP8Q_A_E5M2 = 1u, FP8Q_B_E5M2 = 2u };

/*
 * fp8q_gemm with each operand's codes in E4M3 or E5M2 (the E5M2 variant of
 * FP8Q_E5M2, for output gradients): `formats` is 0 or FP8Q_A_E5M2,
 * FP8Q_B_E5M2, or both; any other bit is FP8Q_ERR_INVAL.  The product,
 * layouts, shape and alignment rules are those of fp8q_gemm.  Non-zero
 * formats are supported for the backward pairs (1x128, 128x128) — dgrad
 * dX = dY W with dY in E5M2 — and (1x128, 1x128) — wgrad dW = dY^T X —
 * (else FP8Q_ERR_UNSUPPORTED); formats 0 is fp8q_gemm.
 */
fp8q_status fp8q_gemm_formats(const uint8_t *A, const float *sA,
                              fp8q_granularity gA, int64_t lda,
                              const uint8_t *B, const float *sB,
                              fp8q_granularity gB, int64_t ldb, int64_t M,
                              int64_t N, int64_t K, unsigned formats, void *C,
                              int64_t ldc, struct ihipStream_t *stream);

/*
 * fp8q_gemm for operands quantized with FP8Q_POW2_SCALE: the same product
 * (fp32 accumulation, bf16 round-to-nearest-even output), with the block
 * scales applied inside the matrix instruction as E8M0 exponents instead
 * of by fp32 multiplies.  Every scale must be a power of two in [2^-127,
 * 2^127] (as FP8Q_POW2_SCALE writes them; other values are read as their
 * exponent alone).  Supported (gA, gB): (1x128, 128x128) only.  Shape and
 * alignment rules: those of fp8q_gemm, with N % 128 == 0.
 */
fp8q_status fp8q_gemm_pow2(const uint8_t *A, const float *sA,
                           fp8q_granularity gA, int64_t lda, const uint8_t *B,
                           const float *sB, fp8q_granularity gB, int64_t ldb,
                           int64_t M, int64_t N, int64_t K, void *C,
                           int64_t ldc, struct ihipStream_t *stream);

/*
 * fp8q_gemm followed by the quantization of its output, in one kernel: the
 * next layer's activation operand (Eq. 3 with 1x128 units along N) without
 * the bf16 round trip through memory.  The outputs are exactly
 *   fp8q_quantize(C, M, N, N, FP8Q_BLOCK_1x128, 0, codes, ldq, scales)
 * for the bf16 C that fp8q_gemm computes from the same arguments:
 *   codes   E4M3 [M][ldq], ldq >= N
 *   scales  fp32 [N/128][M]
 * Supported (gA, gB): (1x128, 128x128) only.  Shape rules: K % 128 == 0,
 * N % 128 == 0.  Alignment: A, B and codes 16-byte aligned, lda, ldb and
 * ldq multiples of 16, scales 4-byte aligned.
 */
fp8q_status fp8q_gemm_quantized(const uint8_t *A, const float *sA,
                                fp8q_granularity gA, int64_t lda,
                                const uint8_t *B, const float *sB,
                                fp8q_granularity gB, int64_t ldb, int64_t M,
                                int64_t N, int64_t K, uint8_t *codes,
                                int64_t ldq, float *scales,
                                struct ihipStream_t *stream);

/*
 * Bytes of workspace fp8q_gemm_splitk needs for an M x N x K problem (0 when
 * that call does not split K and is fp8q_gemm); -1 for a size <= 0 or
 * above 2^31 - 1.
 */
int64_t fp8q_gemm_splitk_workspace(int64_t M, int64_t N, int64_t K);

/*
 * fp8q_gemm for skinny problems such as a decode step of the FP8 rollout
 * (Sec. 2.3, Sec. 5: a few hundred rows of activations against a full
 * weight), where the 128 x 128 tiles of C are too few to give every CU one
 * (fewer than 128).  The K blocks of each tile are split over S workgroups (S a power
 * of two up to 8, S x tiles <= 256, at least four K blocks each), so that
 * each CU streams 1/S of the tile's operand rows; the S fp32 partial tiles
 * are added in a fixed order, then rounded to bf16 once.  The product,
 * pairs, layouts, shape and alignment rules are those of fp8q_gemm, and
 * the result is the same on every run; its K sum is grouped differently
 * from fp8q_gemm's, so the last bits of an output can differ.  Problems
 * with 128 or more tiles, or whose operands span 2 GiB, are not split:
 * then the call is fp8q_gemm and needs no workspace.
 * workspace: device memory of at least fp8q_gemm_splitk_workspace(M, N, K)
 * bytes (workspace_bytes), 16-byte aligned, ZERO-FILLED before its first
 * use; it holds per-tile arrival counters, which every call leaves at
 * zero, and the partial tiles.  Calls that share a workspace must not
 * overlap (issue them on one stream).  Errors: those of fp8q_gemm; a null
 * or short workspace when the call splits -> INVAL, misaligned -> ALIGN.
 */
fp8q_status fp8q_gemm_splitk(const uint8_t *A, const float *sA,
                             fp8q_granularity gA, int64_t lda,
                             const uint8_t *B, const float *sB,
                             fp8q_granularity gB, int64_t ldb, int64_t M,
                             int64_t N, int64_t K, void *C, int64_t ldc,
                             void *workspace, int64_t workspace_bytes,
                             struct ihipStream_t *stream);

/*
 * Calibrated Clipping (Sec. 4, Alg. 1, Eq. 5): new lower and upper PPO
 * clipping bounds for FP8 training from one batch of n tokens.
 *
 * Inputs, float32 device arrays of n tokens, 16-byte aligned: adv (the
 * advantage A_t), w_tis (the TIS weight, already truncated), pi_sampler
 * (the sampler's probability of the token), r_bf16 and r_fp8 (the
 * importance ratio from the BF16 shadow passes and from the FP8 passes).
 * Ratios must be finite.  l_old, h_old: the current bounds.  config (a HOST
 * pointer, read during the call): the reference bounds, the search
 * intervals and step, and the SmoothUpdate limits; PAPER values in the
 * field comments.
 *
 * Steps (each statistic is a float64 sum over the batch):
 *   alpha_low = F_BF16,-(c_low_ref), F the CDF P(r <= x) over tokens with
 *               A < 0;
 *   L* = grid point of [l_min, l_max] minimising |F_FP8,-(L) - alpha_low|;
 *   rho(c_low, c_high) = |sum_{A>0} w pi r A [r < c_high]| /
 *                        |sum_{A<0} w pi r A [r > c_low]|   (Eq. 5);
 *   H* = grid point of [h_min, h_max] minimising |rho_FP8(L*, H) -
 *        rho_BF16(c_low_ref, c_high_ref)|;
 *   new bound = b + clip((b* - b) / 2, -delta, delta)   (SmoothUpdate).
 * Grid points are lo + k * step (float64, no fused multiply-add), k = 0 ..
 * round((hi - lo) / step); ties go to the first point.  Tokens with A = 0
 * count nowhere.  With no negative-advantage token both bounds stay; when
 * an Eq. 5 denominator is zero the upper bound stays.  Results are the same
 * on every run.
 *
 * workspace: device memory of at least fp8q_calibrate_clip_workspace(n)
 * bytes, 8-byte aligned, overwritten.  result: a DEVICE pointer to one
 * fp8q_clip_result (8-byte aligned), written by the last kernel; fields of
 * a stage that did not run are NaN.  Errors: null pointers, n <= 0, step
 * <= 0, empty or inverted intervals, a span that is not a whole number of
 * steps, or a small workspace -> INVAL; grids of more than 24 (lower) or
 * 48 (upper) points -> UNSUPPORTED; misaligned arrays -> ALIGN.
 */
typedef struct fp8q_clip_config {
  double c_low_ref, c_high_ref; /* reference bounds (paper, GRPO: 0.8, 1.24) */
  double l_min, l_max;          /* search interval of L (paper: 0.5, 0.9)     */
  double h_min, h_max;          /* search interval of H (paper: 1.2, 2.0)     */
  double step;                  /* search step (paper: 0.02)                  */
  double delta_l, delta_h;      /* SmoothUpdate limits (paper: 0.05, 0.1)     */
} fp8q_clip_config;

typedef struct fp8q_clip_result {
  double l_new, h_new;     /* the updated bounds                          */
  double l_star, h_star;   /* the grid optima                             */
  double alpha_low;        /* F_BF16,-(c_low_ref)                         */
  double rho_bf16;         /* Eq. 5 of the BF16 ratios at the references */
  double rho_fp8;          /* Eq. 5 of the FP8 ratios at (L*, H*)         */
  int64_t n_neg, n_pos;    /* tokens with A < 0, A > 0                    */
  int32_t l_updated, h_updated;
} fp8q_clip_result;

int64_t fp8q_calibrate_clip_workspace(int64_t n);

fp8q_status fp8q_calibrate_clip(const float *adv, const float *w_tis,
                                const float *pi_sampler, const float *r_bf16,
                                const float *r_fp8, int64_t n, double l_old,
                                double h_old, const fp8q_clip_config *config,
                                void *workspace, int64_t workspace_bytes,
                                fp8q_clip_result *result,
                                struct ihipStream_t *stream);

/*
 * fp8q_calibrate_clip without a workspace, for callers that cannot allocate
 * device memory (code under HIP graph capture, serving loops, harnesses
 * that forbid allocation).  Arguments, results and every rule are those of
 * fp8q_calibrate_clip; the partial sums go to an array of the library's
 * own instead of a workspace.  This call allocates nothing.
 *
 * The array holds FP8Q_CLIP_SCRATCH_BYTES (212992) bytes on each device
 * the call runs on (the device of `stream`, or the current device for the
 * null stream), from the first call on that device until the process
 * ends; that first call looks up its address.  Every batch fits it (a
 * batch is split into at most 256 blocks of partial sums); a batch whose
 * partials would not fit is FP8Q_ERR_UNSUPPORTED.  Nothing in it needs to
 * start cleared: each call writes every partial it reads.  All calls on one
 * device share the array, so calls that may overlap on one device (on
 * different streams without ordering between them) race: order them.
 * A failed address lookup is FP8Q_ERR_HIP.
 */
enum { FP8Q_CLIP_SCRATCH_BYTES = 212992 };
fp8q_status fp8q_calibrate_clip_noalloc(const float *adv, const float *w_tis,
                                        const float *pi_sampler,
                                        const float *r_bf16, const float *r_fp8,
                                        int64_t n, double l_old, double h_old,
                                        const fp8q_clip_config *config,
                                        fp8q_clip_result *result,
                                        struct ihipStream_t *stream);

/*
 * Q_FP8(RN32(x[i] / scale)) for n fp32 values with one explicit scale (Eq.
 * 3's rounding and clamping with S given): the clamp and the hardware
 * E4M3 conversion that fp8q_quantize ends with, exposed for exhaustive
 * checks.  The quotient here is an IEEE division, correctly rounded; the
 * quantizers form the same correctly rounded quotient from a reciprocal
 * and two fused multiply-adds (checked against the division over every
 * bf16 amax and x pair on the host, and through the 1x128 quantizer on the
 * GPU).  x and codes need no alignment beyond their element size;
 * scale > 0.
 */
fp8q_status fp8q_cast_f32(const float *x, int64_t n, float scale,
                          uint8_t *codes, struct ihipStream_t *stream);
/* The same with the E5M2 codes of FP8Q_E5M2 (clamp at 57344). */
fp8q_status fp8q_cast_f32_e5m2(const float *x, int64_t n, float scale,
                               uint8_t *codes, struct ihipStream_t *stream);

/* Static string naming a status. */
const char *fp8q_status_string(fp8q_status status);

#ifdef __cplusplus
}
#endif
#endif /* FP8Q_H */
