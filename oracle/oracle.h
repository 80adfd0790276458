/*
 * Oracle for FP8 scaled quantization and the scaled FP8 GEMM.
 *
 * TEST INFRASTRUCTURE ONLY.  This is a plain, slow, single-threaded CPU
 * statement of what the hot path computes, used to check the HIP library.
 * Only the test suite, the smoke check and the CPU-baseline leg of the
 * benchmark may load it.  It shares no code, header, table or constant with
 * the HIP library, and the HIP library never calls it.
 *
 * Method (paper, Sec. 2.2 "FP8 Quantization", Eq. 3):
 *     S_X = max|X| / F_max,   X_hat = Q_FP8(X / S_X),   X_tilde = S_X * X_hat
 * with the max taken per scaling unit: the whole tensor, each row, or each
 * block (Sec. 2.2, the paragraph on tensorwise / rowwise / blockwise scaling).
 *
 * Readings fixed here where the paper is silent (each is listed with its
 * reason in the design notes of the repository):
 *   - FP8 format is OCP E4M3 ("fn"), F_max = 448.
 *   - S is an fp32 number: S = RN32(amax / 448); if that is 0, S = 1.
 *   - The quotient X/S is a correctly rounded fp32 division (not a
 *     multiplication by a reciprocal).
 *   - Q_FP8 rounds that fp32 quotient to nearest, ties to even mantissa,
 *     and clamps magnitudes above 448 to 448.  The sign of zero is kept.
 *   - fp32 subnormals are kept (no flush to zero).
 * Variants offered next to the paper's method (flags of oracle_quantize):
 *   - ORACLE_E5M2: the format is OCP E5M2, F_max = 57344 (for gradients).
 *   - ORACLE_POW2_SCALE: S is the smallest power of two with F_max S >= amax,
 *     at least 2^-127, and 1 when amax is 0.
 *
 * Scale layouts (fp32, "rows" and "cols" are those of the OUTPUT matrix,
 * which is the input matrix or, with ORACLE_OUT_TRANSPOSED, its transpose):
 *   TENSOR   [1]
 *   ROW      [rows]                 one per row
 *   COL      [cols]                 one per column
 *   1x128    [cols/128][rows]       128 consecutive elements of one row;
 *                                   stored block-column major
 *   128x1    [rows/128][cols]       128 consecutive elements of one column
 *   128x128  [rows/128][cols/128]   128 x 128 tiles, row major
 * Granularities are stated on the INPUT matrix; with ORACLE_OUT_TRANSPOSED
 * the units are the same sets of elements, and the output is laid out as
 * the transpose (so 1x128 on X becomes 128x1 on X^T, ROW becomes COL).
 * Every dimension a block granularity splits must be a multiple of 128.
 */
#ifndef FP8_ORACLE_H
#define FP8_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
  ORACLE_TENSOR = 0,
  ORACLE_ROW = 1,
  ORACLE_COL = 2,
  ORACLE_BLOCK_1x128 = 3,
  ORACLE_BLOCK_128x1 = 4,
  ORACLE_BLOCK_128x128 = 5
};
enum { ORACLE_OUT_TRANSPOSED = 1, ORACLE_POW2_SCALE = 2, ORACLE_E5M2 = 4 };
/* Operand formats of oracle_gemm_rows_fmt. */
enum { ORACLE_FMT_E4M3 = 0, ORACLE_FMT_E5M2 = 1 };

/* Value of an OCP E4M3 byte; NaN for 0x7F and 0xFF. */
double oracle_e4m3_decode(uint8_t code);

/* Q_FP8 of an fp32 value: nearest E4M3 value, ties to even mantissa,
 * magnitudes >= 448 clamp to 448, sign kept (also for zero).
 * NaN input returns 0x7F (never produced for finite input). */
uint8_t oracle_e4m3_encode(float v);

/* Value of an OCP E5M2 byte: +-inf for 0x7C / 0xFC, NaN for 0x7D..0x7F and
 * 0xFD..0xFF. */
double oracle_e5m2_decode(uint8_t code);

/* Q_FP8 into E5M2: nearest E5M2 value, ties to even mantissa, magnitudes
 * >= 57344 clamp to 57344 (never infinity), sign kept.  NaN returns 0x7F. */
uint8_t oracle_e5m2_encode(float v);

/* Eq. 3 applied per scaling unit.  x_bf16 is row-major [rows][ldx] bf16
 * bit patterns; codes is [rows][ldc] (or [cols][ldc] when transposed).
 * Returns 0 on success, -1 on a bad argument. */
int oracle_quantize(const uint16_t *x_bf16, int64_t rows, int64_t cols,
                    int64_t ldx, int granularity, unsigned flags,
                    uint8_t *codes, int64_t ldc, float *scales);

/* One element of Eq. 3 with an explicit scale: Q_FP8(RN32(x / scale)). */
uint8_t oracle_cast_f32(float x, float scale);
/* Same over an array; used to check the device cast routine. */
void oracle_cast_f32_array(const float *x, int64_t n, float scale,
                           uint8_t *codes);
/* The E5M2 form: oracle_e5m2_encode(RN32(x[i] / scale)). */
void oracle_cast_f32_e5m2_array(const float *x, int64_t n, float scale,
                                uint8_t *codes);

/* Exact product of the dequantized operands of the FP8 linear layer:
 *   C[m][n] = sum_k (S_A(m,k) * A_hat[m][k]) * (S_B(n,k) * B_hat[n][k])
 * A codes are [M][lda] (K contiguous), B codes are [N][ldb] (K contiguous),
 * scales in the layouts above for the matrices A[M,K] and B[N,K].
 * Computed for the listed rows m only; out is [nrows][N] fp64.
 * Integer block products are exact (int64), the scaled sum is taken in
 * binary128 and rounded once to fp64.
 * Supported granularity pairs: (TENSOR,TENSOR), (ROW,ROW),
 * (1x128,128x128), (1x128,1x128).  Returns 0, or -1 on a bad argument. */
int oracle_gemm_rows(const uint8_t *A, const float *sA, int gA, int64_t lda,
                     const uint8_t *B, const float *sB, int gB, int64_t ldb,
                     int64_t M, int64_t N, int64_t K, const int64_t *rows,
                     int64_t nrows, double *out);
/* The same with the codes of A and of B each in E4M3 or E5M2
 * (ORACLE_FMT_*). */
int oracle_gemm_rows_fmt(const uint8_t *A, const float *sA, int gA,
                         int64_t lda, int fmtA, const uint8_t *B,
                         const float *sB, int gB, int64_t ldb, int fmtB,
                         int64_t M, int64_t N, int64_t K, const int64_t *rows,
                         int64_t nrows, double *out);

#ifdef __cplusplus
}
#endif
#endif
