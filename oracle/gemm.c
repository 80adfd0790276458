/*
 * Oracle GEMM (test infrastructure only): the exact product of the
 * dequantized FP8 operands X_tilde = S_X * X_hat of Eq. 3 (paper Sec. 2.2),
 * i.e. the linear layer evaluated on the FP8-quantized forward/backward
 * operands (Sec. 3, the FP8-quantized forward passes; Sec. 5.3, the FP8
 * training engine).
 *
 *   C[m][n] = sum_k (S_A(m,k) * A_hat[m][k]) * (S_B(n,k) * B_hat[n][k])
 *
 * Every E4M3 value times 2^9 is an integer v with |v| <= 229376, and every
 * finite E5M2 value times 2^16 an integer with |v| <= 57344 * 2^16 < 2^32,
 * so over a run of k on which both scales are constant the sum I of
 * v_A * v_B is an exact 128-bit integer.  Each run then contributes
 * S_A * S_B * I * 2^-(shift_A + shift_B); S_A * S_B is exact in fp64 (two
 * 24-bit significands).  For two E4M3 operands I < 2^51, so its product with
 * S_A * S_B is exact in binary128, where the runs are summed, and the single
 * final rounding is to fp64.  With an E5M2 operand I can need up to 80 bits
 * and that product may round in binary128 (relative error 2^-113, far below
 * the final fp64 rounding).
 *
 * E5M2 operands are the variant offered next to the paper's E4M3 for
 * gradients; the paper leaves the FP8 format open.
 */
#include <math.h>
#include <stdlib.h>

#include "oracle.h"

/* acc * 2^e for a binary128 value, by repeated exact halving (no libquadmath). */
static __float128 ldexpq_(__float128 acc, int e) {
  for (; e < 0; ++e) acc *= 0.5;
  return acc;
}

/* Scale of element (r, c) of a [rows, cols] operand under granularity g. */
static float scale_at(const float *s, int g, int64_t rows, int64_t cols,
                      int64_t r, int64_t c) {
  switch (g) {
    case ORACLE_TENSOR: return s[0];
    case ORACLE_ROW: return s[r];
    case ORACLE_BLOCK_1x128: return s[(c / 128) * rows + r];
    case ORACLE_BLOCK_128x128: return s[(r / 128) * (cols / 128) + c / 128];
    default: return NAN;
  }
}

static int pair_supported(int gA, int gB) {
  return (gA == ORACLE_TENSOR && gB == ORACLE_TENSOR) ||
         (gA == ORACLE_ROW && gB == ORACLE_ROW) ||
         (gA == ORACLE_BLOCK_1x128 && gB == ORACLE_BLOCK_128x128) ||
         (gA == ORACLE_BLOCK_1x128 && gB == ORACLE_BLOCK_1x128);
}

/* Integer images v[c] = decode(c) * 2^shift of every code of a format
 * (0 for the non-finite codes); returns the shift. */
static int images(int fmt, __int128 *v) {
  int shift = fmt == ORACLE_FMT_E5M2 ? 16 : 9;
  for (int c = 0; c < 256; ++c) {
    double d = fmt == ORACLE_FMT_E5M2 ? oracle_e5m2_decode((uint8_t)c)
                                      : oracle_e4m3_decode((uint8_t)c);
    v[c] = isfinite(d) ? (__int128)ldexp(d, shift) : 0;
  }
  return shift;
}

int oracle_gemm_rows(const uint8_t *A, const float *sA, int gA, int64_t lda,
                     const uint8_t *B, const float *sB, int gB, int64_t ldb,
                     int64_t M, int64_t N, int64_t K, const int64_t *rows,
                     int64_t nrows, double *out) {
  return oracle_gemm_rows_fmt(A, sA, gA, lda, ORACLE_FMT_E4M3, B, sB, gB, ldb,
                              ORACLE_FMT_E4M3, M, N, K, rows, nrows, out);
}

int oracle_gemm_rows_fmt(const uint8_t *A, const float *sA, int gA,
                         int64_t lda, int fmtA, const uint8_t *B,
                         const float *sB, int gB, int64_t ldb, int fmtB,
                         int64_t M, int64_t N, int64_t K, const int64_t *rows,
                         int64_t nrows, double *out) {
  if (!A || !sA || !B || !sB || !rows || !out) return -1;
  if ((fmtA != ORACLE_FMT_E4M3 && fmtA != ORACLE_FMT_E5M2) ||
      (fmtB != ORACLE_FMT_E4M3 && fmtB != ORACLE_FMT_E5M2))
    return -1;
  if (M <= 0 || N <= 0 || K <= 0 || lda < K || ldb < K || nrows < 0)
    return -1;
  if (!pair_supported(gA, gB)) return -1;
  int blocked = gA == ORACLE_BLOCK_1x128;
  if (blocked && K % 128) return -1;
  if (gB == ORACLE_BLOCK_128x128 && N % 128) return -1;

  __int128 vA[256], vB[256];
  int shift = images(fmtA, vA) + images(fmtB, vB);
  int both_e4m3 = fmtA == ORACLE_FMT_E4M3 && fmtB == ORACLE_FMT_E4M3;
  /* the runs of k on which both scales are constant */
  int64_t run = blocked ? 128 : K;

  for (int64_t i = 0; i < nrows; ++i) {
    int64_t m = rows[i];
    if (m < 0 || m >= M) return -1;
    for (int64_t n = 0; n < N; ++n) {
      __float128 acc = 0;
      for (int64_t k0 = 0; k0 < K; k0 += run) {
        __int128 dot = 0;
        if (both_e4m3) { /* |v_A v_B| < 2^36: the run's sum fits int64 */
          int64_t d = 0;
          for (int64_t k = k0; k < k0 + run; ++k)
            d += (int64_t)vA[A[m * lda + k]] * (int64_t)vB[B[n * ldb + k]];
          dot = d;
        } else {
          for (int64_t k = k0; k < k0 + run; ++k)
            dot += vA[A[m * lda + k]] * vB[B[n * ldb + k]];
        }
        double sa = scale_at(sA, gA, M, K, m, k0);
        double sb = scale_at(sB, gB, N, K, n, k0);
        acc += (__float128)(sa * sb) * (__float128)dot;
      }
      out[i * N + n] = (double)ldexpq_(acc, -shift); /* exact power of two */
    }
  }
  return 0;
}
