/*
 * Oracle GEMM (test infrastructure only): the exact product of the
 * dequantized FP8 operands X_tilde = S_X * X_hat of Eq. 3 (paper Sec. 2.2),
 * i.e. the linear layer evaluated on the FP8-quantized forward/backward
 * operands (Sec. 3, the FP8-quantized forward passes; Sec. 5.3, the FP8
 * training engine).
 *
 *   C[m][n] = sum_k (S_A(m,k) * A_hat[m][k]) * (S_B(n,k) * B_hat[n][k])
 *
 * Every E4M3 value times 2^9 is an integer v with |v| <= 229376, so over a
 * run of k on which both scales are constant the sum of v_A * v_B is an
 * exact int64.  Each run then contributes S_A * S_B * I * 2^-18; S_A * S_B
 * is exact in fp64 (two 24-bit significands) and the product with I (< 2^51)
 * is exact in binary128, where the runs are summed.  The single final
 * rounding is to fp64.
 */
#include <math.h>
#include <stdlib.h>

#include "oracle.h"

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

int oracle_gemm_rows(const uint8_t *A, const float *sA, int gA, int64_t lda,
                     const uint8_t *B, const float *sB, int gB, int64_t ldb,
                     int64_t M, int64_t N, int64_t K, const int64_t *rows,
                     int64_t nrows, double *out) {
  if (!A || !sA || !B || !sB || !rows || !out) return -1;
  if (M <= 0 || N <= 0 || K <= 0 || lda < K || ldb < K || nrows < 0)
    return -1;
  if (!pair_supported(gA, gB)) return -1;
  int blocked = gA == ORACLE_BLOCK_1x128;
  if (blocked && K % 128) return -1;
  if (gB == ORACLE_BLOCK_128x128 && N % 128) return -1;

  /* integer image of every code: decode(c) * 2^9 */
  int64_t v[256];
  for (int c = 0; c < 256; ++c) {
    double d = oracle_e4m3_decode((uint8_t)c);
    v[c] = isnan(d) ? 0 : (int64_t)ldexp(d, 9);
  }
  /* the runs of k on which both scales are constant */
  int64_t run = blocked ? 128 : K;

  for (int64_t i = 0; i < nrows; ++i) {
    int64_t m = rows[i];
    if (m < 0 || m >= M) return -1;
    for (int64_t n = 0; n < N; ++n) {
      __float128 acc = 0;
      for (int64_t k0 = 0; k0 < K; k0 += run) {
        int64_t dot = 0;
        for (int64_t k = k0; k < k0 + run; ++k)
          dot += v[A[m * lda + k]] * v[B[n * ldb + k]];
        double sa = scale_at(sA, gA, M, K, m, k0);
        double sb = scale_at(sB, gB, N, K, n, k0);
        acc += (__float128)(sa * sb) * (__float128)dot;
      }
      out[i * N + n] = (double)(acc / 262144); /* 2^-18, exact */
    }
  }
  return 0;
}
