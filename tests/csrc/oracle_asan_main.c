/*
 * Test driver: every oracle entry point on heap buffers of exactly the
 * sizes its contract names, for a build with AddressSanitizer and
 * UndefinedBehaviorSanitizer (any read or write past a buffer, any signed
 * overflow, shift or conversion out of range aborts the run).  Shapes
 * cover every granularity, flag and transposition, ragged last units
 * (rows and columns that are not multiples of 128 where the oracle takes
 * them, and its refusal where it does not), padded leading dimensions,
 * and every GEMM pair and format.  Exit status 0 when every call returns
 * what its contract says.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "oracle.h"

static uint64_t state = 0x9E3779B97F4A7C15ull;
static uint32_t next_u32(void) {
  state ^= state << 13;
  state ^= state >> 7;
  state ^= state << 17;
  return (uint32_t)(state >> 11);
}

/* a finite bf16 pattern: exponents spread over the normal range and
 * subnormals, both signs, zeros now and then */
static uint16_t finite_bf16(void) {
  uint32_t r = next_u32();
  if ((r & 63) == 0) return (uint16_t)(r & 0x8000u);
  uint32_t e = 100 + (r >> 8) % 60;        /* 2^-27 .. 2^32 */
  if ((r & 255) == 1) e = 0;               /* a subnormal */
  return (uint16_t)((r & 0x8000u) | (e << 7) | ((r >> 16) & 0x7Fu));
}

static void *xmalloc(size_t n) {
  void *p = malloc(n ? n : 1);
  if (!p) {
    fprintf(stderr, "out of memory\n");
    exit(2);
  }
  return p;
}

static int64_t scales_for(int64_t rows, int64_t cols, int g) {
  switch (g) {
    case ORACLE_TENSOR: return 1;
    case ORACLE_ROW: return rows;
    case ORACLE_COL: return cols;
    case ORACLE_BLOCK_1x128: return rows * ((cols + 127) / 128);
    case ORACLE_BLOCK_128x1: return ((rows + 127) / 128) * cols;
    default: return ((rows + 127) / 128) * ((cols + 127) / 128);
  }
}

static int quantize_case(int64_t rows, int64_t cols, int64_t pad, int g, unsigned flags) {
  const int transposed = (flags & ORACLE_OUT_TRANSPOSED) != 0;
  const int64_t ldx = cols + pad, orows = transposed ? cols : rows, ocols = transposed ? rows : cols;
  const int64_t ldc = ocols + pad;
  int og = g;
  if (transposed) {
    if (g == ORACLE_ROW) og = ORACLE_COL;
    else if (g == ORACLE_COL) og = ORACLE_ROW;
    else if (g == ORACLE_BLOCK_1x128) og = ORACLE_BLOCK_128x1;
    else if (g == ORACLE_BLOCK_128x1) og = ORACLE_BLOCK_1x128;
  }
  uint16_t *x = xmalloc(sizeof(uint16_t) * (size_t)(rows * ldx));
  for (int64_t i = 0; i < rows * ldx; ++i) x[i] = finite_bf16();
  uint8_t *codes = xmalloc((size_t)(orows * ldc));
  const int64_t ns = scales_for(orows, ocols, og);
  float *scales = xmalloc(sizeof(float) * (size_t)ns);
  const int rc = oracle_quantize(x, rows, cols, ldx, g, flags, codes, ldc, scales);
  free(x);
  free(codes);
  free(scales);
  /* a dimension that 128-blocks split must be a multiple of 128 */
  const int split_cols = g == ORACLE_BLOCK_1x128 || g == ORACLE_BLOCK_128x128;
  const int split_rows = g == ORACLE_BLOCK_128x1 || g == ORACLE_BLOCK_128x128;
  const int want = ((split_cols && cols % 128) || (split_rows && rows % 128)) ? -1 : 0;
  if (rc != want)
    fprintf(stderr, "quantize %lld x %lld g=%d flags=%u: rc %d, expected %d\n", (long long)rows, (long long)cols, g,
            flags, rc, want);
  return rc != want;
}

static int gemm_case(int64_t M, int64_t N, int64_t K, int gA, int gB, int fa, int fb) {
  const int64_t lda = K + 16, ldb = K + 32;
  uint8_t *A = xmalloc((size_t)(M * lda)), *B = xmalloc((size_t)(N * ldb));
  for (int64_t i = 0; i < M * lda; ++i) {
    uint8_t c = (uint8_t)next_u32();
    /* no NaN / infinity codes */
    A[i] = fa ? (uint8_t)((c & 0x80) | ((c & 0x7F) % 0x7C)) : (uint8_t)((c & 0x80) | ((c & 0x7F) % 0x7F));
  }
  for (int64_t i = 0; i < N * ldb; ++i) {
    uint8_t c = (uint8_t)next_u32();
    B[i] = fb ? (uint8_t)((c & 0x80) | ((c & 0x7F) % 0x7C)) : (uint8_t)((c & 0x80) | ((c & 0x7F) % 0x7F));
  }
  const int64_t na = scales_for(M, K, gA), nb = scales_for(N, K, gB);
  float *sA = xmalloc(sizeof(float) * (size_t)na), *sB = xmalloc(sizeof(float) * (size_t)nb);
  for (int64_t i = 0; i < na; ++i) sA[i] = ldexpf(1.0f + (float)(next_u32() % 1000) / 1000.0f, (int)(next_u32() % 20) - 10);
  for (int64_t i = 0; i < nb; ++i) sB[i] = ldexpf(1.0f + (float)(next_u32() % 1000) / 1000.0f, (int)(next_u32() % 20) - 10);
  const int64_t nrows = M < 5 ? M : 5;
  int64_t *rows = xmalloc(sizeof(int64_t) * (size_t)nrows);
  for (int64_t i = 0; i < nrows; ++i) rows[i] = (i * 7919) % M;
  rows[nrows - 1] = M - 1;
  double *out = xmalloc(sizeof(double) * (size_t)(nrows * N));
  const int rc = oracle_gemm_rows_fmt(A, sA, gA, lda, fa, B, sB, gB, ldb, fb, M, N, K, rows, nrows, out);
  int bad = rc != 0;
  for (int64_t i = 0; i < nrows * N && !bad; ++i) bad = !isfinite(out[i]);
  free(A);
  free(B);
  free(sA);
  free(sB);
  free(rows);
  free(out);
  if (bad) fprintf(stderr, "gemm %lld %lld %lld pair %d %d fmt %d %d: rc %d\n", (long long)M, (long long)N,
                   (long long)K, gA, gB, fa, fb, rc);
  return bad;
}

int main(void) {
  int fails = 0;
  /* codec, every code and a spread of fp32 values */
  for (int c = 0; c < 256; ++c) {
    (void)oracle_e4m3_decode((uint8_t)c);
    (void)oracle_e5m2_decode((uint8_t)c);
  }
  for (int i = 0; i < 200000; ++i) {
    uint32_t b = next_u32();
    float v;
    memcpy(&v, &b, 4);
    (void)oracle_e4m3_encode(v);
    (void)oracle_e5m2_encode(v);
  }
  {
    const int64_t n = 4099;
    float *x = xmalloc(sizeof(float) * n);
    uint8_t *c = xmalloc((size_t)n);
    for (int64_t i = 0; i < n; ++i) x[i] = ldexpf((float)((int)(next_u32() % 2001) - 1000), (int)(next_u32() % 40) - 20);
    oracle_cast_f32_array(x, n, 0.37f, c);
    oracle_cast_f32_e5m2_array(x, n, 3.0e-5f, c);
    free(x);
    free(c);
  }
  /* quantizer: every granularity and flag set, ragged and padded */
  const int64_t shapes[][2] = {{256, 384}, {272, 400}, {1, 128}, {300, 130}, {128, 128}};
  for (int s = 0; s < 5; ++s)
    for (int g = ORACLE_TENSOR; g <= ORACLE_BLOCK_128x128; ++g)
      for (unsigned flags = 0; flags < 8; ++flags)
        for (int pad = 0; pad <= 16; pad += 16) fails += quantize_case(shapes[s][0], shapes[s][1], pad, g, flags);
  /* GEMM: every pair, every format combination */
  const int pairs[][2] = {{ORACLE_TENSOR, ORACLE_TENSOR}, {ORACLE_ROW, ORACLE_ROW},
                          {ORACLE_BLOCK_1x128, ORACLE_BLOCK_128x128}, {ORACLE_BLOCK_1x128, ORACLE_BLOCK_1x128}};
  for (int p = 0; p < 4; ++p)
    for (int fa = 0; fa < 2; ++fa)
      for (int fb = 0; fb < 2; ++fb) {
        fails += gemm_case(67, 256, 384, pairs[p][0], pairs[p][1], fa, fb);
        fails += gemm_case(3, 128, 128, pairs[p][0], pairs[p][1], fa, fb);
      }
  if (fails) fprintf(stderr, "%d failed calls\n", fails);
  printf("oracle sanitizer run: %d failures\n", fails);
  return fails ? 1 : 0;
}
