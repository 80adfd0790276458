/*
 * Oracle quantizer (test infrastructure only): Eq. 3 of the paper
 * (Sec. 2.2) applied independently to every scaling unit.
 *
 *   amax = max |x| over the unit                (exact)
 *   S    = RN32(amax / 448), S := 1 if that is 0
 *   code = Q_FP8(RN32(x / S))                    (oracle_e4m3_encode)
 *
 * Tensorwise, rowwise and blockwise units follow the paragraph on scaling
 * granularity in Sec. 2.2; the 1x128 / 128x1 / 128x128 block shapes are the
 * ones the FP8 linear layer uses for activations, wgrad operands and weights.
 *
 * With ORACLE_E5M2 the FP8 format is E5M2 instead: F_max = 57344 replaces
 * 448 in the scale and the codes are E5M2 (oracle_e5m2_encode).
 */
#include <math.h>
#include <stdlib.h>
#include <string.h>

#include "oracle.h"

static float bf16_to_float(uint16_t bits) {
  uint32_t w = (uint32_t)bits << 16;
  float f;
  memcpy(&f, &w, sizeof f);
  return f;
}

/* Granularity as seen on the transposed matrix. */
static int transposed_granularity(int g) {
  switch (g) {
    case ORACLE_ROW: return ORACLE_COL;
    case ORACLE_COL: return ORACLE_ROW;
    case ORACLE_BLOCK_1x128: return ORACLE_BLOCK_128x1;
    case ORACLE_BLOCK_128x1: return ORACLE_BLOCK_1x128;
    default: return g;
  }
}

static int64_t scale_count(int g, int64_t rows, int64_t cols) {
  switch (g) {
    case ORACLE_TENSOR: return 1;
    case ORACLE_ROW: return rows;
    case ORACLE_COL: return cols;
    case ORACLE_BLOCK_1x128: return rows * (cols / 128);
    case ORACLE_BLOCK_128x1: return (rows / 128) * cols;
    case ORACLE_BLOCK_128x128: return (rows / 128) * (cols / 128);
    default: return -1;
  }
}

/* Position in the scale array of the unit holding element (r, c) of a
 * [rows, cols] matrix quantized with granularity g (layouts in oracle.h). */
static int64_t scale_index(int g, int64_t rows, int64_t cols, int64_t r,
                           int64_t c) {
  switch (g) {
    case ORACLE_TENSOR: return 0;
    case ORACLE_ROW: return r;
    case ORACLE_COL: return c;
    case ORACLE_BLOCK_1x128: return (c / 128) * rows + r;
    case ORACLE_BLOCK_128x1: return (r / 128) * cols + c;
    case ORACLE_BLOCK_128x128: return (r / 128) * (cols / 128) + c / 128;
    default: return -1;
  }
}

/* F_max is 448 (E4M3) or 57344 (E5M2); both are exact in fp32. */
static float scale_from_amax(float amax, float fmax) {
  float s = amax / fmax; /* one correctly rounded fp32 division */
  if (s == 0.0f) s = 1.0f;
  return s;
}

/* The power-of-two variant (not the paper's scale): the smallest power of
 * two S with F_max S >= amax, at least 2^-127, and 1 for amax = 0.  Found
 * by exact comparisons of F_max * 2^k with amax in double. */
static float pow2_scale_from_amax(float amax, float fmax) {
  if (amax == 0.0f) return 1.0f;
  int k = ilogb(amax) - ilogb(fmax);
  while (ldexp((double)fmax, k) < (double)amax) ++k;
  while (ldexp((double)fmax, k - 1) >= (double)amax) --k;
  if (k < -127) k = -127;
  return (float)ldexp(1.0, k);
}

uint8_t oracle_cast_f32(float x, float scale) {
  float q = x / scale; /* one correctly rounded fp32 division */
  return oracle_e4m3_encode(q);
}

void oracle_cast_f32_array(const float *x, int64_t n, float scale,
                           uint8_t *codes) {
  for (int64_t i = 0; i < n; ++i) codes[i] = oracle_cast_f32(x[i], scale);
}

void oracle_cast_f32_e5m2_array(const float *x, int64_t n, float scale,
                                uint8_t *codes) {
  for (int64_t i = 0; i < n; ++i) codes[i] = oracle_e5m2_encode(x[i] / scale);
}

int oracle_quantize(const uint16_t *x_bf16, int64_t rows, int64_t cols,
                    int64_t ldx, int granularity, unsigned flags,
                    uint8_t *codes, int64_t ldc, float *scales) {
  if (!x_bf16 || !codes || !scales) return -1;
  if (rows <= 0 || cols <= 0 || ldx < cols) return -1;
  if (granularity < ORACLE_TENSOR || granularity > ORACLE_BLOCK_128x128)
    return -1;
  int splits_cols = granularity == ORACLE_BLOCK_1x128 ||
                    granularity == ORACLE_BLOCK_128x128;
  int splits_rows = granularity == ORACLE_BLOCK_128x1 ||
                    granularity == ORACLE_BLOCK_128x128;
  if ((splits_cols && cols % 128) || (splits_rows && rows % 128)) return -1;

  int transposed = (flags & ORACLE_OUT_TRANSPOSED) != 0;
  int64_t orows = transposed ? cols : rows;
  int64_t ocols = transposed ? rows : cols;
  int og = transposed ? transposed_granularity(granularity) : granularity;
  if (ldc < ocols) return -1;

  int64_t nunits = scale_count(og, orows, ocols);
  float *amax = (float *)calloc((size_t)nunits, sizeof(float));
  if (!amax) return -1;

  /* amax of every unit */
  for (int64_t r = 0; r < rows; ++r) {
    for (int64_t c = 0; c < cols; ++c) {
      float a = fabsf(bf16_to_float(x_bf16[r * ldx + c]));
      int64_t orr = transposed ? c : r, occ = transposed ? r : c;
      int64_t u = scale_index(og, orows, ocols, orr, occ);
      if (a > amax[u]) amax[u] = a;
    }
  }
  /* S of every unit */
  int pow2 = (flags & ORACLE_POW2_SCALE) != 0;
  int e5m2 = (flags & ORACLE_E5M2) != 0;
  float fmax = e5m2 ? 57344.0f : 448.0f;
  for (int64_t u = 0; u < nunits; ++u)
    scales[u] = pow2 ? pow2_scale_from_amax(amax[u], fmax)
                     : scale_from_amax(amax[u], fmax);
  /* codes */
  for (int64_t r = 0; r < rows; ++r) {
    for (int64_t c = 0; c < cols; ++c) {
      float x = bf16_to_float(x_bf16[r * ldx + c]);
      int64_t orr = transposed ? c : r, occ = transposed ? r : c;
      int64_t u = scale_index(og, orows, ocols, orr, occ);
      float q = x / scales[u]; /* one correctly rounded fp32 division */
      codes[orr * ldc + occ] = e5m2 ? oracle_e5m2_encode(q) : oracle_e4m3_encode(q);
    }
  }
  free(amax);
  return 0;
}
