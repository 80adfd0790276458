/*
 * Test helper for the GEMM with quantized output (test_gpu_d_gemm_quant.py):
 * the check of the 1x128 output units whose bf16 values the model bound
 * does not fix.  Each element of such a unit can hold any bf16 value of its
 * interval [lo, hi] (both zeros when the interval holds 0).  The unit
 * passes when
 *   - its GPU scale lies between RN32(amax_lo / 448) and RN32(amax_hi /
 *     448), amax_lo being the largest over the unit's elements of the
 *     smallest magnitude in the element's interval, amax_hi the largest
 *     magnitude of any of them (the scales of the smallest and largest amax
 *     the unit's bf16 values can have), and
 *   - every code is the oracle's cast, with that GPU scale, of some bf16
 *     value of its element's interval.
 * Bit patterns are bf16 ([rows][cols], cols = 128 units), codes E4M3,
 * scales [rows][units].  Returns the number of failing units and the first
 * (row, unit, what) with what = 1 for the scale, 2 for a code.
 */
#include <stdint.h>
#include <string.h>

#include "oracle.h"

static float bf(uint16_t b) {
  const uint32_t u = (uint32_t)b << 16;
  float f;
  memcpy(&f, &u, 4);
  return f;
}

/* Calls visit(c) for every bf16 pattern c of value in [bf(lo), bf(hi)], in
 * increasing value, -0 and +0 both when 0 is inside; returns the count. */
#define FOR_EACH_BF16(lo, hi, c, body)                  \
  do {                                                  \
    const float hi_v_ = bf(hi);                         \
    uint16_t c = (lo);                                  \
    while (bf(c) <= hi_v_) {                            \
      body;                                             \
      if (c == 0x8000) {                                \
        c = 0x0000;                                     \
      } else if (c == 0x0000) {                         \
        c = 0x0001;                                     \
      } else {                                          \
        c = (c & 0x8000) ? (uint16_t)(c - 1) : (uint16_t)(c + 1); \
      }                                                 \
    }                                                   \
  } while (0)

int64_t unit_check(const uint16_t *lo, const uint16_t *hi, const uint8_t *got, const float *scales,
                   const uint8_t *check, int64_t rows, int64_t cols, int64_t *first) {
  const int64_t units = cols / 128;
  int64_t bad = 0;
  for (int64_t r = 0; r < rows; ++r) {
    for (int64_t u = 0; u < units; ++u) {
      if (!check[r * units + u]) continue;
      const int64_t e0 = r * cols + u * 128;
      float amax_lo = 0.0f, amax_hi = 0.0f;
      for (int64_t k = 0; k < 128; ++k) {
        float mn = -1.0f, mx = 0.0f;
        FOR_EACH_BF16(lo[e0 + k], hi[e0 + k], c, {
          const float m = bf(c) < 0 ? -bf(c) : bf(c);
          if (mn < 0 || m < mn) mn = m;
          if (m > mx) mx = m;
        });
        if (mn > amax_lo) amax_lo = mn;
        if (mx > amax_hi) amax_hi = mx;
      }
      const float s_lo = amax_lo / 448.0f, s_hi = amax_hi / 448.0f, s = scales[r * units + u];
      int what = 0;
      if (!(s_lo <= s && s <= s_hi)) what = 1;
      for (int64_t k = 0; !what && k < 128; ++k) {
        int ok = 0;
        FOR_EACH_BF16(lo[e0 + k], hi[e0 + k], c, {
          if (!ok && oracle_cast_f32(bf(c), s) == got[e0 + k]) ok = 1;
        });
        if (!ok) what = 2;
      }
      if (what) {
        if (bad == 0) {
          first[0] = r;
          first[1] = u;
          first[2] = what;
        }
        ++bad;
      }
    }
  }
  return bad;
}
