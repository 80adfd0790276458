/*
 * OCP E5M2 codec for the oracle (test infrastructure only).
 *
 * The paper leaves "the chosen FP8 format" of Eq. 3 (Sec. 2.2) open; E5M2
 * for gradients is a variant offered next to E4M3.  OCP 8-bit floating
 * point E5M2: 1 sign bit, 5 exponent bits (bias 15), 2 mantissa bits,
 * infinities at S.11111.00, NaN at S.11111.{01,10,11}, largest finite
 * magnitude 57344 = 1.75 * 2^15, subnormals m * 2^-16.
 */
#include <math.h>
#include <stdint.h>

#include "oracle.h"

double oracle_e5m2_decode(uint8_t code) {
  int sign = code >> 7;
  int e = (code >> 2) & 31;
  int m = code & 3;
  double mag;
  if (e == 31)
    mag = (m == 0) ? INFINITY : NAN;
  else if (e == 0)
    mag = ldexp((double)m, -16);            /* subnormal: m/4 * 2^(1-15)  */
  else
    mag = ldexp((double)(4 + m), e - 17);   /* (1 + m/4) * 2^(e-15)       */
  return sign ? -mag : mag;
}

/* Q_FP8 into E5M2: the nearest finite member of the set, found by a search
 * of the increasing non-negative finite codes 0x00..0x7B and a comparison
 * with the midpoint of the two neighbours; a tie goes to the even code.
 * Magnitudes at or above 57344 clamp to 57344 (Q_FP8 clamps, so the
 * infinities are never produced). */
uint8_t oracle_e5m2_encode(float v) {
  if (isnan(v)) return 0x7F;
  uint8_t sign = signbit(v) ? 0x80 : 0x00;
  double a = fabs((double)v);
  if (a >= 57344.0) return (uint8_t)(sign | 0x7B);

  int lo = 0, hi = 0x7B; /* invariant: decode(lo) <= a < decode(hi) */
  while (hi - lo > 1) {
    int mid = (lo + hi) / 2;
    if (oracle_e5m2_decode((uint8_t)mid) <= a)
      lo = mid;
    else
      hi = mid;
  }
  double below = oracle_e5m2_decode((uint8_t)lo);
  double above = oracle_e5m2_decode((uint8_t)hi);
  double midpoint = 0.5 * (below + above); /* exact: 4 significant bits */
  int code;
  if (a < midpoint)
    code = lo;
  else if (a > midpoint)
    code = hi;
  else
    code = (lo % 2 == 0) ? lo : hi;
  return (uint8_t)(sign | code);
}
