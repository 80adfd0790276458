/*
 * OCP E4M3 codec for the oracle (test infrastructure only).
 *
 * Q_FP8 of Eq. 3 (paper Sec. 2.2) is "rounding and clamping to the FP8
 * representable set".  The set is OCP 8-bit floating point E4M3: 1 sign
 * bit, 4 exponent bits (bias 7), 3 mantissa bits, no infinities, NaN only at
 * S.1111.111, largest finite magnitude 448, subnormals m * 2^-9.
 */
#include <math.h>
#include <stdint.h>

#include "oracle.h"

double oracle_e4m3_decode(uint8_t code) {
  int sign = code >> 7;
  int e = (code >> 3) & 15;
  int m = code & 7;
  if (e == 15 && m == 7) return NAN;
  double mag;
  if (e == 0)
    mag = ldexp((double)m, -9);             /* subnormal: m/8 * 2^(1-7)   */
  else
    mag = ldexp((double)(8 + m), e - 10);   /* (1 + m/8) * 2^(e-7)        */
  return sign ? -mag : mag;
}

/* Rounding to the nearest member of the set by its definition: locate the
 * two non-negative finite neighbours of |v| (codes 0x00..0x7E are in
 * increasing order of value) and compare |v| with their midpoint.  A tie
 * goes to the neighbour whose mantissa is even, which is the even code. */
uint8_t oracle_e4m3_encode(float v) {
  if (isnan(v)) return 0x7F;
  uint8_t sign = signbit(v) ? 0x80 : 0x00;
  double a = fabs((double)v);
  if (a >= 448.0) return (uint8_t)(sign | 0x7E); /* clamp: 448 is the max */

  /* largest code lo in [0, 126] with decode(lo) <= a (decode(0) = 0 <= a) */
  int lo = 0, hi = 126; /* invariant: decode(lo) <= a < decode(hi) */
  while (hi - lo > 1) {
    int mid = (lo + hi) / 2;
    if (oracle_e4m3_decode((uint8_t)mid) <= a)
      lo = mid;
    else
      hi = mid;
  }
  double below = oracle_e4m3_decode((uint8_t)lo);
  double above = oracle_e4m3_decode((uint8_t)hi);
  double midpoint = 0.5 * (below + above); /* exact: 5 significant bits */
  int code;
  if (a < midpoint)
    code = lo;
  else if (a > midpoint)
    code = hi;
  else
    code = (lo % 2 == 0) ? lo : hi;
  return (uint8_t)(sign | code);
}
