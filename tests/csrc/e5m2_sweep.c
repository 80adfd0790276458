/*
 * Test helper: compares the oracle's E5M2 encoder with an independently
 * written one over ranges of fp32 bit patterns, on several threads.
 *
 * The independent encoder scales |v| onto the integer grid of its E5M2
 * binade with frexp/ldexp (exact), rounds with nearbyint under the default
 * round-to-nearest-even mode, and assembles the code from exponent and
 * mantissa fields (2 mantissa bits, bias 15, clamp at 57344).  It shares no
 * code with the oracle (which searches the value table and compares
 * against midpoints).
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <string.h>

extern uint8_t oracle_e5m2_encode(float v);

static uint8_t independent_encode(float v) {
  uint8_t sign = signbit(v) ? 0x80 : 0x00;
  double a = fabs((double)v);
  if (a >= 57344.0) return (uint8_t)(sign | 0x7B);
  int e2;
  (void)frexp(a, &e2);               /* a = f * 2^e2, f in [0.5, 1)        */
  int E = (a == 0.0) ? -14 : e2 - 1; /* a in [2^E, 2^(E+1))                */
  if (E < -14) E = -14;              /* subnormals share the E = -14 grid  */
  double q = nearbyint(ldexp(a, 2 - E)); /* multiples of 2^(E-2)           */
  if (q >= 8.0) { q = 4.0; E += 1; }     /* carried into the next binade   */
  int code;
  if (q < 4.0)                       /* only when E == -14: subnormal      */
    code = (int)q;
  else
    code = ((E + 15) << 2) | ((int)q - 4);
  return (uint8_t)(sign | code);
}

struct job {
  uint64_t start, end, stride;
  uint64_t mismatches, checked;
  uint32_t first_bad;
};

static void *worker(void *arg) {
  struct job *j = (struct job *)arg;
  j->mismatches = 0;
  j->checked = 0;
  j->first_bad = 0;
  for (uint64_t b = j->start; b < j->end; b += j->stride) {
    uint32_t bits = (uint32_t)b;
    float v;
    memcpy(&v, &bits, sizeof v);
    if (isnan(v)) continue;
    ++j->checked;
    if (oracle_e5m2_encode(v) != independent_encode(v)) {
      if (j->mismatches == 0) j->first_bad = bits;
      ++j->mismatches;
    }
  }
  return 0;
}

/* Checks bit patterns start, start+stride, ... < end.  Returns the number
 * of mismatches; *checked gets the number of non-NaN patterns compared and
 * *first_bad the first mismatching pattern. */
uint64_t sweep(uint64_t start, uint64_t end, uint64_t stride, int threads,
               uint64_t *checked, uint32_t *first_bad) {
  if (threads < 1) threads = 1;
  if (threads > 64) threads = 64;
  pthread_t tid[64];
  struct job jobs[64];
  uint64_t n = (end - start + stride - 1) / stride;
  uint64_t per = (n + threads - 1) / threads;
  for (int t = 0; t < threads; ++t) {
    uint64_t s = start + (uint64_t)t * per * stride;
    uint64_t e = s + per * stride;
    if (s > end) s = end;
    if (e > end) e = end;
    jobs[t].start = s;
    jobs[t].end = e;
    jobs[t].stride = stride;
    pthread_create(&tid[t], 0, worker, &jobs[t]);
  }
  uint64_t bad = 0, total = 0;
  *first_bad = 0;
  for (int t = 0; t < threads; ++t) {
    pthread_join(tid[t], 0);
    if (jobs[t].mismatches && !bad) *first_bad = jobs[t].first_bad;
    bad += jobs[t].mismatches;
    total += jobs[t].checked;
  }
  *checked = total;
  return bad;
}
