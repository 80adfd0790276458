/*
 * Test helper: checks the quotient sequence the HIP quantizer uses for
 * RN32(x / S) against the correctly rounded division, over every pair of a
 * positive finite bf16 amax and a bf16 x with |x| <= amax (both signs, both
 * zeros), and reports the pairs whose E4M3 code (sign included) differs;
 * div_sweep_fmt does the same for E5M2 codes, with F_max = 57344.
 *
 * Kernel sequence, for S = RN32(amax / F_max) (1 if 0) and r = RN32(1 / S):
 *   q0 = RN(x r);  e = RN(q0 S - x) (one FMA);  q = RN(q0 - e r) (one FMA)
 * used when S >= 2^-90; smaller S take the IEEE division.  Host fmaf and
 * float multiply are the same IEEE operations as v_fma_f32 / v_mul_f32
 * with round-to-nearest-even and subnormals kept.
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <string.h>

static float f32(uint32_t b) { float x; memcpy(&x, &b, 4); return x; }

/* E4M3 code of an fp32 value, written from the format (sign, RNE,
 * clamp at 448), independent of the oracle. */
static uint32_t code_of(float v) {
  uint32_t s = signbit(v) ? 0x80u : 0u;
  double a = fabs((double)v);
  if (a >= 448.0) return s | 0x7Eu;
  int e2;
  (void)frexp(a, &e2);
  int E = (a == 0.0) ? -6 : e2 - 1;
  if (E < -6) E = -6;
  double q = nearbyint(ldexp(a, 3 - E));
  if (q >= 16.0) { q = 8.0; E += 1; }
  return s | (q < 8.0 ? (uint32_t)q : (uint32_t)(((E + 7) << 3) | ((int)q - 8)));
}

/* E5M2 code of an fp32 value, written from the format (sign, RNE, clamp
 * at 57344): 2 mantissa bits, normal binades from 2^-14, subnormal grid
 * 2^-16. */
static uint32_t code_of_e5m2(float v) {
  uint32_t s = signbit(v) ? 0x80u : 0u;
  double a = fabs((double)v);
  if (a >= 57344.0) return s | 0x7Bu;
  int e2;
  (void)frexp(a, &e2);
  int E = (a == 0.0) ? -14 : e2 - 1;
  if (E < -14) E = -14;
  double q = nearbyint(ldexp(a, 2 - E));
  if (q >= 8.0) { q = 4.0; E += 1; }
  return s | (q < 4.0 ? (uint32_t)q : (uint32_t)(((E + 15) << 2) | ((int)q - 4)));
}

struct job { uint32_t a_lo, a_hi; int e5m2; uint64_t pairs, bad; uint32_t bad_a, bad_x; };

static void *worker(void *p) {
  struct job *j = (struct job *)p;
  for (uint32_t ai = j->a_lo; ai < j->a_hi; ++ai) {
    float amax = f32(ai << 16);
    float S = amax / (j->e5m2 ? 57344.0f : 448.0f);
    if (S == 0.0f) S = 1.0f;
    float r = 1.0f / S;
    int fast = S >= 0x1p-90f;
    for (uint32_t xi = 0; xi <= ai; ++xi) {
      for (uint32_t sign = 0; sign <= 0x8000u; sign += 0x8000u) {
        float x = f32((xi | sign) << 16);
        float exact = x / S;
        float q;
        if (fast) {
          float q0 = x * r;
          float e = fmaf(q0, S, -x);
          q = fmaf(-e, r, q0);
        } else {
          q = x / S;
        }
        ++j->pairs;
        uint32_t cq = j->e5m2 ? code_of_e5m2(q) : code_of(q);
        uint32_t ce = j->e5m2 ? code_of_e5m2(exact) : code_of(exact);
        if (cq != ce) {
          if (!j->bad) { j->bad_a = ai; j->bad_x = xi | sign; }
          ++j->bad;
        }
      }
    }
  }
  return 0;
}

/* Returns the number of differing pairs; *pairs gets the count checked.
 * e5m2 selects the E5M2 codes and F_max. */
uint64_t div_sweep_fmt(int threads, int e5m2, uint64_t *pairs, uint32_t *bad_a, uint32_t *bad_x) {
  if (threads < 1) threads = 1;
  if (threads > 64) threads = 64;
  pthread_t tid[64];
  struct job jobs[64];
  /* positive finite bf16 amax 0x0001 .. 0x7F7F; the work per amax grows
   * with it, so split by equal shares of sum(amax) */
  double total = 0.5 * 0x7F7F * (double)0x7F80;
  uint32_t lo = 1;
  for (int t = 0; t < threads; ++t) {
    double target = total * (t + 1) / threads;
    uint32_t hi = (t == threads - 1) ? 0x7F80u : (uint32_t)sqrt(2.0 * target);
    if (hi < lo) hi = lo;
    if (hi > 0x7F80u) hi = 0x7F80u;
    jobs[t] = (struct job){lo, hi, e5m2, 0, 0, 0, 0};
    pthread_create(&tid[t], 0, worker, &jobs[t]);
    lo = hi;
  }
  uint64_t bad = 0, n = 0;
  *bad_a = *bad_x = 0;
  for (int t = 0; t < threads; ++t) {
    pthread_join(tid[t], 0);
    if (jobs[t].bad && !bad) { *bad_a = jobs[t].bad_a; *bad_x = jobs[t].bad_x; }
    bad += jobs[t].bad;
    n += jobs[t].pairs;
  }
  *pairs = n;
  return bad;
}

uint64_t div_sweep(int threads, uint64_t *pairs, uint32_t *bad_a, uint32_t *bad_x) {
  return div_sweep_fmt(threads, 0, pairs, bad_a, bad_x);
}
