/* Exhaustive check of the quantizer's fp32 division step.
 *
 * The kernel computes fl32(a / s) from r = fl32(1 / s) as
 *     q0 = fl32(a * r);  e = fma(q0, s, -a);  q = fma(-e, r, q0).
 * Scaling a or s by a power of two scales q0, e and q by the same power while
 * all of them stay in the normal range, so it suffices to check mantissas:
 *   (A) every fp32 a in [1, 2) against every divisor in [1, 2) with at most
 *       4 significant bits (the E4M3 block scales, and 6 and 7);
 *   (B) every bf16 a in [1, 2) against every fp32 divisor in [1, 2) (the
 *       tensor scale s32; X is bf16).
 * (C) signed zeros: a = +-0 returns a zero of the same sign, also with the
 *     zero divisor the kernel encodes as s = 0, r = 0.
 * (D) the two-term reciprocal step for the block-scale divisors: with rh =
 *     1 / s rounded toward zero and rl = fl32(fma(-rh, s, 1) / s) >= 0 (the
 *     residual 1 - rh s is exact), q = fma(a, rh, fl32(a * rl)).  Every fp32 a
 *     in [1, 2) against every divisor in [1, 2) with at most 4 significant
 *     bits, and signed zeros (rl >= 0 gives both addends the sign of a; also
 *     with the zero scale, rh = rl = 0).  Here the scaling argument
 *     additionally needs a * rl to stay normal.
 * (E) the same two-term step for the tensor scale (X / s32, X bf16): s32 has
 *     24 significant bits and the step is not exact for every pair, so the
 *     kernel checks the 128 bf16 mantissas against s32 at launch and falls
 *     back to Markstein's step when one differs.  This part lists every fp32
 *     s32 in [1, 2) with such a mantissa (and the mantissas), which the GPU
 *     tests use to drive the fallback; it is a census, not a pass/fail check.
 * Exit status 0 iff every case of (A)-(D) equals the IEEE quotient (C's a / s,
 * correctly rounded to nearest even).  Built with -mfma so fmaf is one fused
 * operation.
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdio.h>
#include <string.h>

static float from_bits(uint32_t b) { float x; memcpy(&x, &b, 4); return x; }
static uint32_t to_bits(float x) { uint32_t b; memcpy(&b, &x, 4); return b; }

static float step(float a, float s, float r) {
  const float q0 = a * r;
  /* volatile keeps the compiler from rewriting -fma(q0, s, -a) as
     fma(-q0, s, a), which differs for a zero a (the kernel's compiler keeps
     the form as written) */
  volatile float e = fmaf(q0, s, -a);
  return fmaf(-e, r, q0);
}

static int same_as_ieee(float a, float s) {
  volatile float r = 1.0f / s;
  volatile float want = a / s;
  return to_bits(step(a, s, r)) == to_bits(want);
}

static float step2(float a, float rh, float rl) {
  volatile float t = a * rl;
  return fmaf(a, rh, t);
}

/* rh = 1 / s rounded toward zero, rl = the remainder (1 - rh s) / s >= 0 */
static void two_term_reciprocal(float s, float* rh, float* rl) {
  volatile float h = 1.0f / s;
  volatile float e = fmaf(-h, s, 1.0f);
  if (e < 0.0f) {
    h = from_bits(to_bits(h) - 1u);
    e = fmaf(-h, s, 1.0f);
  }
  *rh = h;
  *rl = e / s;
}

typedef struct { uint32_t lo, hi; long bad; } range_t;

enum { kMaxCensus = 64 };
typedef struct { uint32_t lo, hi; int n; uint32_t s[kMaxCensus], a[kMaxCensus]; } census_t;

static void* part_e(void* p) {
  census_t* j = (census_t*)p;
  for (uint32_t sm = j->lo; sm < j->hi; ++sm) {
    const float s = from_bits(0x3F800000u | sm);
    float rh, rl;
    two_term_reciprocal(s, &rh, &rl);
    for (uint32_t am = 0; am < 128; ++am) {
      const float a = from_bits(0x3F800000u | (am << 16));
      volatile float want = a / s;
      if (to_bits(step2(a, rh, rl)) != to_bits(want) && j->n < kMaxCensus) {
        j->s[j->n] = to_bits(s);
        j->a[j->n] = to_bits(a);
        j->n++;
      }
    }
  }
  return NULL;
}

static void* part_b(void* p) {
  range_t* j = (range_t*)p;
  for (uint32_t sm = j->lo; sm < j->hi; ++sm) {
    const float s = from_bits(0x3F800000u | sm);
    for (uint32_t am = 0; am < 128; ++am)
      if (!same_as_ieee(from_bits(0x3F800000u | (am << 16)), s)) j->bad++;
  }
  return NULL;
}

int main(void) {
  long bad_a = 0, bad_b = 0, bad_c = 0;
  for (uint32_t m = 0; m < 8; ++m) {
    const float s = 1.0f + (float)m / 8.0f;
    for (uint32_t am = 0; am < (1u << 23); ++am)
      if (!same_as_ieee(from_bits(0x3F800000u | am), s)) bad_a++;
  }
  enum { kThreads = 8 };
  pthread_t t[kThreads];
  range_t jobs[kThreads];
  for (int i = 0; i < kThreads; ++i) {
    jobs[i].lo = (1u << 23) / kThreads * (uint32_t)i;
    jobs[i].hi = (1u << 23) / kThreads * (uint32_t)(i + 1);
    jobs[i].bad = 0;
    pthread_create(&t[i], NULL, part_b, &jobs[i]);
  }
  for (int i = 0; i < kThreads; ++i) {
    pthread_join(t[i], NULL);
    bad_b += jobs[i].bad;
  }
  const float divisors[] = {1.0f, 1.375f, 6.0f, 7.0f, 448.0f, 0x1p-9f, 3.0e-5f};
  for (unsigned i = 0; i < sizeof divisors / sizeof divisors[0]; ++i) {
    const float s = divisors[i], r = 1.0f / s;
    if (to_bits(step(0.0f, s, r)) != 0u) bad_c++;
    if (to_bits(step(-0.0f, s, r)) != 0x80000000u) bad_c++;
  }
  const float dividends[] = {0.0f, -0.0f, 1.5f, -1.5f, 0x1p-20f, -3000.0f};
  for (unsigned i = 0; i < sizeof dividends / sizeof dividends[0]; ++i) {
    const float a = dividends[i], q = step(a, 0.0f, 0.0f);
    if (q != 0.0f || signbit(q) != signbit(a)) bad_c++;
  }
  long bad_d = 0;
  for (uint32_t m = 0; m < 8; ++m) {
    const float s = 1.0f + (float)m / 8.0f;
    float rh, rl;
    two_term_reciprocal(s, &rh, &rl);
    if (rl < 0.0f || signbit(rl)) bad_d++;
    for (uint32_t am = 0; am < (1u << 23); ++am) {
      const float a = from_bits(0x3F800000u | am);
      volatile float want = a / s;
      if (to_bits(step2(a, rh, rl)) != to_bits(want)) bad_d++;
    }
    if (to_bits(step2(0.0f, rh, rl)) != 0u) bad_d++;
    if (to_bits(step2(-0.0f, rh, rl)) != 0x80000000u) bad_d++;
  }
  for (unsigned i = 0; i < sizeof dividends / sizeof dividends[0]; ++i) {
    const float a = dividends[i], q = step2(a, 0.0f, 0.0f);
    if (q != 0.0f || signbit(q) != signbit(a)) bad_d++;
  }
  printf("A: %ld of %ld mismatched\n", bad_a, 8L << 23);
  printf("B: %ld of %ld mismatched\n", bad_b, 128L << 23);
  printf("C: %ld signed-zero mismatches\n", bad_c);
  printf("D: %ld of %ld mismatched (two-term reciprocal)\n", bad_d, 8L << 23);
  census_t cj[kThreads];
  for (int i = 0; i < kThreads; ++i) {
    cj[i].lo = (1u << 23) / kThreads * (uint32_t)i;
    cj[i].hi = (1u << 23) / kThreads * (uint32_t)(i + 1);
    cj[i].n = 0;
    pthread_create(&t[i], NULL, part_e, &cj[i]);
  }
  int n_e = 0;
  for (int i = 0; i < kThreads; ++i) {
    pthread_join(t[i], NULL);
    n_e += cj[i].n;
  }
  printf("E: %d tensor-scale pairs take the fallback\n", n_e);
  for (int i = 0; i < kThreads; ++i)
    for (int k = 0; k < cj[i].n; ++k) printf("E s32 0x%08x X 0x%08x\n", cj[i].s[k], cj[i].a[k]);
  return (bad_a || bad_b || bad_c || bad_d) ? 1 : 0;
}
