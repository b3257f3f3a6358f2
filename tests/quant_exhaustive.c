/*
 * Exhaustive check of the activation quantize's reciprocal path (the 8-bit
 * activation cast of FlashDrive Sec. 3.4, read as per-token absmax / 127 with
 * round-half-even codes).
 *
 * The kernels do not divide each element by the token scale.  With the
 * row's absmax a >= 2^-96 they form, in IEEE binary32:
 *     s   = fl(a / 127)        (the stored scale)
 *     inv = fl(1 / s)
 *     p   = fl(x * inv)
 *     e   = fma(-s, p, x)      (the exact residual x - s p, rounded once)
 *     r   = fma(e, inv, p)     (one Markstein correction of the quotient)
 *     code = low byte of the bits of fl(r + 1.5 * 2^23)
 * This program checks, for every pair of bf16 values (x, a) with a a finite
 * normal >= 2^-96 and |x| <= a, that the code equals the definition
 *     (int8) nearbyint(fl(x / s))      (round-half-even, no clamp reached)
 * and prints the number of pairs and of mismatches.  It must be built with
 * -ffp-contract=off so that the separately rounded products stay separate.
 * Threads split the range of a.
 *
 * Usage: quant_exhaustive [threads [variant [a_first a_last]]]
 *   variant 0 (default) checks the kernels' formula; variant 1 drops the
 *   correction (code from p itself), a formula known to be wrong for some
 *   pairs, so that a run with it shows that the check can fail.  a_first and
 *   a_last (hex bf16 patterns, inclusive) narrow the range of a.
 */
#include <fenv.h>
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

static float from_bf16(uint32_t b) {
  uint32_t u = b << 16;
  float f;
  memcpy(&f, &u, 4);
  return f;
}

static uint32_t bits(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  return u;
}

/* bf16 patterns of a: 2^-96 (biased exponent 31) up to the largest finite value */
#define A_FIRST 0x0F80u
#define A_LAST 0x7F7Fu

static int g_variant = 0;

struct job {
  uint32_t a_lo, a_hi; /* [a_lo, a_hi) */
  long pairs, bad;
  uint32_t bad_x, bad_a;
};

static void* run(void* arg) {
  struct job* j = (struct job*)arg;
  fesetround(FE_TONEAREST);
  for (uint32_t ab = j->a_lo; ab < j->a_hi; ++ab) {
    const float a = from_bf16(ab);
    const float s = a / 127.0f;
    const float inv = 1.0f / s;
    /* every bf16 magnitude <= a, both signs */
    for (uint32_t mb = 0; mb <= ab; ++mb) {
      for (int sign = 0; sign < 2; ++sign) {
        if (sign && mb == 0) continue; /* -0 gives the code of +0 on both sides */
        const float x = from_bf16(mb | (sign ? 0x8000u : 0u));
        const float p = x * inv;
        const float e = fmaf(-s, p, x);
        const float r = g_variant == 1 ? p : fmaf(e, inv, p);
        const int8_t fast = (int8_t)(bits(r + 12582912.0f) & 0xFFu);
        const float q = nearbyintf(x / s);
        const int8_t ref = (int8_t)(q > 127.0f ? 127 : q < -127.0f ? -127 : (int)q);
        ++j->pairs;
        if (fast != ref) {
          if (!j->bad) {
            j->bad_x = mb | (sign ? 0x8000u : 0u);
            j->bad_a = ab;
          }
          ++j->bad;
        }
      }
    }
  }
  return NULL;
}

int main(int argc, char** argv) {
  int nthreads = argc > 1 ? atoi(argv[1]) : 8;
  if (nthreads < 1) nthreads = 1;
  if (nthreads > 256) nthreads = 256;
  if (argc > 2) g_variant = atoi(argv[2]);
  uint32_t a_first = A_FIRST, a_last = A_LAST;
  if (argc > 4) {
    a_first = (uint32_t)strtoul(argv[3], NULL, 16);
    a_last = (uint32_t)strtoul(argv[4], NULL, 16);
    if (a_first < A_FIRST || a_last > A_LAST || a_first > a_last) {
      fprintf(stderr, "a range outside [0x%04x, 0x%04x]\n", A_FIRST, A_LAST);
      return 2;
    }
  }
  /* the work for a grows with a's pattern (~2 ab pairs): split the pattern
   * range so that every thread gets about the same number of pairs */
  struct job jobs[256];
  pthread_t tid[256];
  const double lo2 = (double)a_first * a_first, hi2 = (double)(a_last + 1) * (a_last + 1);
  uint32_t prev = a_first;
  for (int t = 0; t < nthreads; ++t) {
    uint32_t next = t == nthreads - 1 ? a_last + 1 : (uint32_t)sqrt(lo2 + (hi2 - lo2) * (t + 1) / nthreads);
    if (next < prev) next = prev;
    jobs[t] = (struct job){prev, next, 0, 0, 0, 0};
    prev = next;
  }
  for (int t = 0; t < nthreads; ++t) pthread_create(&tid[t], NULL, run, &jobs[t]);
  long pairs = 0, bad = 0;
  uint32_t bx = 0, ba = 0;
  for (int t = 0; t < nthreads; ++t) {
    pthread_join(tid[t], NULL);
    pairs += jobs[t].pairs;
    if (jobs[t].bad && !bad) {
      bx = jobs[t].bad_x;
      ba = jobs[t].bad_a;
    }
    bad += jobs[t].bad;
  }
  printf("pairs=%ld mismatches=%ld", pairs, bad);
  if (bad) printf(" first: x=0x%04x a=0x%04x", bx, ba);
  printf("\n");
  return bad != 0;
}
