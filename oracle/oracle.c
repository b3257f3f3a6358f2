/*
 * CPU oracle for the W4A8 linear layer  y = dequant(quant8(x) . int4(W)^T).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may include, link,
 * load or call this file.  It exists so that tests/, the package smoke check
 * and the CPU-baseline leg of bench.py can compare the HIP kernels with a
 * plain, slow, obviously correct definition.  It shares no code, header,
 * table or constant with the GPU sources.
 *
 * What the method computes (FlashDrive, Sec. 3.4 "Quantization"): backbone
 * weights are held as 4-bit integers and the activations entering every
 * backbone linear layer are cast to 8 bits, so the product runs on integer
 * hardware (Sec. 4.2, "Algorithm-level gains", reading Table 1: prefill gains
 * from the INT8 contraction, decode from the 4x smaller weight stream).  The paper fixes
 * no scale granularity, rounding or output precision; the readings used here are:
 *   - activations: per-token symmetric scale s = absmax/127 (fp32), codes
 *     q = clamp(round_half_even(x / s), -127, 127), an all-zero row has s = 0
 *     and q = 0;
 *   - weights: two's-complement integers in [-8, 7] with either one fp32
 *     scale per output channel, or one fp16 scale per 128 consecutive k per
 *     output channel;
 *   - contraction: exact integer sum, here in int64, k ascending;
 *   - dequant: the real value is y = s_x[m] * s_w[n] * acc[m,n] (per
 *     channel) or y = s_x[m] * sum_g s_g[g][n] * p_g[m,n] (group), reported
 *     in fp64; the fp32 value y32 follows one fixed op order,
 *     ((float)acc * s_x) * s_w, resp. t += (float)p_g * s_g (no fma) then
 *     t * s_x, and the bf16 output is the round-to-nearest-even of y32.
 * The quantization decision (an fp32 quotient rounded to an integer) is made
 * in fp32 because that is the precision the kernel takes it in; every other
 * reference value is an integer or fp64.
 *
 * Build: gcc -O2 -ffp-contract=off -std=c11 -fPIC -shared -pthread.
 * Parity pins for every function live in tests/test_oracle.py.
 */
#define _POSIX_C_SOURCE 200809L
#include <fenv.h>
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORACLE_OK 0
#define ORACLE_EINVAL 1
#define ORACLE_ENONFINITE 2
#define ORACLE_EOVERFLOW 3

#define GROUP 128

/* bf16 bit pattern -> float: the bf16 value is the upper half of an IEEE
 * binary32 pattern, so the conversion is exact. */
float oracle_bf16_to_f32(uint16_t b) {
  uint32_t u = (uint32_t)b << 16;
  float f;
  memcpy(&f, &u, sizeof f);
  return f;
}

/* float -> bf16, round to nearest, ties to even, on the bit pattern.  NaN
 * maps to the canonical quiet NaN 0x7FC0. */
uint16_t oracle_f32_to_bf16(float f) {
  uint32_t u;
  memcpy(&u, &f, sizeof u);
  if ((u & 0x7F800000u) == 0x7F800000u && (u & 0x007FFFFFu) != 0) return 0x7FC0;
  uint32_t lsb = (u >> 16) & 1u;
  u += 0x7FFFu + lsb;
  return (uint16_t)(u >> 16);
}

/* IEEE binary16 bit pattern -> float, written out from the format
 * definition: sign, 5-bit biased exponent, 10-bit fraction. */
float oracle_f16_to_f32(uint16_t h) {
  int sign = (h >> 15) & 1;
  int e = (h >> 10) & 0x1F;
  int m = h & 0x3FF;
  float v;
  if (e == 0) {
    v = ldexpf((float)m, -24);              /* subnormal: m * 2^-24 */
  } else if (e == 31) {
    v = m ? NAN : INFINITY;
  } else {
    v = ldexpf((float)(m | 0x400), e - 25); /* (1024 + m) * 2^(e-15-10) */
  }
  return sign ? -v : v;
}

/* Per-token symmetric int8 quantization of one row of K bf16 values. */
static int quantize_row(const uint16_t* x, int64_t K, int8_t* q, float* s_out) {
  float a = 0.0f;
  for (int64_t k = 0; k < K; ++k) {
    float v = oracle_bf16_to_f32(x[k]);
    if (!isfinite(v)) return ORACLE_ENONFINITE;
    float av = fabsf(v);
    if (av > a) a = av;
  }
  if (a == 0.0f) {
    *s_out = 0.0f;
    for (int64_t k = 0; k < K; ++k) q[k] = 0;
    return ORACLE_OK;
  }
  float s = a / 127.0f;                 /* one fp32 IEEE division */
  *s_out = s;
  for (int64_t k = 0; k < K; ++k) {
    float r = oracle_bf16_to_f32(x[k]) / s; /* one fp32 IEEE division */
    float t = nearbyintf(r);                /* ties to even (FE_TONEAREST) */
    if (t > 127.0f) t = 127.0f;
    if (t < -127.0f) t = -127.0f;
    q[k] = (int8_t)t;
  }
  return ORACLE_OK;
}

int oracle_quantize_act(const uint16_t* x, int64_t M, int64_t K, int8_t* q, float* s) {
  if (M < 0 || K < 1 || (M > 0 && (!x || !q || !s))) return ORACLE_EINVAL;
  if (fegetround() != FE_TONEAREST) return ORACLE_EINVAL;
  for (int64_t m = 0; m < M; ++m) {
    int rc = quantize_row(x + m * K, K, q + m * K, s + m);
    if (rc) return rc;
  }
  return ORACLE_OK;
}

/* ---- linear layer ------------------------------------------------------ */

typedef struct {
  const int8_t* q; const float* s_x;
  const int8_t* w; const float* s_w; const uint16_t* s_g;
  int64_t M, N, K;
  int64_t m0, m1;
  int32_t* acc_out; float* y32_out; uint16_t* y_out; double* y64_out; double* bound_out;
  int rc;
} job_t;

static void* linear_rows(void* arg) {
  job_t* j = (job_t*)arg;
  const int64_t N = j->N, K = j->K, G = K / GROUP;
  const int group_mode = j->s_g != NULL;
  int64_t* part = NULL;
  if (group_mode) {
    part = (int64_t*)malloc((size_t)G * sizeof(int64_t));
    if (!part) { j->rc = ORACLE_EINVAL; return NULL; }
  }
  for (int64_t m = j->m0; m < j->m1; ++m) {
    const int8_t* qm = j->q + m * K;
    const float sx = j->s_x[m];
    for (int64_t n = 0; n < N; ++n) {
      const int8_t* wn = j->w + n * K;
      int64_t acc = 0;
      if (group_mode) {
        for (int64_t g = 0; g < G; ++g) {
          int64_t p = 0;
          for (int64_t k = g * GROUP; k < (g + 1) * GROUP; ++k) p += (int64_t)qm[k] * (int64_t)wn[k];
          part[g] = p;
          acc += p;
        }
      } else {
        for (int64_t k = 0; k < K; ++k) acc += (int64_t)qm[k] * (int64_t)wn[k];
      }
      if (acc > INT32_MAX || acc < INT32_MIN) { j->rc = ORACLE_EOVERFLOW; free(part); return NULL; }
      const int64_t o = m * N + n;
      if (j->acc_out) j->acc_out[o] = (int32_t)acc;
      float y32;
      double y64, bound;
      if (group_mode) {
        float t = 0.0f;
        double t64 = 0.0, b64 = 0.0;
        for (int64_t g = 0; g < G; ++g) {
          float sg = oracle_f16_to_f32(j->s_g[g * N + n]);
          float prod = (float)part[g] * sg;   /* separate multiply ... */
          t = t + prod;                       /* ... and add (no fma)  */
          t64 += (double)part[g] * (double)sg;
          b64 += fabs((double)part[g]) * (double)sg;
        }
        y32 = t * sx;
        y64 = t64 * (double)sx;
        bound = b64 * (double)sx;
      } else {
        float f = (float)acc;
        y32 = (f * sx) * j->s_w[n];
        y64 = (double)acc * (double)sx * (double)j->s_w[n];
        bound = fabs(y64);
      }
      if (j->y32_out) j->y32_out[o] = y32;
      if (j->y_out) j->y_out[o] = oracle_f32_to_bf16(y32);
      if (j->y64_out) j->y64_out[o] = y64;
      if (j->bound_out) j->bound_out[o] = bound;
    }
  }
  free(part);
  return NULL;
}

/*
 * Full linear layer on already quantized activations.
 *   q      int8 [M][K] codes, s_x fp32 [M] per-token scales
 *   w      int8 [N][K] weight integers in [-8, 7] (unpacked, row = output channel)
 *   s_w    fp32 [N] per-channel scales, or NULL
 *   s_g    fp16 bits [K/128][N] group scales, or NULL (exactly one of s_w, s_g)
 * Outputs (each may be NULL), all [M][N] row-major:
 *   acc_out int32 sum over all K; y32_out fp32 in the fixed op order; y_out bf16
 *   of y32; y64_out fp64 real value; bound_out fp64 cancellation-free
 *   magnitude s_x * sum_g |p_g| s_g (group) or |y64| (per channel).
 * nthreads > 1 splits the token rows over POSIX threads; results do not
 * depend on it.
 */
int oracle_linear_q(const int8_t* q, const float* s_x, int64_t M, int64_t K,
                    const int8_t* w, int64_t N, const float* s_w, const uint16_t* s_g,
                    int nthreads,
                    int32_t* acc_out, float* y32_out, uint16_t* y_out,
                    double* y64_out, double* bound_out) {
  if (M < 0 || N < 1 || K < 1) return ORACLE_EINVAL;
  if ((s_w == NULL) == (s_g == NULL)) return ORACLE_EINVAL;
  if (s_g && K % GROUP) return ORACLE_EINVAL;
  if (M == 0) return ORACLE_OK;
  if (!q || !s_x || !w) return ORACLE_EINVAL;
  for (int64_t i = 0; i < N * K; ++i)
    if (w[i] < -8 || w[i] > 7) return ORACLE_EINVAL;
  if (nthreads < 1) nthreads = 1;
  if (nthreads > M) nthreads = (int)M;
  job_t* jobs = (job_t*)calloc((size_t)nthreads, sizeof(job_t));
  pthread_t* th = (pthread_t*)calloc((size_t)nthreads, sizeof(pthread_t));
  if (!jobs || !th) { free(jobs); free(th); return ORACLE_EINVAL; }
  for (int t = 0; t < nthreads; ++t) {
    job_t* j = &jobs[t];
    j->q = q; j->s_x = s_x; j->w = w; j->s_w = s_w; j->s_g = s_g;
    j->M = M; j->N = N; j->K = K;
    j->m0 = M * t / nthreads; j->m1 = M * (t + 1) / nthreads;
    j->acc_out = acc_out; j->y32_out = y32_out; j->y_out = y_out;
    j->y64_out = y64_out; j->bound_out = bound_out; j->rc = ORACLE_OK;
  }
  for (int t = 1; t < nthreads; ++t) pthread_create(&th[t], NULL, linear_rows, &jobs[t]);
  linear_rows(&jobs[0]);
  for (int t = 1; t < nthreads; ++t) pthread_join(th[t], NULL);
  int rc = ORACLE_OK;
  for (int t = 0; t < nthreads; ++t) if (jobs[t].rc) rc = jobs[t].rc;
  free(jobs); free(th);
  return rc;
}

/* The whole path from bf16 activations: quantize each token, then
 * oracle_linear_q.  q_out [M][K] and sx_out [M] may be NULL. */
int oracle_linear(const uint16_t* x, int64_t M, int64_t K,
                  const int8_t* w, int64_t N, const float* s_w, const uint16_t* s_g,
                  int nthreads, int8_t* q_out, float* sx_out,
                  int32_t* acc_out, float* y32_out, uint16_t* y_out,
                  double* y64_out, double* bound_out) {
  if (M < 0 || K < 1) return ORACLE_EINVAL;
  if (M == 0) return ORACLE_OK;
  int8_t* q = q_out ? q_out : (int8_t*)malloc((size_t)(M * K));
  float* s = sx_out ? sx_out : (float*)malloc((size_t)M * sizeof(float));
  int rc = (!q || !s) ? ORACLE_EINVAL : oracle_quantize_act(x, M, K, q, s);
  if (rc == ORACLE_OK)
    rc = oracle_linear_q(q, s, M, K, w, N, s_w, s_g, nthreads, acc_out, y32_out, y_out, y64_out, bound_out);
  if (!q_out) free(q);
  if (!sx_out) free(s);
  return rc;
}
