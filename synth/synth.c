/*
 * Seeded synthetic inputs (see synth.h).  Plain C99 + pthreads.
 *
 * Counter layout (all draws are independent functions of their counter):
 *   stream 0: matrix entries, element e = i*N + j uses counters 8e .. 8e+7
 *   stream 1: row scales, row i uses counters 2i, 2i+1
 *   other streams: vectors (caller-chosen)
 */
#include "synth.h"

#include <math.h>
#include <pthread.h>
#include <string.h>
#include <unistd.h>

#define GOLDEN 0x9E3779B97F4A7C15ull

/* SplitMix64 output function. */
static uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

/* The (ctr+1)-th output of a SplitMix64 generator whose state starts at
 * key = mix64(seed + GOLDEN*(stream+1)). */
uint64_t eqs_u64(uint64_t seed, uint64_t stream, uint64_t ctr) {
  uint64_t key = mix64(seed + GOLDEN * (stream + 1));
  return mix64(key + GOLDEN * (ctr + 1));
}

double eqs_uniform(uint64_t seed, uint64_t stream, uint64_t ctr) {
  return ((double)(eqs_u64(seed, stream, ctr) >> 11) + 0.5) * 0x1p-53;
}

void eqs_normal_pair(uint64_t seed, uint64_t stream, uint64_t ctr,
                     double *z0, double *z1) {
  const double two_pi = 6.283185307179586476925286766559;
  double u1 = eqs_uniform(seed, stream, ctr);
  double u2 = eqs_uniform(seed, stream, ctr + 1);
  double r = sqrt(-2.0 * log(u1));
  *z0 = r * cos(two_pi * u2);
  *z1 = r * sin(two_pi * u2);
}

uint16_t eqs_to_bf16(double v) {
  if (v == 0.0) return signbit(v) ? 0x8000u : 0u;
  int e;
  double m = frexp(v, &e);            /* v = m * 2^e, 0.5 <= |m| < 1 */
  double r = nearbyint(ldexp(m, 8));  /* 8 significant bits, ties to even */
  float f = (float)ldexp(r, e - 8);   /* exact: <= 8 significant bits */
  uint32_t b;
  memcpy(&b, &f, sizeof b);
  return (uint16_t)(b >> 16);
}

static double entry(const eqs_weight_spec *s, uint64_t seed, uint64_t e) {
  uint64_t c = 8 * e;
  double z[8];
  if (s->kind == EQS_STUDENT_T) {
    int need = s->nu + 1; /* z[0] numerator, z[1..nu] chi-square terms */
    for (int k = 0; k < need; k += 2) eqs_normal_pair(seed, 0, c + k, &z[k], &z[k + 1]);
    double chi2 = 0.0;
    for (int k = 1; k <= s->nu; ++k) chi2 += z[k] * z[k];
    return z[0] / sqrt(chi2 / s->nu);
  }
  /* EQS_GAUSS_OUTLIER */
  eqs_normal_pair(seed, 0, c, &z[0], &z[1]);
  if (eqs_uniform(seed, 0, c + 2) < s->outlier_p)
    return eqs_uniform(seed, 0, c + 3) < 0.5 ? s->outlier_mag : -s->outlier_mag;
  return z[0];
}

typedef struct job {
  const eqs_weight_spec *spec;
  uint64_t seed;
  uint32_t N, r0, r1;
  uint16_t *w;
} job;

static void *run_rows(void *p) {
  job *j = (job *)p;
  for (uint32_t i = j->r0; i < j->r1; ++i) {
    double z0, z1;
    eqs_normal_pair(j->seed, 1, 2ull * i, &z0, &z1);
    double r = exp(j->spec->row_sigma * z0);
    uint16_t *row = j->w + (uint64_t)i * j->N;
    for (uint32_t c = 0; c < j->N; ++c)
      row[c] = eqs_to_bf16(r * entry(j->spec, j->seed, (uint64_t)i * j->N + c));
  }
  return NULL;
}

int eqs_weights(const eqs_weight_spec *spec, uint64_t seed, uint32_t M,
                uint32_t N, uint16_t *w, int nthreads) {
  if (!spec || !w || M == 0 || N == 0) return -1;
  if (spec->kind == EQS_STUDENT_T && (spec->nu < 1 || spec->nu > 7)) return -1;
  if (spec->kind != EQS_STUDENT_T && spec->kind != EQS_GAUSS_OUTLIER) return -1;
  if (nthreads <= 0) { /* one per online CPU, at most 16 */
    long n = sysconf(_SC_NPROCESSORS_ONLN);
    nthreads = n > 16 ? 16 : (n > 0 ? (int)n : 1);
  }
  if (nthreads > 64) nthreads = 64;
  if ((uint32_t)nthreads > M) nthreads = (int)M;
  pthread_t th[64];
  job jobs[64];
  for (int t = 0; t < nthreads; ++t) {
    jobs[t].spec = spec;
    jobs[t].seed = seed;
    jobs[t].N = N;
    jobs[t].r0 = (uint32_t)((uint64_t)M * t / nthreads);
    jobs[t].r1 = (uint32_t)((uint64_t)M * (t + 1) / nthreads);
    jobs[t].w = w;
  }
  int started = 0;
  for (int t = 1; t < nthreads; ++t) {
    if (pthread_create(&th[t], NULL, run_rows, &jobs[t]) != 0) break;
    started = t;
  }
  run_rows(&jobs[0]);
  for (int t = started + 1; t < nthreads; ++t) run_rows(&jobs[t]); /* not started */
  for (int t = 1; t <= started; ++t) pthread_join(th[t], NULL);
  return 0;
}

int eqs_vector(uint64_t seed, uint64_t stream, uint64_t n, uint16_t *x) {
  if (!x) return -1;
  for (uint64_t k = 0; k < n; k += 2) {
    double z0, z1;
    eqs_normal_pair(seed, stream, k, &z0, &z1);
    x[k] = eqs_to_bf16(z0);
    if (k + 1 < n) x[k + 1] = eqs_to_bf16(z1);
  }
  return 0;
}
