/*
 * Seeded synthetic inputs for the EntQuant decode path.
 *
 * This module only makes inputs: BF16 weight matrices with the value
 * distributions of the workloads (Student-t or Gaussian-with-outliers
 * entries times a log-normal per-row scale) and BF16 activation vectors.
 * It holds none of the method's arithmetic (no quantiser, no coder, no
 * dequantiser); both the product encoder and the test oracle take their
 * weights from here.
 *
 * Random numbers: a counter-based generator built on the SplitMix64
 * finaliser (Steele, Lea, Flood, "Fast splittable pseudorandom number
 * generators", OOPSLA 2014; constants as in Vigna's splitmix64.c).
 * Every draw is a pure function of (seed, stream, counter), so output is
 * identical for any thread count.
 */
#ifndef EQ_SYNTH_H
#define EQ_SYNTH_H
#include <stdint.h>
#include <stddef.h>

#ifdef __cplusplus
extern "C" {
#endif

/* One 64-bit draw for (seed, stream, counter). */
uint64_t eqs_u64(uint64_t seed, uint64_t stream, uint64_t ctr);

/* Uniform in the open interval (0,1): ((u >> 11) + 0.5) * 2^-53. */
double eqs_uniform(uint64_t seed, uint64_t stream, uint64_t ctr);

/* Two independent N(0,1) draws by Box-Muller from the uniforms at
 * counters ctr and ctr+1. */
void eqs_normal_pair(uint64_t seed, uint64_t stream, uint64_t ctr,
                     double *z0, double *z1);

/* Round a double to the nearest BF16 value (ties to even significand),
 * returned as its 16-bit pattern. Inputs are finite and well inside the
 * BF16 range here. */
uint16_t eqs_to_bf16(double v);

/* Entry distributions. */
enum {
  EQS_STUDENT_T = 1,      /* t with integer nu degrees of freedom       */
  EQS_GAUSS_OUTLIER = 2   /* N(0,1), replaced w.p. p by +-mag            */
};

typedef struct eqs_weight_spec {
  int32_t kind;           /* EQS_STUDENT_T or EQS_GAUSS_OUTLIER          */
  int32_t nu;             /* Student-t degrees of freedom (1..7)         */
  double row_sigma;       /* per-row scale r_i = exp(row_sigma * Z_i)    */
  double outlier_p;       /* EQS_GAUSS_OUTLIER: outlier probability      */
  double outlier_mag;     /* EQS_GAUSS_OUTLIER: outlier magnitude        */
} eqs_weight_spec;

/* Fill w[M*N] (row-major BF16 bit patterns) with
 * W_ij = bf16(r_i * e_ij).  Returns 0, or -1 on bad arguments.
 * nthreads <= 0 uses one thread per online CPU, at most 16 (at most 64
 * threads in any case). */
int eqs_weights(const eqs_weight_spec *spec, uint64_t seed, uint32_t M,
                uint32_t N, uint16_t *w, int nthreads);

/* Fill x[n] with bf16(N(0,1)) draws from (seed, stream). */
int eqs_vector(uint64_t seed, uint64_t stream, uint64_t n, uint16_t *x);

#ifdef __cplusplus
}
#endif
#endif
