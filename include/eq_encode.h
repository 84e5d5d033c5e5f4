/*
 * libeq host encoder: builds the compressed-layer container that the decode
 * entry points of eq.h consume.
 *
 * It follows the encoding scheme of the paper (EntQuant, arXiv 2601.22787,
 * Sec. 2.2, Alg. 1): per-output-row scales starting from AbsMax
 * (eq. absmax), quantisation Q (Sec. 2.1) to the base format -- Float8
 * E4M3FN (Qmax 448) or Int8 (Qmax 127, the ablation of Sec. 3.5) --,
 * row-major flattening, then ANS entropy coding in fixed-size chunks
 * (App. A.1).
 * The scale choice here is a single multiplier alpha on the AbsMax scales,
 * chosen so that the codes reach a target empirical entropy
 * (eq. emp_entropy); it stands in for the paper's lambda-regularised scale
 * optimisation.  Container layout: see eq.h.
 *
 * Host memory only; no GPU is touched.  Thread-safe; every call is
 * independent.
 */
#ifndef EQ_ENCODE_H
#define EQ_ENCODE_H
#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct eqe_params {
  uint32_t prob_bits;   /* P: probability precision, 8..12 (12 recommended)          */
  uint32_t chunk_syms;  /* C: symbols per chunk, a positive multiple of lanes       */
  uint32_t lanes;       /* W: interleaved coder states per chunk, 64, 128 or 256    */
  uint32_t threads;     /* worker threads; 0 = one per online CPU, at most 16       */
  uint64_t seed;        /* recorded in the header (generator seed), not used        */
  float target_bits;    /* recorded in the header, not used                         */
  uint32_t base_format; /* 1 = E4M3FN (0 is read as 1), 2 = Int8                    */
} eqe_params;

/* Bisection on log2(alpha) over [-4, 24] (40 steps) for the alpha whose codes'
 * empirical entropy is closest to target_bits.  If sample_rows > 0 and
 * smaller than M, the search quantises only sample_rows evenly spaced rows.
 * base_format: as in eqe_params.  *h_out (optional) receives the entropy of
 * the chosen alpha over the rows searched.  Returns alpha, or a negative
 * value on bad arguments. */
float eqe_alpha_search(const uint16_t *w_bf16, uint32_t M, uint32_t N, double target_bits,
                       uint32_t sample_rows, uint32_t threads, uint32_t base_format,
                       double *h_out);

/* Quantise w (M x N BF16, row-major, host) with scales bf16(alpha * absmax /
 * Qmax) to the base format of params and encode it.  On success *blob receives a buffer from malloc holding the
 * whole container (free it with eqe_free) and *blob_bytes its size.
 * Returns 0, -1 (bad arguments: M*N >= 2^32, lanes not 64/128/256, C not a
 * multiple of lanes, P outside 8..12, unknown base format) or -5 (out of memory). */
int eqe_encode(const uint16_t *w_bf16, uint32_t M, uint32_t N, float alpha,
               const eqe_params *params, uint8_t **blob, uint64_t *blob_bytes);

/* Encode w with the given per-row scales (BF16 bit patterns, M of them,
 * each positive and within [2^-117, 2^120)) instead of alpha * AbsMax, e.g.
 * the result of eqe_rd_scales.  Same outputs and return codes as eqe_encode
 * (-1 also for an unusable scale); the header's alpha field is 0. */
int eqe_encode_scaled(const uint16_t *w_bf16, uint32_t M, uint32_t N, const uint16_t *scale_bf16,
                      const eqe_params *params, uint8_t **blob, uint64_t *blob_bytes);

/* ---- scale optimisation: Sec. 2.2, eq. optimization (Alg. 1) ----
 * F(S) = ||W - S W_q||_1 / ||W||_1 + lambda * ||W_q||_1 / (M N),  W_q = Q(W / S),
 * minimised over the per-row scales S from the AbsMax start (eq. absmax)
 * with L-BFGS and the straight-through estimator for Q's rounding. */
typedef struct eqe_rd_params {
  double lambda;        /* regularisation weight (>= 0)                              */
  double lr;            /* L-BFGS step length; <= 0: 0.25 if lambda > 30, else 1.0  */
  uint32_t iters;       /* L-BFGS iterations; 0: 200                                 */
  uint32_t history;     /* L-BFGS curvature pairs kept; 0: 20                        */
  uint32_t threads;     /* 0: one per online CPU, at most 16                         */
  uint32_t base_format; /* 1 = E4M3FN (0 is read as 1), 2 = Int8                     */
} eqe_rd_params;

/* F at the scales `scale` (M positive doubles); *grad (optional, M doubles)
 * receives the straight-through gradient (dQ/du = 1 inside [-Qmax, Qmax], 0
 * where the clamp is active) and *distortion (optional) the first term.
 * Returns NaN on bad arguments. */
double eqe_rd_objective(const uint16_t *w_bf16, uint32_t M, uint32_t N, uint32_t base_format,
                        double lambda, const double *scale, uint32_t threads, double *grad,
                        double *distortion);

/* Optimise the scales; outputs (each optional): the scales as doubles, the
 * same rounded to BF16 (nearest, ties to even) for eqe_encode_scaled, and
 * the lowest F reached.  Returns 0, -1 (bad arguments) or -5 (memory). */
int eqe_rd_scales(const uint16_t *w_bf16, uint32_t M, uint32_t N, const eqe_rd_params *params,
                  double *scale, uint16_t *scale_bf16, double *objective);

/* lambda whose optimised BF16 scales give codes with empirical entropy
 * (eq. emp_entropy) closest to target_bits: bisection on log2(lambda) over
 * [-8, 16] (14 steps), optimising and measuring on sample_rows evenly spaced
 * rows (all rows if 0 or >= M); params->lambda is ignored.  Returns 0 and
 * writes *lambda and *h (entropy on the rows searched), or -1 / -5. */
int eqe_rd_lambda_search(const uint16_t *w_bf16, uint32_t M, uint32_t N, double target_bits,
                         uint32_t sample_rows, const eqe_rd_params *params, double *lambda,
                         double *h);

/* ---- container version 2 (decoded by the same entry points of eq.h) ----
 * Version 2 codes the same quantised codes with two choices of this library
 * where the paper leaves the coder to a closed one (App. A.1):
 *  - vec order: the M x N code matrix is cut into tiles of TR rows by TC
 *    columns (the last tile row and column may be smaller); tile (b, t),
 *    t < NT = ceil(N / TC), is chunk b * NT + t, and row s of a tile is the
 *    segment of coder state s (TR states per chunk), in column order;
 *  - alphabet: phrases.  A segment is parsed greedily from its start: the
 *    four codes at the position if they are in the quad dictionary DQ, else
 *    the two codes if they are in the pair dictionary DP, else one code.
 *    The alphabet is DQ, then DP, then the codes emitted alone (DS), each in
 *    ascending order of its codes read as a little-endian integer; the
 *    frequencies are the symbols' counts normalised to 2^R as for version 1.
 *    DP: the pairs at positions 0, 2, 4, ... of all segments whose count
 *    times 2^(R+2) is at least the number of pairs counted, at most the
 *    2^(R-2) most frequent (ties: lower value).  DQ: likewise for the quads
 *    at positions 0, 4, 8, ..., with the threshold tau times the number of
 *    quads counted and at most 2^(R-1) of them.  Entries the parse never
 *    emits are dropped.  tau is the one of 8, 4, 2, 1 whose alphabet needs
 *    the fewest bits, sum over symbols of count * log2(2^R / f) in fp64
 *    summed in alphabet order (ties: the larger tau);
 *  - coder: interleaved rANS with the state arithmetic at 2^16 and
 *    frequencies F = f * 2^(16 - R); step t decodes the t-th symbol of every
 *    state whose segment is not yet complete, then those states take a word
 *    in ascending order when x < 2^16 (layout of the container: eq.h);
 *  - row order (optional): the tiles are cut over the rows taken by
 *    ascending phrase count of their parse (summed over the row's segments;
 *    ties: lower row).  A tile takes as many decode steps as its longest
 *    segment has phrases, so alike rows in a tile shorten it.  The alphabet
 *    does not depend on the order. */
typedef struct eqe_params2 {
  uint32_t res_bits;    /* R: frequency resolution, 10..12 (12 recommended)          */
  uint32_t tile_rows;   /* TR: coder states per chunk, 64, 128 or 256                */
  uint32_t tile_cols;   /* TC: a positive multiple of 4                              */
  uint32_t threads;     /* worker threads; 0 = one per online CPU, at most 16       */
  uint64_t seed;        /* recorded in the header, not used                         */
  float target_bits;    /* recorded in the header, not used                         */
  uint32_t base_format; /* 1 = E4M3FN (0 is read as 1), 2 = Int8                    */
  uint32_t row_order;   /* 1: tiles cut over the rows by ascending phrase count
                           (ties: lower row), recorded in the order section; 0:
                           matrix order                                          */
} eqe_params2;

/* Quantise w (M x N BF16, host) with scales bf16(alpha * absmax / Qmax), or
 * with the given BF16 scales when scale_bf16 is non-null (alpha is then
 * recorded as 0), and write a version-2 container to *blob (malloc'd; free
 * with eqe_free).  Returns 0, -1 (bad arguments, including TR * TC >= 2^32
 * and an unusable given scale) or -5 (out of memory). */
int eqe_encode2(const uint16_t *w_bf16, uint32_t M, uint32_t N, float alpha,
                const uint16_t *scale_bf16, const eqe_params2 *params, uint8_t **blob,
                uint64_t *blob_bytes);

void eqe_free(void *p);

#ifdef __cplusplus
}
#endif
#endif
