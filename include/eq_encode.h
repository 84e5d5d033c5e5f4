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
  uint32_t prob_bits;   /* P: probability precision, 1..12 (12 recommended)          */
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
 * multiple of lanes, P outside 1..12, unknown base format) or -5 (out of memory). */
int eqe_encode(const uint16_t *w_bf16, uint32_t M, uint32_t N, float alpha,
               const eqe_params *params, uint8_t **blob, uint64_t *blob_bytes);

void eqe_free(void *p);

#ifdef __cplusplus
}
#endif
#endif
