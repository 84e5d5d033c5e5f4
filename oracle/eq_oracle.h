/*
 * EntQuant CPU oracle -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, scalar C implementation of what the decode path computes,
 * used to check the GPU library.  Only the test suite, the package smoke
 * check and the CPU-baseline leg of the benchmark may load it; the product
 * library never links, calls or falls back to it.  It shares no code with
 * the product library.
 *
 * Paper: "Float8@2bits: Entropy Coding Enables Data-Free Model
 * Compression" (EntQuant, arXiv 2601.22787).
 *   Sec. 2.1  quantiser Q (round to nearest representable value of the
 *             base format, clamp to +-Qmax), AbsMax scale, dequantiser
 *             W_hat = s * W_q, channel-wise scales (one per output row),
 *             linear layer y = x W_hat^T + b.
 *   Sec. 2.2  empirical entropy (eq. emp_entropy); Alg. 1 (AbsMax init,
 *             scale choice, quantise, vec, ANS encode); Alg. 2 (ANS decode,
 *             view, QMatMul + bias).
 *   App. A.1  Float8 E4M3 base format, signed zeros resolved, byte-level
 *             ANS in fixed-size chunks.
 *   Sec. 3.5  Int8 as the alternative base format (symmetric, Sec. 2.1).
 *   App. B.1  closed-form entropy of a sparse mixture, Tab. sparsity_entropy.
 *
 * The paper's ANS coder is a closed library whose format it does not give.
 * The coder here is interleaved rANS (Duda 2014; Giesen 2014 for the
 * interleaving), with these parameters, all recorded in the container:
 *   P      probability precision, M = 2^P: 1 <= P <= 12 for the coder
 *          functions; a container takes 8 <= P <= 12 (a decoder may then
 *          compute f * (x >> P) with 24-bit operands)
 *   W      lanes: independent coder states per chunk (multiple of 64)
 *   state  32-bit, normalised interval [2^16, 2^32), 16-bit stream words
 * Symbol k of a chunk belongs to lane k mod W at step k div W.
 *
 * Every floating-point reading the paper leaves open is fixed here:
 *   E4M3FN (OCP), Qmax = 448, ties to even, clamp before rounding, one
 *   fp32 division W/s, -0 stored as +0, BF16 scales
 *   s = bf16(fp64(alpha * absmax / 448)) (all-zero row: s = 1),
 *   dequantised weight = bf16(s * v(q)) rounded once from the exact product.
 * Int8: Qmax = 127 (0x80 never occurs), clamp, then nearest integer with
 *   ties to even; s = bf16(fp64(alpha * absmax / 127)).
 *
 * Parity pins for every function are in the test suite; none is unpinned.
 */
#ifndef EQ_ORACLE_H
#define EQ_ORACLE_H
#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define OR_OK 0
#define OR_EINVAL (-1)
#define OR_EFORMAT (-2)
#define OR_ECORRUPT (-4)
#define OR_ENOMEM (-5)

/* ---- number formats (Sec. 2.1, App. A.1; Int8: Sec. 3.5 ablation) ---- */
#define OR_FMT_E4M3 1 /* Float8 E4M3FN, Qmax 448 (the default base format) */
#define OR_FMT_INT8 2 /* Int8 two's complement, symmetric, Qmax 127 */
double or_e4m3_value(uint8_t code);   /* NaN for 0x7F / 0xFF */
uint8_t or_e4m3_round(float v);       /* nearest E4M3FN code, ties to even */
double or_int8_value(uint8_t code);   /* (int8_t)code */
uint8_t or_int8_round(float v);       /* nearest integer in [-127, 127], ties to even */
double or_qmax(uint32_t fmt);
double or_code_value(uint32_t fmt, uint8_t code);
double or_bf16_value(uint16_t bits);
uint16_t or_bf16_round(double v);     /* nearest BF16, ties to even */

/* ---- entropy (eq. emp_entropy; App. B.1) ---- */
double or_entropy_counts(const uint64_t *counts, uint32_t n_bins);
double or_entropy_codes(const uint8_t *q, uint64_t n);
double or_sparsity_entropy(double s, double h_nz);

/* ---- quantiser / dequantiser (Sec. 2.1) ---- */
void or_row_scales(const uint16_t *w, uint32_t M, uint32_t N, float alpha, uint32_t fmt,
                   uint16_t *scale);
void or_quantize(const uint16_t *w, uint32_t M, uint32_t N, const uint16_t *scale, uint32_t fmt,
                 uint8_t *q);
void or_dequant(const uint8_t *q, uint32_t M, uint32_t N, const uint16_t *scale, uint32_t fmt,
                uint16_t *w_hat);
/* Bisection on log2(alpha) in [-4, 24] for the alpha whose entropy is
 * closest to target (the stand-in for the paper's lambda optimisation). */
float or_alpha_search(const uint16_t *w, uint32_t M, uint32_t N, double target_bits,
                      uint32_t fmt, double *h_out);

/* ---- frequency table (ANS metadata) ---- */
int or_freq_table(const uint64_t counts[256], uint32_t P, uint8_t *sym, uint16_t *freq,
                  uint32_t *K);

/* ---- one chunk of interleaved rANS ---- */
int or_rans_encode(const uint8_t *q, uint32_t n, uint32_t lanes, uint32_t P,
                   const uint8_t *sym, const uint16_t *freq, uint32_t K,
                   uint16_t *words, uint32_t max_words, uint32_t *n_words, uint32_t *states);
int or_rans_decode(const uint16_t *words, uint32_t n_words, const uint32_t *states,
                   uint32_t n, uint32_t lanes, uint32_t P, const uint8_t *sym,
                   const uint16_t *freq, uint32_t K, uint8_t *q);

/* ---- container (all sections of one compressed layer) ---- */
typedef struct or_info {
  uint32_t rows, cols, chunk_syms, n_chunks, lanes, prob_bits, n_syms, base_format;
  uint64_t total_words, padded_words, seed, file_bytes;
  float alpha, target_bits, entropy_bits;
  uint64_t off_scale, off_sym, off_freq, off_chunk_off, off_chunk_state, off_words;
} or_info;

int or_container_build(const uint16_t *w, uint32_t M, uint32_t N, float alpha, uint32_t fmt,
                       uint32_t P, uint32_t chunk_syms, uint32_t lanes, uint64_t seed,
                       float target_bits, uint8_t **blob, uint64_t *blob_bytes);
void or_free(void *p);
int or_container_info(const uint8_t *blob, uint64_t blob_bytes, or_info *info);
int or_container_decode_chunk(const uint8_t *blob, uint64_t blob_bytes, uint32_t chunk,
                              uint8_t *q);
int or_container_decode(const uint8_t *blob, uint64_t blob_bytes, uint8_t *q);

/* ---- scale optimisation (Sec. 2.2 eq. optimization; Alg. 1) ----
 * F(S) = sum|W - S*W_q| / sum|W| + lambda * sum|W_q| / (M N), W_q = Q(W/S)
 * (u = W/S in fp32, as the quantiser), with the straight-through gradient
 * dQ/du = 1 where |u| <= Qmax and 0 where the clamp acts. */
double or_rd_objective(const uint16_t *w, uint32_t M, uint32_t N, uint32_t fmt, double lambda,
                       const double *s, double *grad, double *dist);
/* Generic L-BFGS with a fixed step (two-loop recursion), for the objective
 * fg (returns f, writes the gradient); lower (optional) bounds each x_i from
 * below; returns the best iterate in x and its f in *f_out. */
typedef double (*or_fg_fn)(const double *x, double *g, void *ctx);
int or_lbfgs(uint32_t n, double *x, or_fg_fn fg, void *ctx, const double *lower, uint32_t iters,
             uint32_t history, double lr, double *f_out);
/* AbsMax start, then or_lbfgs on or_rd_objective with lower bound 1e-6 x start. */
int or_rd_scales(const uint16_t *w, uint32_t M, uint32_t N, uint32_t fmt, double lambda,
                 uint32_t iters, uint32_t history, double lr, double *s_out, double *f_out);
/* Test problem for or_lbfgs: f(x) = 1/2 sum a_i (x_i - c_i)^2 + 1/2 b (sum (x_i - c_i))^2. */
int or_lbfgs_quadratic(uint32_t n, const double *a, double b, const double *c, uint32_t iters,
                       uint32_t history, double lr, double *x, double *f_out);
/* Container with the given BF16 scales (else as or_container_build; alpha 0). */
int or_container_build_scaled(const uint16_t *w, uint32_t M, uint32_t N, const uint16_t *scale,
                              uint32_t fmt, uint32_t P, uint32_t chunk_syms, uint32_t lanes,
                              uint64_t seed, float target_bits, uint8_t **blob,
                              uint64_t *blob_bytes);

/* ---- container version 2: tile order and aligned phrases (eq_phrase.c) ----
 * Tiles of TR rows x TC columns are the chunks (row s of a tile is the
 * segment of coder state s); each segment is coded as aligned quads, pairs
 * and single codes from a per-layer dictionary; rANS at M = 2^16 with
 * frequencies in multiples of 2^(16-R). */
typedef struct or_info2 {
  uint32_t rows, cols, chunk_syms, n_chunks, lanes, prob_bits, n_syms, base_format;
  uint32_t tile_cols, n_quads, n_pairs, n_singles, tau;
  uint64_t total_words, padded_words, seed, file_bytes;
  float alpha, target_bits, entropy_bits;
  uint64_t off_scale, off_phr, off_freq, off_chunk_off, off_chunk_state, off_words;
  uint32_t flags;      /* bit 0: the rows are tiled in a stored order       */
  uint64_t off_order;  /* the order section (M uint32), 0 without one       */
} or_info2;

/* counts of n symbols (each >= 1) to frequencies >= 1 summing to 2^R, by the
 * rule of or_freq_table (a frequency of 2^16 is stored as 0) */
int or_freq_norm(const uint64_t *cnt, uint32_t n, uint32_t R, uint16_t *freq);
void or_tile_geometry(uint32_t M, uint32_t N, uint32_t TR, uint32_t TC, uint32_t c,
                      uint32_t *row0, uint32_t *col0, uint32_t *rows, uint32_t *cols);
/* DQ (<= 2^(R-1) values, quad share threshold tau * 2^-(R+2)) and DP
 * (<= 2^(R-2) values), each ascending */
int or_phrase_dict(const uint8_t *q, uint32_t M, uint32_t N, uint32_t TR, uint32_t TC,
                   uint32_t R, uint32_t tau, uint32_t *quads, uint32_t *n_quads, uint32_t *pairs,
                   uint32_t *n_pairs);
/* symbol indices of one segment (quads, then pairs, then singles) */
int or_phrase_parse(const uint8_t *u, uint32_t w, const uint32_t *quads, uint32_t nq,
                    const uint32_t *pairs, uint32_t np, const uint8_t *singles, uint32_t ns,
                    uint32_t *out, uint32_t *n_out);
int or_prans_encode(const uint32_t *tok, const uint64_t *off, const uint32_t *len, uint32_t W,
                    const uint16_t *freq, uint32_t n_sym, uint32_t R, uint16_t *words,
                    uint64_t max_words, uint64_t *n_words, uint32_t *states);
int or_prans_decode(const uint16_t *words, uint64_t n_words, const uint32_t *states,
                    const uint32_t *need, uint32_t W, const uint16_t *freq, const uint8_t *plen,
                    uint32_t n_sym, uint32_t R, uint32_t *tok, const uint64_t *off,
                    uint32_t *got);
/* row_order 1: tiles cut over the rows by ascending phrase count (eq_phrase.c,
 * item 4); 0: matrix order */
int or_container2_build(const uint16_t *w, uint32_t M, uint32_t N, float alpha,
                        const uint16_t *given_scale, uint32_t fmt, uint32_t R, uint32_t TR,
                        uint32_t TC, uint32_t row_order, uint64_t seed, float target_bits,
                        uint8_t **blob, uint64_t *blob_bytes);
int or_container2_info(const uint8_t *blob, uint64_t blob_bytes, or_info2 *info);
/* the matrix row of stored row k (info from or_container2_info) */
uint32_t or_container2_row(const uint8_t *blob, const or_info2 *info, uint32_t k);
int or_container2_decode_chunk(const uint8_t *blob, uint64_t blob_bytes, uint32_t chunk,
                               uint8_t *tile);
int or_container2_decode(const uint8_t *blob, uint64_t blob_bytes, uint8_t *q);

/* ---- linear layer (Sec. 2.1): y[b][i] = sum_j w_hat[i][j] x[b][j] + bias[i] in fp64 ---- */
void or_gemv(const uint16_t *w_hat, uint32_t M, uint32_t N, const uint16_t *x, uint32_t B,
             const uint16_t *bias, double *y);

#ifdef __cplusplus
}
#endif
#endif
