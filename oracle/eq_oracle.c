/*
 * EntQuant CPU oracle -- TEST INFRASTRUCTURE ONLY (see eq_oracle.h).
 *
 * Plain scalar C99, compiled without fast-math and without FMA
 * contraction.  Each function names the passage of the paper it follows.
 */
#include "eq_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>

/* ------------------------------------------------------------------ */
/* Number formats                                                      */
/* ------------------------------------------------------------------ */

/* E4M3FN (OCP 8-bit float; the Float8 base format of App. A.1):
 * sign S, exponent E (4 bits, bias 7), mantissa M (3 bits).
 *   E = 0       : (-1)^S * 2^-6 * M/8            (subnormal, incl. zero)
 *   E = 1..15   : (-1)^S * 2^(E-7) * (1 + M/8)
 *   E=15, M=7   : NaN (no infinities)                                   */
double or_e4m3_value(uint8_t code) {
  int s = code >> 7, e = (code >> 3) & 15, m = code & 7;
  if (e == 15 && m == 7) return NAN;
  double mag = (e == 0) ? ldexp(m / 8.0, -6) : ldexp(1.0 + m / 8.0, e - 7);
  return s ? -mag : mag;
}

/* Round to the nearest representable E4M3FN value (Sec. 2.1, "rounding to
 * the nearest representable value"), after clamping to [-Qmax, Qmax] with
 * Qmax = 448.  Ties go to the even code (even mantissa).  -0 becomes +0
 * (App. A.1: signed zeros resolved). */
uint8_t or_e4m3_round(float v) {
  double a = fabs((double)v);
  if (a > 448.0) a = 448.0;
  /* codes 0x00..0x7E are the non-negative finite values in increasing
   * order; find the largest one not above a (binary search) */
  int lo = 0, hi = 0x7E;
  while (lo < hi) {
    int mid = (lo + hi + 1) / 2;
    if (or_e4m3_value((uint8_t)mid) <= a) lo = mid;
    else hi = mid - 1;
  }
  int c = lo;
  if (or_e4m3_value((uint8_t)lo) != a) {
    double dlo = a - or_e4m3_value((uint8_t)lo);
    double dhi = or_e4m3_value((uint8_t)(lo + 1)) - a;
    if (dhi < dlo || (dhi == dlo && ((lo + 1) & 1) == 0)) c = lo + 1;
  }
  if (c == 0) return 0; /* +0 */
  return (uint8_t)((v < 0.0f ? 0x80 : 0x00) | c);
}

/* Int8 (the paper's alternative base format, Sec. 2.1 and Sec. 3.5):
 * two's complement byte, symmetric range [-Qmax, Qmax] with Qmax = 127, so
 * the code 0x80 (-128) never occurs. */
double or_int8_value(uint8_t code) { return (double)(int8_t)code; }

/* Nearest integer after clamping to [-127, 127] (Sec. 2.1 quantiser); a
 * value exactly halfway between two integers goes to the even one. */
uint8_t or_int8_round(float v) {
  double a = (double)v;
  if (a > 127.0) a = 127.0;
  if (a < -127.0) a = -127.0;
  double r = floor(a);
  double d = a - r; /* exact, in [0, 1) */
  if (d > 0.5 || (d == 0.5 && fmod(r, 2.0) != 0.0)) r += 1.0;
  int iv = (int)r;
  return (uint8_t)(int8_t)iv;
}

double or_qmax(uint32_t fmt) { return fmt == OR_FMT_INT8 ? 127.0 : 448.0; }

double or_code_value(uint32_t fmt, uint8_t code) {
  return fmt == OR_FMT_INT8 ? or_int8_value(code) : or_e4m3_value(code);
}

static uint8_t round_to_format(uint32_t fmt, float v) {
  return fmt == OR_FMT_INT8 ? or_int8_round(v) : or_e4m3_round(v);
}

double or_bf16_value(uint16_t bits) {
  uint32_t u = (uint32_t)bits << 16;
  float f;
  memcpy(&f, &u, sizeof f);
  return (double)f;
}

/* Nearest BF16 value (8 significant bits, fp32 exponent range), ties to the
 * even significand.  The two grid neighbours of |v| are found from the
 * binade of |v|; both differences are exact in fp64. */
uint16_t or_bf16_round(double v) {
  if (v == 0.0) return signbit(v) ? 0x8000 : 0x0000;
  double a = fabs(v);
  int e2;
  frexp(a, &e2);              /* a in [2^(e2-1), 2^e2) */
  int lsb_exp = e2 - 1 - 7;   /* spacing of 8-bit significands in that binade */
  if (lsb_exp < -133) lsb_exp = -133; /* BF16 subnormal spacing */
  double ulp = ldexp(1.0, lsb_exp);
  double k = floor(a / ulp);  /* exact: a/ulp < 2^9 */
  double lo = k * ulp, hi = (k + 1.0) * ulp;
  double pick;
  if (a - lo < hi - a) pick = lo;
  else if (a - lo > hi - a) pick = hi;
  else pick = (fmod(k, 2.0) == 0.0) ? lo : hi;
  float f = (float)pick;      /* exact */
  uint32_t u;
  memcpy(&u, &f, sizeof u);
  u >>= 16;
  if (v < 0.0) u |= 0x8000;
  return (uint16_t)u;
}

/* ------------------------------------------------------------------ */
/* Entropy                                                              */
/* ------------------------------------------------------------------ */

/* Empirical entropy, eq. emp_entropy: -(1/n) sum_k log2 p(x_k) with p the
 * relative frequency; summed per distinct value. */
double or_entropy_counts(const uint64_t *counts, uint32_t n_bins) {
  uint64_t n = 0;
  for (uint32_t i = 0; i < n_bins; ++i) n += counts[i];
  if (n == 0) return 0.0;
  double h = 0.0;
  for (uint32_t i = 0; i < n_bins; ++i) {
    if (counts[i] == 0) continue;
    double p = (double)counts[i] / (double)n;
    h -= p * log2(p);
  }
  return h;
}

double or_entropy_codes(const uint8_t *q, uint64_t n) {
  uint64_t counts[256] = {0};
  for (uint64_t k = 0; k < n; ++k) counts[q[k]]++;
  return or_entropy_counts(counts, 256);
}

/* App. B.1: H(s) = -s log2 s - (1-s) log2(1-s) + (1-s) H_nz. */
double or_sparsity_entropy(double s, double h_nz) {
  double h = 0.0;
  if (s > 0.0) h -= s * log2(s);
  if (s < 1.0) h -= (1.0 - s) * log2(1.0 - s);
  return h + (1.0 - s) * h_nz;
}

/* ------------------------------------------------------------------ */
/* Quantiser and dequantiser (Sec. 2.1)                                 */
/* ------------------------------------------------------------------ */

/* Channel-wise scales, one per output row.  AbsMax (eq. absmax) gives
 * max|W_i|/Qmax (Qmax of the base format); alpha multiplies it (alpha = 1
 * is plain AbsMax).  Stored in BF16. */
void or_row_scales(const uint16_t *w, uint32_t M, uint32_t N, float alpha, uint32_t fmt,
                   uint16_t *scale) {
  for (uint32_t i = 0; i < M; ++i) {
    double amax = 0.0;
    for (uint32_t j = 0; j < N; ++j) {
      double a = fabs(or_bf16_value(w[(uint64_t)i * N + j]));
      if (a > amax) amax = a;
    }
    scale[i] = (amax == 0.0) ? 0x3F80 /* 1.0 */
                             : or_bf16_round((double)alpha * amax / or_qmax(fmt));
  }
}

/* W_q = clamp(round(W/s), -Qmax, Qmax) with one fp32 division, rounded in
 * the base format. */
void or_quantize(const uint16_t *w, uint32_t M, uint32_t N, const uint16_t *scale, uint32_t fmt,
                 uint8_t *q) {
  for (uint32_t i = 0; i < M; ++i) {
    float s = (float)or_bf16_value(scale[i]);
    for (uint32_t j = 0; j < N; ++j) {
      uint64_t k = (uint64_t)i * N + j;
      float v = (float)or_bf16_value(w[k]) / s;
      q[k] = round_to_format(fmt, v);
    }
  }
}

/* W_hat = s * W_q: the product of the 8-bit BF16 significand and a code
 * value of at most 7 significant bits (4 for E4M3) is exact in fp32; it is
 * rounded once to BF16. */
void or_dequant(const uint8_t *q, uint32_t M, uint32_t N, const uint16_t *scale, uint32_t fmt,
                uint16_t *w_hat) {
  for (uint32_t i = 0; i < M; ++i) {
    double s = or_bf16_value(scale[i]);
    for (uint32_t j = 0; j < N; ++j) {
      uint64_t k = (uint64_t)i * N + j;
      w_hat[k] = or_bf16_round(s * or_code_value(fmt, q[k]));
    }
  }
}

static double entropy_at(const uint16_t *w, uint32_t M, uint32_t N, float alpha, uint32_t fmt,
                         uint16_t *scale, uint8_t *q) {
  or_row_scales(w, M, N, alpha, fmt, scale);
  or_quantize(w, M, N, scale, fmt, q);
  return or_entropy_codes(q, (uint64_t)M * N);
}

float or_alpha_search(const uint16_t *w, uint32_t M, uint32_t N, double target_bits,
                      uint32_t fmt, double *h_out) {
  uint16_t *scale = (uint16_t *)malloc(sizeof(uint16_t) * M);
  uint8_t *q = (uint8_t *)malloc((size_t)M * N);
  if (!scale || !q) {
    free(scale);
    free(q);
    return NAN;
  }
  double lo = -4.0, hi = 24.0;
  float best = 1.0f;
  double best_err = INFINITY, best_h = 0.0;
  for (int it = 0; it < 40; ++it) {
    double mid = 0.5 * (lo + hi);
    float alpha = (float)exp2(mid);
    double h = entropy_at(w, M, N, alpha, fmt, scale, q);
    double err = fabs(h - target_bits);
    if (err < best_err) {
      best_err = err;
      best = alpha;
      best_h = h;
    }
    if (h > target_bits) lo = mid; /* larger scale -> fewer levels -> lower entropy */
    else hi = mid;
  }
  free(scale);
  free(q);
  if (h_out) *h_out = best_h;
  return best;
}

/* ------------------------------------------------------------------ */
/* Frequency table: the ANS metadata of Sec. 2.2                        */
/* ------------------------------------------------------------------ */

/* Present symbols in ascending code order; f_k = max(1, floor(n_k 2^P / n));
 * a positive deficit is handed out one unit at a time in order of
 * decreasing remainder n_k 2^P mod n (ties: lower code first), cycling; a
 * negative one is taken one unit at a time from the largest f_k > 1 (ties:
 * lower code first).  Sum of f_k is exactly 2^P. */
int or_freq_table(const uint64_t counts[256], uint32_t P, uint8_t *sym, uint16_t *freq,
                  uint32_t *K_out) {
  if (P < 1 || P > 12) return OR_EINVAL;
  uint64_t M = 1ull << P, n = 0;
  uint32_t K = 0;
  uint64_t cnt[256], rem[256];
  int64_t f[256];
  for (int c = 0; c < 256; ++c) {
    if (counts[c] == 0) continue;
    sym[K] = (uint8_t)c;
    cnt[K] = counts[c];
    n += counts[c];
    ++K;
  }
  if (K == 0 || K > M) return OR_EINVAL;
  *K_out = K;
  if (K == 1) {
    freq[0] = (uint16_t)M;
    return OR_OK;
  }
  int64_t total = 0;
  for (uint32_t k = 0; k < K; ++k) {
    uint64_t scaled = cnt[k] * M;
    f[k] = (int64_t)(scaled / n);
    rem[k] = scaled % n;
    if (f[k] < 1) f[k] = 1;
    total += f[k];
  }
  int64_t d = (int64_t)M - total;
  if (d > 0) {
    /* order of decreasing remainder, ties by ascending code (stable) */
    uint32_t order[256];
    for (uint32_t k = 0; k < K; ++k) order[k] = k;
    for (uint32_t a = 1; a < K; ++a) { /* insertion sort, stable */
      uint32_t v = order[a];
      int32_t b = (int32_t)a - 1;
      while (b >= 0 && rem[order[b]] < rem[v]) {
        order[b + 1] = order[b];
        --b;
      }
      order[b + 1] = v;
    }
    for (uint32_t i = 0; d > 0; i = (i + 1) % K, --d) f[order[i]] += 1;
  }
  while (d < 0) {
    uint32_t best = K;
    for (uint32_t k = 0; k < K; ++k)
      if (f[k] > 1 && (best == K || f[k] > f[best])) best = k;
    if (best == K) return OR_EINVAL;
    f[best] -= 1;
    ++d;
  }
  for (uint32_t k = 0; k < K; ++k) freq[k] = (uint16_t)f[k];
  return OR_OK;
}

/* ------------------------------------------------------------------ */
/* Interleaved rANS, one chunk                                          */
/* ------------------------------------------------------------------ */

#define RANS_L 65536u /* lower end of the normalised state interval */

static int sym_index(const uint8_t *sym, uint32_t K, uint8_t code) {
  for (uint32_t k = 0; k < K; ++k)
    if (sym[k] == code) return (int)k;
  return -1;
}

/* Encode n symbols.  Steps t = T-1 .. 0, lanes W-1 .. 0 (active lanes
 * only): if x >= f * 2^(32-P) push the low 16 bits and shift x down by 16;
 * then x = floor(x/f) * 2^P + (x mod f) + cum.  The chunk's stream is the
 * pushed words in reverse order; the final x of each lane is stored. */
int or_rans_encode(const uint8_t *q, uint32_t n, uint32_t lanes, uint32_t P,
                   const uint8_t *sym, const uint16_t *freq, uint32_t K,
                   uint16_t *words, uint32_t max_words, uint32_t *n_words, uint32_t *states) {
  if (lanes == 0 || P < 1 || P > 12) return OR_EINVAL;
  uint64_t cum[256];
  uint64_t acc = 0;
  for (uint32_t k = 0; k < K; ++k) {
    cum[k] = acc;
    acc += freq[k];
  }
  if (acc != (1ull << P)) return OR_EINVAL;
  uint64_t *x = (uint64_t *)malloc(sizeof(uint64_t) * lanes);
  if (!x) return OR_ENOMEM;
  for (uint32_t l = 0; l < lanes; ++l) x[l] = RANS_L;
  uint32_t pushed = 0;
  uint32_t T = (n + lanes - 1) / lanes;
  for (uint32_t t = T; t-- > 0;) {
    for (uint32_t l = lanes; l-- > 0;) {
      uint64_t k = (uint64_t)t * lanes + l;
      if (k >= n) continue;
      int s = sym_index(sym, K, q[k]);
      if (s < 0) {
        free(x);
        return OR_EINVAL;
      }
      uint64_t f = freq[s];
      if (x[l] >= (f << (32 - P))) {
        if (pushed >= max_words) {
          free(x);
          return OR_ENOMEM;
        }
        words[pushed++] = (uint16_t)(x[l] & 0xFFFF);
        x[l] >>= 16;
      }
      x[l] = (x[l] / f) * (1ull << P) + (x[l] % f) + cum[s];
    }
  }
  for (uint32_t a = 0, b = pushed; a + 1 < b; ++a, --b) { /* reverse */
    uint16_t tmp = words[a];
    words[a] = words[b - 1];
    words[b - 1] = tmp;
  }
  for (uint32_t l = 0; l < lanes; ++l) states[l] = (uint32_t)x[l];
  *n_words = pushed;
  free(x);
  return OR_OK;
}

/* Decode n symbols.  Step t = 0 .. T-1: every active lane finds the symbol
 * whose interval [cum, cum+f) holds slot = x mod 2^P and sets
 * x = f * (x >> P) + slot - cum; then, in ascending lane order, each active
 * lane with x < 2^16 reads the next stream word: x = (x << 16) | word.
 * At the end every lane must be back at 2^16 and the stream used up
 * exactly; anything else is corruption. */
int or_rans_decode(const uint16_t *words, uint32_t n_words, const uint32_t *states,
                   uint32_t n, uint32_t lanes, uint32_t P, const uint8_t *sym,
                   const uint16_t *freq, uint32_t K, uint8_t *q) {
  if (lanes == 0 || P < 1 || P > 12) return OR_EINVAL;
  uint32_t M = 1u << P;
  uint32_t cum[257];
  cum[0] = 0;
  for (uint32_t k = 0; k < K; ++k) cum[k + 1] = cum[k] + freq[k];
  if (cum[K] != M) return OR_EINVAL;
  /* slot -> symbol index, from the intervals */
  uint16_t *slot_sym = (uint16_t *)malloc(sizeof(uint16_t) * M);
  uint64_t *x = (uint64_t *)malloc(sizeof(uint64_t) * lanes);
  if (!slot_sym || !x) {
    free(slot_sym);
    free(x);
    return OR_ENOMEM;
  }
  for (uint32_t k = 0; k < K; ++k)
    for (uint32_t s = cum[k]; s < cum[k + 1]; ++s) slot_sym[s] = (uint16_t)k;
  for (uint32_t l = 0; l < lanes; ++l) x[l] = states[l];
  int rc = OR_OK;
  uint32_t p = 0;
  uint32_t T = (n + lanes - 1) / lanes;
  for (uint32_t t = 0; t < T; ++t) {
    for (uint32_t l = 0; l < lanes; ++l) {
      uint64_t k = (uint64_t)t * lanes + l;
      if (k >= n) continue;
      uint32_t slot = (uint32_t)(x[l] & (M - 1));
      uint32_t s = slot_sym[slot];
      x[l] = (uint64_t)freq[s] * (x[l] >> P) + slot - cum[s];
      q[k] = sym[s];
    }
    for (uint32_t l = 0; l < lanes; ++l) {
      uint64_t k = (uint64_t)t * lanes + l;
      if (k >= n) continue;
      if (x[l] < RANS_L) {
        uint32_t wv = 0;
        if (p < n_words) wv = words[p];
        else rc = OR_ECORRUPT;
        ++p;
        x[l] = (x[l] << 16) | wv;
      }
    }
  }
  for (uint32_t l = 0; l < lanes; ++l)
    if (x[l] != RANS_L) rc = OR_ECORRUPT;
  if (p != n_words) rc = OR_ECORRUPT;
  free(slot_sym);
  free(x);
  return rc;
}

/* ------------------------------------------------------------------ */
/* Container: header (256 B) and 256-B aligned sections, little-endian. */
/* ------------------------------------------------------------------ */
/* header offsets */
enum {
  H_MAGIC = 0, H_VERSION = 4, H_HEADER_BYTES = 8, H_FORMAT = 12, H_ROWS = 16, H_COLS = 20,
  H_CHUNK = 24, H_NCHUNKS = 28, H_LANES = 32, H_PBITS = 36, H_NSYMS = 40, H_FLAGS = 44,
  H_TOTAL_WORDS = 48, H_PADDED_WORDS = 56, H_SEED = 64, H_ALPHA = 72, H_TARGET = 76,
  H_ENTROPY = 80, H_OFF_SCALE = 88, H_OFF_SYM = 96, H_OFF_FREQ = 104, H_OFF_CHUNK_OFF = 112,
  H_OFF_CHUNK_STATE = 120, H_OFF_WORDS = 128, H_FILE_BYTES = 136, HEADER_BYTES = 256
};

static void put32(uint8_t *b, size_t o, uint32_t v) {
  for (int i = 0; i < 4; ++i) b[o + i] = (uint8_t)(v >> (8 * i));
}
static void put64(uint8_t *b, size_t o, uint64_t v) {
  for (int i = 0; i < 8; ++i) b[o + i] = (uint8_t)(v >> (8 * i));
}
static void putf(uint8_t *b, size_t o, float v) {
  uint32_t u;
  memcpy(&u, &v, 4);
  put32(b, o, u);
}
static uint32_t get32(const uint8_t *b, size_t o) {
  uint32_t v = 0;
  for (int i = 0; i < 4; ++i) v |= (uint32_t)b[o + i] << (8 * i);
  return v;
}
static uint64_t get64(const uint8_t *b, size_t o) {
  uint64_t v = 0;
  for (int i = 0; i < 8; ++i) v |= (uint64_t)b[o + i] << (8 * i);
  return v;
}
static float getf(const uint8_t *b, size_t o) {
  uint32_t u = get32(b, o);
  float v;
  memcpy(&v, &u, 4);
  return v;
}
static uint64_t align256(uint64_t v) { return (v + 255) & ~(uint64_t)255; }

/* Words appended after the last chunk: zeros, so a reader may fetch a
 * little past the end of any chunk without leaving the section. */
static uint64_t padded_words_for(uint64_t total) { return (total + 1024 + 127) & ~(uint64_t)127; }

/* Alg. 1: scales (alpha * AbsMax, or the given ones), Q (base format fmt),
 * vec (row-major), ANS encode per chunk. */
static int container_build(const uint16_t *w, uint32_t M, uint32_t N, float alpha,
                           const uint16_t *given, uint32_t fmt, uint32_t P, uint32_t chunk_syms,
                           uint32_t lanes, uint64_t seed, float target_bits, uint8_t **blob_out,
                           uint64_t *blob_bytes) {
  if (!w || M == 0 || N == 0 || P < 8 || P > 12 || lanes == 0 || lanes % 64 != 0 ||
      chunk_syms == 0 || chunk_syms % lanes != 0 || (fmt != OR_FMT_E4M3 && fmt != OR_FMT_INT8))
    return OR_EINVAL;
  uint64_t n = (uint64_t)M * N;
  if (n >= (1ull << 32)) return OR_EINVAL;
  uint32_t n_chunks = (uint32_t)((n + chunk_syms - 1) / chunk_syms);
  uint16_t *scale = (uint16_t *)malloc(sizeof(uint16_t) * M);
  uint8_t *q = (uint8_t *)malloc((size_t)n);
  /* a chunk never needs more than one word per symbol */
  uint16_t *words = (uint16_t *)malloc(sizeof(uint16_t) * (size_t)n);
  uint32_t *chunk_off = (uint32_t *)malloc(sizeof(uint32_t) * ((size_t)n_chunks + 1));
  uint32_t *states = (uint32_t *)malloc(sizeof(uint32_t) * (size_t)n_chunks * lanes);
  int rc = OR_OK;
  if (!scale || !q || !words || !chunk_off || !states) {
    rc = OR_ENOMEM;
    goto done;
  }
  if (given) memcpy(scale, given, sizeof(uint16_t) * M);
  else or_row_scales(w, M, N, alpha, fmt, scale);
  or_quantize(w, M, N, scale, fmt, q);
  uint64_t counts[256] = {0};
  for (uint64_t k = 0; k < n; ++k) counts[q[k]]++;
  uint8_t sym[256];
  uint16_t freq[256];
  uint32_t K;
  rc = or_freq_table(counts, P, sym, freq, &K);
  if (rc != OR_OK) goto done;
  uint64_t total = 0;
  for (uint32_t c = 0; c < n_chunks; ++c) {
    uint64_t k0 = (uint64_t)c * chunk_syms;
    uint32_t nc = (uint32_t)((n - k0) < chunk_syms ? (n - k0) : chunk_syms);
    uint32_t nw = 0;
    chunk_off[c] = (uint32_t)total;
    rc = or_rans_encode(q + k0, nc, lanes, P, sym, freq, K, words + total,
                        (uint32_t)(n - total), &nw, states + (uint64_t)c * lanes);
    if (rc != OR_OK) goto done;
    total += nw;
  }
  chunk_off[n_chunks] = (uint32_t)total;

  uint64_t padded = padded_words_for(total);
  uint64_t o_scale = HEADER_BYTES;
  uint64_t o_sym = align256(o_scale + 2ull * M);
  uint64_t o_freq = align256(o_sym + K);
  uint64_t o_coff = align256(o_freq + 2ull * K);
  uint64_t o_cst = align256(o_coff + 4ull * (n_chunks + 1));
  uint64_t o_words = align256(o_cst + 4ull * n_chunks * lanes);
  uint64_t bytes = align256(o_words + 2ull * padded);
  uint8_t *b = (uint8_t *)calloc(1, bytes);
  if (!b) {
    rc = OR_ENOMEM;
    goto done;
  }
  memcpy(b + H_MAGIC, "EQC1", 4);
  put32(b, H_VERSION, 1);
  put32(b, H_HEADER_BYTES, HEADER_BYTES);
  put32(b, H_FORMAT, fmt);
  put32(b, H_ROWS, M);
  put32(b, H_COLS, N);
  put32(b, H_CHUNK, chunk_syms);
  put32(b, H_NCHUNKS, n_chunks);
  put32(b, H_LANES, lanes);
  put32(b, H_PBITS, P);
  put32(b, H_NSYMS, K);
  put32(b, H_FLAGS, 0);
  put64(b, H_TOTAL_WORDS, total);
  put64(b, H_PADDED_WORDS, padded);
  put64(b, H_SEED, seed);
  putf(b, H_ALPHA, given ? 0.0f : alpha);
  putf(b, H_TARGET, target_bits);
  putf(b, H_ENTROPY, (float)or_entropy_counts(counts, 256));
  put64(b, H_OFF_SCALE, o_scale);
  put64(b, H_OFF_SYM, o_sym);
  put64(b, H_OFF_FREQ, o_freq);
  put64(b, H_OFF_CHUNK_OFF, o_coff);
  put64(b, H_OFF_CHUNK_STATE, o_cst);
  put64(b, H_OFF_WORDS, o_words);
  put64(b, H_FILE_BYTES, bytes);
  for (uint32_t i = 0; i < M; ++i) {
    b[o_scale + 2ull * i] = (uint8_t)scale[i];
    b[o_scale + 2ull * i + 1] = (uint8_t)(scale[i] >> 8);
  }
  for (uint32_t k = 0; k < K; ++k) {
    b[o_sym + k] = sym[k];
    b[o_freq + 2ull * k] = (uint8_t)freq[k];
    b[o_freq + 2ull * k + 1] = (uint8_t)(freq[k] >> 8);
  }
  for (uint32_t c = 0; c <= n_chunks; ++c) put32(b, o_coff + 4ull * c, chunk_off[c]);
  for (uint64_t s = 0; s < (uint64_t)n_chunks * lanes; ++s) put32(b, o_cst + 4 * s, states[s]);
  for (uint64_t k = 0; k < total; ++k) {
    b[o_words + 2 * k] = (uint8_t)words[k];
    b[o_words + 2 * k + 1] = (uint8_t)(words[k] >> 8);
  }
  *blob_out = b;
  *blob_bytes = bytes;
done:
  free(scale);
  free(q);
  free(words);
  free(chunk_off);
  free(states);
  return rc;
}

int or_container_build(const uint16_t *w, uint32_t M, uint32_t N, float alpha, uint32_t fmt,
                       uint32_t P, uint32_t chunk_syms, uint32_t lanes, uint64_t seed,
                       float target_bits, uint8_t **blob_out, uint64_t *blob_bytes) {
  return container_build(w, M, N, alpha, NULL, fmt, P, chunk_syms, lanes, seed, target_bits,
                         blob_out, blob_bytes);
}

int or_container_build_scaled(const uint16_t *w, uint32_t M, uint32_t N, const uint16_t *scale,
                              uint32_t fmt, uint32_t P, uint32_t chunk_syms, uint32_t lanes,
                              uint64_t seed, float target_bits, uint8_t **blob_out,
                              uint64_t *blob_bytes) {
  if (!scale) return OR_EINVAL;
  return container_build(w, M, N, 0.0f, scale, fmt, P, chunk_syms, lanes, seed, target_bits,
                         blob_out, blob_bytes);
}

void or_free(void *p) { free(p); }

int or_container_info(const uint8_t *b, uint64_t bytes, or_info *h) {
  if (!b || bytes < HEADER_BYTES || memcmp(b, "EQC1", 4) != 0) return OR_EFORMAT;
  if (get32(b, H_VERSION) != 1 || get32(b, H_HEADER_BYTES) != HEADER_BYTES) return OR_EFORMAT;
  h->base_format = get32(b, H_FORMAT);
  h->rows = get32(b, H_ROWS);
  h->cols = get32(b, H_COLS);
  h->chunk_syms = get32(b, H_CHUNK);
  h->n_chunks = get32(b, H_NCHUNKS);
  h->lanes = get32(b, H_LANES);
  h->prob_bits = get32(b, H_PBITS);
  h->n_syms = get32(b, H_NSYMS);
  h->total_words = get64(b, H_TOTAL_WORDS);
  h->padded_words = get64(b, H_PADDED_WORDS);
  h->seed = get64(b, H_SEED);
  h->alpha = getf(b, H_ALPHA);
  h->target_bits = getf(b, H_TARGET);
  h->entropy_bits = getf(b, H_ENTROPY);
  h->off_scale = get64(b, H_OFF_SCALE);
  h->off_sym = get64(b, H_OFF_SYM);
  h->off_freq = get64(b, H_OFF_FREQ);
  h->off_chunk_off = get64(b, H_OFF_CHUNK_OFF);
  h->off_chunk_state = get64(b, H_OFF_CHUNK_STATE);
  h->off_words = get64(b, H_OFF_WORDS);
  h->file_bytes = get64(b, H_FILE_BYTES);
  uint64_t n = (uint64_t)h->rows * h->cols;
  if ((h->base_format != OR_FMT_E4M3 && h->base_format != OR_FMT_INT8) || n == 0 || n >= (1ull << 32) || h->lanes == 0 ||
      h->lanes % 64 != 0 || h->chunk_syms == 0 || h->chunk_syms % h->lanes != 0 ||
      h->prob_bits < 8 || h->prob_bits > 12 || h->n_syms < 1 || h->n_syms > 256 ||
      h->n_chunks != (n + h->chunk_syms - 1) / h->chunk_syms ||
      h->padded_words < h->total_words || h->file_bytes > bytes)
    return OR_EFORMAT;
  if (h->off_scale + 2ull * h->rows > h->file_bytes ||
      h->off_sym + h->n_syms > h->file_bytes ||
      h->off_freq + 2ull * h->n_syms > h->file_bytes ||
      h->off_chunk_off + 4ull * (h->n_chunks + 1) > h->file_bytes ||
      h->off_chunk_state + 4ull * h->n_chunks * h->lanes > h->file_bytes ||
      h->off_words + 2ull * h->padded_words > h->file_bytes)
    return OR_EFORMAT;
  return OR_OK;
}

/* Alg. 2, entropy decoding for one chunk. */
int or_container_decode_chunk(const uint8_t *b, uint64_t bytes, uint32_t c, uint8_t *q) {
  or_info h;
  int rc = or_container_info(b, bytes, &h);
  if (rc != OR_OK) return rc;
  if (c >= h.n_chunks) return OR_EINVAL;
  uint8_t sym[256];
  uint16_t freq[256];
  for (uint32_t k = 0; k < h.n_syms; ++k) {
    sym[k] = b[h.off_sym + k];
    freq[k] = (uint16_t)(b[h.off_freq + 2 * k] | (b[h.off_freq + 2 * k + 1] << 8));
  }
  uint32_t w0 = get32(b, h.off_chunk_off + 4ull * c);
  uint32_t w1 = get32(b, h.off_chunk_off + 4ull * (c + 1));
  if (w1 < w0 || w1 > h.total_words) return OR_EFORMAT;
  uint64_t n = (uint64_t)h.rows * h.cols;
  uint64_t k0 = (uint64_t)c * h.chunk_syms;
  uint32_t nc = (uint32_t)((n - k0) < h.chunk_syms ? (n - k0) : h.chunk_syms);
  uint32_t *states = (uint32_t *)malloc(sizeof(uint32_t) * h.lanes);
  uint16_t *words = (uint16_t *)malloc(sizeof(uint16_t) * ((size_t)(w1 - w0) + 1));
  if (!states || !words) {
    free(states);
    free(words);
    return OR_ENOMEM;
  }
  for (uint32_t l = 0; l < h.lanes; ++l)
    states[l] = get32(b, h.off_chunk_state + 4ull * ((uint64_t)c * h.lanes + l));
  for (uint32_t k = 0; k < w1 - w0; ++k) {
    uint64_t o = h.off_words + 2ull * (w0 + k);
    words[k] = (uint16_t)(b[o] | (b[o + 1] << 8));
  }
  rc = or_rans_decode(words, w1 - w0, states, nc, h.lanes, h.prob_bits, sym, freq, h.n_syms, q);
  free(states);
  free(words);
  return rc;
}

int or_container_decode(const uint8_t *b, uint64_t bytes, uint8_t *q) {
  or_info h;
  int rc = or_container_info(b, bytes, &h);
  if (rc != OR_OK) return rc;
  int worst = OR_OK;
  for (uint32_t c = 0; c < h.n_chunks; ++c) {
    rc = or_container_decode_chunk(b, bytes, c, q + (uint64_t)c * h.chunk_syms);
    if (rc != OR_OK && worst == OR_OK) worst = rc;
  }
  return worst;
}

/* ------------------------------------------------------------------ */
/* Scale optimisation, Sec. 2.2 eq. optimization (Alg. 1)                */
/* ------------------------------------------------------------------ */

static double sign_of(double v) { return v > 0.0 ? 1.0 : (v < 0.0 ? -1.0 : 0.0); }

/* d(W, W_hat) = ||W - W_hat||_1 / ||W||_1 (relative entry-wise l1 loss) plus
 * lambda R(W_q) with R the entry-wise l1 norm of the quantised values per
 * entry.  W_hat = s_i * W_q with s_i unrounded.  Straight-through estimator
 * for the rounding of Q: d W_q / d s_i = -W / s_i^2 where |W/s_i| <= Qmax
 * (0 where the clamp acts), so d W_hat / d s_i = W_q + s_i d W_q / d s_i. */
double or_rd_objective(const uint16_t *w, uint32_t M, uint32_t N, uint32_t fmt, double lambda,
                       const double *s, double *grad, double *dist) {
  double wl1 = 0.0;
  for (uint64_t k = 0; k < (uint64_t)M * N; ++k) wl1 += fabs(or_bf16_value(w[k]));
  double qmax = or_qmax(fmt), dsum = 0.0, rsum = 0.0, mn = (double)M * (double)N;
  for (uint32_t i = 0; i < M; ++i) {
    double gd = 0.0, gr = 0.0;
    for (uint32_t j = 0; j < N; ++j) {
      double wv = or_bf16_value(w[(uint64_t)i * N + j]);
      float u = (float)wv / (float)s[i];
      double v = or_code_value(fmt, round_to_format(fmt, u));
      double diff = s[i] * v - wv;
      dsum += fabs(diff);
      rsum += fabs(v);
      double dv = (fabs((double)u) <= qmax) ? -wv / (s[i] * s[i]) : 0.0;
      gd += sign_of(diff) * (v + s[i] * dv);
      gr += sign_of(v) * dv;
    }
    if (grad) grad[i] = (wl1 > 0.0 ? gd / wl1 : 0.0) + lambda * gr / mn;
  }
  double d = wl1 > 0.0 ? dsum / wl1 : 0.0;
  if (dist) *dist = d;
  return d + lambda * rsum / mn;
}

static double vdot(const double *a, const double *b, uint32_t n) {
  double t = 0.0;
  for (uint32_t i = 0; i < n; ++i) t += a[i] * b[i];
  return t;
}

/* L-BFGS (Liu and Nocedal 1989), fixed step length lr.  Direction: the
 * two-loop recursion over the newest `history` pairs (s_k = x_{k+1} - x_k,
 * y_k = g_{k+1} - g_k, kept only if y_k.s_k > 1e-10) with initial matrix
 * (s.y / y.y) I from the newest pair; the first step is lr min(1, 1/|g|_1)
 * along -g.  Stops after `iters` steps, when |g|_inf <= 1e-12, or when f
 * changes by less than 1e-10; the iterate with the lowest f is returned. */
int or_lbfgs(uint32_t n, double *x, or_fg_fn fg, void *ctx, const double *lower, uint32_t iters,
             uint32_t history, double lr, double *f_out) {
  if (n == 0 || history == 0) return OR_EINVAL;
  double *g = malloc(sizeof(double) * n), *gn = malloc(sizeof(double) * n);
  double *xn = malloc(sizeof(double) * n), *q = malloc(sizeof(double) * n);
  double *best = malloc(sizeof(double) * n), *alpha = malloc(sizeof(double) * history);
  double *S = malloc(sizeof(double) * n * history), *Y = malloc(sizeof(double) * n * history);
  double *rho = malloc(sizeof(double) * history);
  int rc = OR_OK;
  if (!g || !gn || !xn || !q || !best || !alpha || !S || !Y || !rho) {
    rc = OR_ENOMEM;
    goto out;
  }
  double f = fg(x, g, ctx), fbest = f;
  memcpy(best, x, sizeof(double) * n);
  uint32_t k = 0; /* pairs stored, oldest first: pair a at S + a n */
  for (uint32_t it = 0; it < iters; ++it) {
    double ginf = 0.0, g1 = 0.0;
    for (uint32_t i = 0; i < n; ++i) {
      if (fabs(g[i]) > ginf) ginf = fabs(g[i]);
      g1 += fabs(g[i]);
    }
    if (ginf <= 1e-12) break;
    memcpy(q, g, sizeof(double) * n);
    for (uint32_t a = k; a-- > 0;) {
      alpha[a] = rho[a] * vdot(S + (uint64_t)a * n, q, n);
      for (uint32_t i = 0; i < n; ++i) q[i] -= alpha[a] * Y[(uint64_t)a * n + i];
    }
    double gamma = 1.0;
    if (k) {
      const double *sl = S + (uint64_t)(k - 1) * n, *yl = Y + (uint64_t)(k - 1) * n;
      gamma = vdot(sl, yl, n) / vdot(yl, yl, n);
    }
    for (uint32_t i = 0; i < n; ++i) q[i] *= gamma;
    for (uint32_t a = 0; a < k; ++a) {
      double beta = rho[a] * vdot(Y + (uint64_t)a * n, q, n);
      for (uint32_t i = 0; i < n; ++i) q[i] += S[(uint64_t)a * n + i] * (alpha[a] - beta);
    }
    double t = lr;
    if (it == 0) t = lr * (1.0 / g1 < 1.0 ? 1.0 / g1 : 1.0);
    for (uint32_t i = 0; i < n; ++i) {
      xn[i] = x[i] - t * q[i];
      if (lower && xn[i] < lower[i]) xn[i] = lower[i];
    }
    double fn = fg(xn, gn, ctx);
    /* curvature pair */
    double ys = 0.0;
    for (uint32_t i = 0; i < n; ++i) ys += (gn[i] - g[i]) * (xn[i] - x[i]);
    if (ys > 1e-10) {
      if (k == history) { /* drop the oldest */
        memmove(S, S + n, sizeof(double) * n * (history - 1));
        memmove(Y, Y + n, sizeof(double) * n * (history - 1));
        memmove(rho, rho + 1, sizeof(double) * (history - 1));
        --k;
      }
      for (uint32_t i = 0; i < n; ++i) {
        S[(uint64_t)k * n + i] = xn[i] - x[i];
        Y[(uint64_t)k * n + i] = gn[i] - g[i];
      }
      rho[k] = 1.0 / ys;
      ++k;
    }
    int flat = fabs(fn - f) < 1e-10;
    memcpy(x, xn, sizeof(double) * n);
    memcpy(g, gn, sizeof(double) * n);
    f = fn;
    if (f < fbest) {
      fbest = f;
      memcpy(best, x, sizeof(double) * n);
    }
    if (flat) break;
  }
  memcpy(x, best, sizeof(double) * n);
  if (f_out) *f_out = fbest;
out:
  free(g);
  free(gn);
  free(xn);
  free(q);
  free(best);
  free(alpha);
  free(S);
  free(Y);
  free(rho);
  return rc;
}

typedef struct {
  const uint16_t *w;
  uint32_t M, N, fmt;
  double lambda;
} rd_ctx;

static double rd_fg(const double *x, double *g, void *ctx) {
  const rd_ctx *c = (const rd_ctx *)ctx;
  return or_rd_objective(c->w, c->M, c->N, c->fmt, c->lambda, x, g, NULL);
}

int or_rd_scales(const uint16_t *w, uint32_t M, uint32_t N, uint32_t fmt, double lambda,
                 uint32_t iters, uint32_t history, double lr, double *s_out, double *f_out) {
  if (!w || !s_out || M == 0 || N == 0 || !(lambda >= 0.0)) return OR_EINVAL;
  double *lower = malloc(sizeof(double) * M);
  if (!lower) return OR_ENOMEM;
  for (uint32_t i = 0; i < M; ++i) { /* eq. absmax: max|W_i| / Qmax (zero rows: 1) */
    double amax = 0.0;
    for (uint32_t j = 0; j < N; ++j) {
      double a = fabs(or_bf16_value(w[(uint64_t)i * N + j]));
      if (a > amax) amax = a;
    }
    s_out[i] = amax > 0.0 ? amax / or_qmax(fmt) : 1.0;
    lower[i] = 1e-6 * s_out[i];
  }
  rd_ctx c = {w, M, N, fmt, lambda};
  int rc = or_lbfgs(M, s_out, rd_fg, &c, lower, iters, history, lr, f_out);
  free(lower);
  return rc;
}

typedef struct {
  uint32_t n;
  const double *a, *c;
  double b;
} quad_ctx;

static double quad_fg(const double *x, double *g, void *ctx) {
  const quad_ctx *q = (const quad_ctx *)ctx;
  double sum = 0.0, f = 0.0;
  for (uint32_t i = 0; i < q->n; ++i) sum += x[i] - q->c[i];
  for (uint32_t i = 0; i < q->n; ++i) {
    double d = x[i] - q->c[i];
    f += 0.5 * q->a[i] * d * d;
    g[i] = q->a[i] * d + q->b * sum;
  }
  return f + 0.5 * q->b * sum * sum;
}

int or_lbfgs_quadratic(uint32_t n, const double *a, double b, const double *c, uint32_t iters,
                       uint32_t history, double lr, double *x, double *f_out) {
  quad_ctx q = {n, a, c, b};
  return or_lbfgs(n, x, quad_fg, &q, NULL, iters, history, lr, f_out);
}

/* ------------------------------------------------------------------ */
/* Linear layer (Sec. 2.1): y = x W_hat^T + b, fp64 accumulation.       */
/* ------------------------------------------------------------------ */
void or_gemv(const uint16_t *w_hat, uint32_t M, uint32_t N, const uint16_t *x, uint32_t B,
             const uint16_t *bias, double *y) {
  for (uint32_t b = 0; b < B; ++b)
    for (uint32_t i = 0; i < M; ++i) {
      double acc = 0.0;
      for (uint32_t j = 0; j < N; ++j)
        acc += or_bf16_value(w_hat[(uint64_t)i * N + j]) * or_bf16_value(x[(uint64_t)b * N + j]);
      y[(uint64_t)b * M + i] = acc + (bias ? or_bf16_value(bias[i]) : 0.0);
    }
}
