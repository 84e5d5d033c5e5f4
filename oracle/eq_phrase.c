/*
 * EntQuant CPU oracle, container version 2 -- TEST INFRASTRUCTURE ONLY
 * (see eq_oracle.h: only the tests, the smoke check and the benchmark's CPU
 * baseline load this library).
 *
 * Version 2 entropy-codes the same quantised codes as version 1 (Alg. 1:
 * quantise, vec, ANS encode; Alg. 2: ANS decode, view) with two choices of
 * ours where the paper leaves the coder to a closed library (App. A.1):
 *
 * 1. Order of vec: the M x N code matrix is cut into tiles of TR rows by TC
 *    columns (the last tile row and column may be smaller); tile (b, t) is
 *    chunk c = b * NT + t, NT = ceil(N / TC), and row s of a tile is the
 *    segment of coder state s (W = TR states per chunk).  Inside a segment
 *    the codes are in column order.  So a chunk's states all walk the same
 *    TC columns, and a state's codes are adjacent in its row.
 *
 * 2. Alphabet: phrases of four, two or one codes.  A segment is parsed
 *    greedily from its start: at each position, the four codes starting
 *    there form one symbol if they are in the quad dictionary DQ, else the
 *    two codes starting there if they are in the pair dictionary DP, else
 *    the single code.  The ANS alphabet is DQ, then DP, then the single
 *    codes DS that the parse emits, each part in ascending order of its
 *    codes read as a little-endian integer.  A symbol's probability is its
 *    count among all symbols, normalised to multiples of 2^-R as in
 *    or_freq_table.
 *
 *    Dictionary rule (encoder side; the container stores the result): the
 *    quads are counted at positions 0, 4, 8, ... of every segment (the
 *    segment's full blocks) and the pairs at positions 0, 2, 4, ...; a pair
 *    enters DP if its count times 2^(R+2) is at least the number of pairs
 *    counted (a share of at least 2^-(R+2)), at most the 2^(R-2) most
 *    frequent (ties: lower value); a quad enters DQ if its count times
 *    2^(R+2) is at least tau times the number of blocks, at most the 2^(R-1)
 *    most frequent.  The encoder takes, among tau = 8, 4, 2, 1, the one whose
 *    alphabet codes the layer in the fewest bits, sum over symbols of
 *    count * log2(2^R / f) (in fp64, summed in alphabet order; ties: the
 *    larger tau).
 *
 * 3. Coder: interleaved rANS with the state arithmetic at M = 2^16 and
 *    frequencies F = f * 2^(16-R) (so a decoder can find the symbol of slot
 *    x mod 2^16 from its top R bits).  State in [2^16, 2^32), 16-bit words.
 *    Step t decodes the t-th symbol of every state that still has codes to
 *    produce (its segment is not complete), then those states, in ascending
 *    order, take the next word if x < 2^16.  States finish at different
 *    steps (segments hold different numbers of symbols).  After the last
 *    step every state is back at 2^16 and the words are used up.
 *
 * 4. Row order (optional, flag bit 0): the tiles of item 1 are cut over the
 *    rows taken in a stored order, row k of the stored matrix being matrix
 *    row order[k] (a permutation, kept in its own section; the scales stay
 *    in matrix order).  A state's segment is then a stretch of matrix row
 *    order[b TR + s].  Encoder rule: the rows by ascending number of
 *    phrases of their parse (item 2, summed over the row's segments), ties
 *    by lower row index.  The alphabet does not depend on the row order (its
 *    counts are sums over segments), so the container equals, section for
 *    section, the matrix-order container of the row-permuted codes, apart
 *    from the scales and the order section.  A tile lasts as long as its
 *    longest segment (the decoder's steps), so rows of like length in one
 *    tile shorten the tiles.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#include "eq_oracle.h"

#define V2_L 65536u

static void put32(uint8_t *b, size_t o, uint32_t v) {
  for (int i = 0; i < 4; ++i) b[o + i] = (uint8_t)(v >> (8 * i));
}
static void put64(uint8_t *b, size_t o, uint64_t v) {
  for (int i = 0; i < 8; ++i) b[o + i] = (uint8_t)(v >> (8 * i));
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
static uint64_t align256(uint64_t v) { return (v + 255) & ~(uint64_t)255; }

/* ------------------------------------------------------------------ */
/* Frequency normalisation: counts of n symbols to f_k >= 1 summing to 2^R */
/* ------------------------------------------------------------------ */

int or_freq_norm(const uint64_t *cnt, uint32_t n, uint32_t R, uint16_t *freq) {
  if (n == 0 || R < 1 || R > 16 || n > (1u << R)) return OR_EINVAL;
  uint64_t total = 0, M = 1ull << R;
  for (uint32_t k = 0; k < n; ++k) {
    if (cnt[k] == 0) return OR_EINVAL;
    total += cnt[k];
  }
  int64_t *f = (int64_t *)malloc(sizeof(int64_t) * n);
  uint64_t *rem = (uint64_t *)malloc(sizeof(uint64_t) * n);
  uint32_t *order = (uint32_t *)malloc(sizeof(uint32_t) * n);
  if (!f || !rem || !order) {
    free(f), free(rem), free(order);
    return OR_ENOMEM;
  }
  int64_t sum = 0;
  for (uint32_t k = 0; k < n; ++k) {
    uint64_t scaled = cnt[k] * M;
    f[k] = (int64_t)(scaled / total);
    rem[k] = scaled % total;
    if (f[k] < 1) f[k] = 1;
    sum += f[k];
  }
  int64_t d = (int64_t)M - sum;
  if (d > 0) { /* largest remainder first, ties by lower index, cycling */
    for (uint32_t k = 0; k < n; ++k) order[k] = k;
    for (uint32_t a = 1; a < n; ++a) {
      uint32_t v = order[a];
      int64_t b = (int64_t)a - 1;
      while (b >= 0 && rem[order[b]] < rem[v]) {
        order[b + 1] = order[b];
        --b;
      }
      order[b + 1] = v;
    }
    for (uint32_t i = 0; d > 0; i = (i + 1) % n, --d) f[order[i]] += 1;
  }
  while (d < 0) { /* take one from the largest f > 1, ties by lower index */
    uint32_t best = n;
    for (uint32_t k = 0; k < n; ++k)
      if (f[k] > 1 && (best == n || f[k] > f[best])) best = k;
    if (best == n) break;
    f[best] -= 1;
    ++d;
  }
  int rc = d == 0 ? OR_OK : OR_EINVAL;
  for (uint32_t k = 0; k < n; ++k) freq[k] = (uint16_t)(f[k] == 65536 ? 0 : f[k]);
  free(f), free(rem), free(order);
  return rc;
}

/* ------------------------------------------------------------------ */
/* Tiles                                                              */
/* ------------------------------------------------------------------ */

void or_tile_geometry(uint32_t M, uint32_t N, uint32_t TR, uint32_t TC, uint32_t c,
                      uint32_t *row0, uint32_t *col0, uint32_t *rows, uint32_t *cols) {
  uint32_t NT = (N + TC - 1) / TC;
  uint32_t b = c / NT, t = c % NT;
  *row0 = b * TR;
  *col0 = t * TC;
  *rows = (M - *row0) < TR ? (M - *row0) : TR;
  *cols = (N - *col0) < TC ? (N - *col0) : TC;
}

/* ------------------------------------------------------------------ */
/* Dictionary and parse                                               */
/* ------------------------------------------------------------------ */

static uint32_t quad_value(const uint8_t *u) {
  return (uint32_t)u[0] | (uint32_t)u[1] << 8 | (uint32_t)u[2] << 16 | (uint32_t)u[3] << 24;
}
static uint32_t pair_value(const uint8_t *u) { return (uint32_t)u[0] | (uint32_t)u[1] << 8; }

typedef struct {
  uint32_t value;
  uint64_t count;
} vc_t;

/* count desc, value asc */
static int by_count(const void *a, const void *b) {
  const vc_t *x = (const vc_t *)a, *y = (const vc_t *)b;
  if (x->count != y->count) return x->count > y->count ? -1 : 1;
  return x->value < y->value ? -1 : (x->value > y->value);
}
static int by_value(const void *a, const void *b) {
  const vc_t *x = (const vc_t *)a, *y = (const vc_t *)b;
  return x->value < y->value ? -1 : (x->value > y->value);
}
static int cmp_u32(const void *a, const void *b) {
  uint32_t x = *(const uint32_t *)a, y = *(const uint32_t *)b;
  return x < y ? -1 : (x > y);
}

/* Distinct values of v[0..n) with their counts (sorted by value). */
static vc_t *histogram(uint32_t *v, uint64_t n, uint64_t *n_out) {
  qsort(v, n, sizeof(uint32_t), cmp_u32);
  vc_t *h = (vc_t *)malloc(sizeof(vc_t) * (n ? n : 1));
  if (!h) return NULL;
  uint64_t k = 0;
  for (uint64_t i = 0; i < n; ++i) {
    if (k && h[k - 1].value == v[i]) h[k - 1].count++;
    else {
      h[k].value = v[i];
      h[k].count = 1;
      ++k;
    }
  }
  *n_out = k;
  return h;
}

static int in_sorted(const uint32_t *s, uint32_t n, uint32_t v) {
  uint32_t lo = 0, hi = n;
  while (lo < hi) {
    uint32_t mid = (lo + hi) / 2;
    if (s[mid] < v) lo = mid + 1;
    else hi = mid;
  }
  return lo < n && s[lo] == v;
}

/* Entries passing the share rule count * 2^(R+2) >= tau * units, at most cap
 * of them by (count desc, value asc); returned sorted by value. */
static uint32_t select_dict(vc_t *h, uint64_t nh, uint64_t units, uint32_t R, uint32_t tau,
                            uint32_t cap, uint32_t *out) {
  qsort(h, nh, sizeof(vc_t), by_count);
  uint32_t k = 0;
  for (uint64_t i = 0; i < nh && k < cap; ++i)
    if ((h[i].count << (R + 2)) >= (uint64_t)tau * units) out[k++] = h[i].value;
  qsort(out, k, sizeof(uint32_t), cmp_u32);
  return k;
}

/* The codes of the segment of tile row `row`, starting at column col0. */
static const uint8_t *segment(const uint8_t *q, uint32_t N, uint32_t row, uint32_t col0) {
  return q + (uint64_t)row * N + col0;
}

/* Counted units: quads at positions 0, 4, ... (step 4, width 4) or pairs at
 * 0, 2, ... (step 2, width 2) of every segment. */
static vc_t *unit_histogram(const uint8_t *q, uint32_t M, uint32_t N, uint32_t TC,
                            uint32_t width, uint64_t *units, uint64_t *nh) {
  uint32_t NT = (N + TC - 1) / TC;
  uint64_t n = 0;
  for (uint32_t t = 0; t < NT; ++t) {
    uint32_t w = (N - t * TC) < TC ? (N - t * TC) : TC;
    n += (uint64_t)M * (w / width);
  }
  uint32_t *v = (uint32_t *)malloc(sizeof(uint32_t) * (n ? n : 1));
  if (!v) return NULL;
  uint64_t k = 0;
  for (uint32_t r = 0; r < M; ++r)
    for (uint32_t t = 0; t < NT; ++t) {
      uint32_t w = (N - t * TC) < TC ? (N - t * TC) : TC;
      const uint8_t *u = segment(q, N, r, t * TC);
      for (uint32_t j = 0; j + width <= w; j += width)
        v[k++] = width == 4 ? quad_value(u + j) : pair_value(u + j);
    }
  vc_t *h = histogram(v, n, nh);
  free(v);
  *units = n;
  return h;
}

int or_phrase_dict(const uint8_t *q, uint32_t M, uint32_t N, uint32_t TR, uint32_t TC,
                   uint32_t R, uint32_t tau, uint32_t *quads, uint32_t *n_quads, uint32_t *pairs,
                   uint32_t *n_pairs) {
  if (!q || M == 0 || N == 0 || TR == 0 || TC == 0 || TC % 4 || R < 10 || R > 12 || tau == 0)
    return OR_EINVAL;
  uint64_t units, nh;
  vc_t *h = unit_histogram(q, M, N, TC, 4, &units, &nh);
  if (!h) return OR_ENOMEM;
  *n_quads = select_dict(h, nh, units, R, tau, 1u << (R - 1), quads);
  free(h);
  h = unit_histogram(q, M, N, TC, 2, &units, &nh);
  if (!h) return OR_ENOMEM;
  *n_pairs = select_dict(h, nh, units, R, 1, 1u << (R - 2), pairs);
  free(h);
  return OR_OK;
}

/* Phrase index of a symbol: quads 0..nq-1, pairs nq.., singles nq+np.. */
typedef struct {
  const uint32_t *quads, *pairs;
  uint32_t nq, np;
  uint8_t single_present[256];
  uint32_t single_index[256];
} dict_t;

static int find_sorted(const uint32_t *s, uint32_t n, uint32_t v) {
  uint32_t lo = 0, hi = n;
  while (lo < hi) {
    uint32_t mid = (lo + hi) / 2;
    if (s[mid] < v) lo = mid + 1;
    else hi = mid;
  }
  return (lo < n && s[lo] == v) ? (int)lo : -1;
}

/* Greedy parse of one segment u[0..w) into symbol indices (at most w of
 * them); returns the count, or -1 if a code that must be emitted alone is
 * not in the dictionary. */
static int64_t parse_segment(const dict_t *d, const uint8_t *u, uint32_t w, uint32_t *out) {
  int64_t n = 0;
  uint32_t j = 0;
  while (j < w) {
    if (j + 4 <= w) {
      int iq = find_sorted(d->quads, d->nq, quad_value(u + j));
      if (iq >= 0) {
        out[n++] = (uint32_t)iq;
        j += 4;
        continue;
      }
    }
    if (j + 2 <= w) {
      int ip = find_sorted(d->pairs, d->np, pair_value(u + j));
      if (ip >= 0) {
        out[n++] = d->nq + (uint32_t)ip;
        j += 2;
        continue;
      }
    }
    if (!d->single_present[u[j]]) return -1;
    out[n++] = d->nq + d->np + d->single_index[u[j]];
    j += 1;
  }
  return n;
}

int or_phrase_parse(const uint8_t *u, uint32_t w, const uint32_t *quads, uint32_t nq,
                    const uint32_t *pairs, uint32_t np, const uint8_t *singles, uint32_t ns,
                    uint32_t *out, uint32_t *n_out) {
  dict_t d;
  memset(&d, 0, sizeof d);
  d.quads = quads, d.pairs = pairs, d.nq = nq, d.np = np;
  for (uint32_t k = 0; k < ns; ++k) {
    d.single_present[singles[k]] = 1;
    d.single_index[singles[k]] = k;
  }
  int64_t n = parse_segment(&d, u, w, out);
  if (n < 0) return OR_EINVAL;
  *n_out = (uint32_t)n;
  return OR_OK;
}

/* The alphabet for one tau: dictionaries, the parse of every segment
 * (tok, with tok_off / tok_len per chunk and state), singles, counts and
 * normalised frequencies. */
typedef struct {
  uint32_t *quads, *pairs, nq, np, ns, n_sym;
  uint8_t singles[256];
  uint64_t *cnt;
  uint16_t *freq;
  double bits;
} alphabet_t;

static void alphabet_free(alphabet_t *a) {
  free(a->quads), free(a->pairs), free(a->cnt), free(a->freq);
  memset(a, 0, sizeof *a);
}

static int build_alphabet(const uint8_t *q, uint32_t M, uint32_t N, uint32_t TR, uint32_t TC,
                          uint32_t R, uint32_t tau, uint32_t n_chunks, uint32_t *tok,
                          uint64_t *tok_off, uint32_t *tok_len, alphabet_t *a) {
  memset(a, 0, sizeof *a);
  a->quads = (uint32_t *)malloc(sizeof(uint32_t) << (R - 1));
  a->pairs = (uint32_t *)malloc(sizeof(uint32_t) << (R - 2));
  if (!a->quads || !a->pairs) return OR_ENOMEM;
  int rc = or_phrase_dict(q, M, N, TR, TC, R, tau, a->quads, &a->nq, a->pairs, &a->np);
  if (rc != OR_OK) return rc;
  /* parse with every code allowed alone, then keep the codes that occur */
  dict_t d;
  memset(&d, 0, sizeof d);
  d.quads = a->quads, d.pairs = a->pairs, d.nq = a->nq, d.np = a->np;
  for (uint32_t c = 0; c < 256; ++c) d.single_present[c] = 1, d.single_index[c] = c;
  uint64_t used = 0;
  for (uint32_t c = 0; c < n_chunks; ++c) {
    uint32_t r0, c0, rows, cols;
    or_tile_geometry(M, N, TR, TC, c, &r0, &c0, &rows, &cols);
    for (uint32_t s = 0; s < TR; ++s) {
      uint64_t idx = (uint64_t)c * TR + s;
      tok_off[idx] = used;
      tok_len[idx] = 0;
      if (s >= rows) continue;
      int64_t k = parse_segment(&d, segment(q, N, r0 + s, c0), cols, tok + used);
      if (k < 0) return OR_EINVAL;
      tok_len[idx] = (uint32_t)k;
      used += (uint64_t)k;
    }
  }
  /* Keep the quads, pairs and single codes that the parse emits (a
   * dictionary entry counted at block positions may never be matched where
   * the parse stands; dropping it changes no decision of the parse). */
  uint32_t base = a->nq + a->np, all = base + 256;
  uint64_t *seen = (uint64_t *)calloc(all, sizeof(uint64_t));
  uint32_t *map = (uint32_t *)malloc(sizeof(uint32_t) * all);
  if (!seen || !map) {
    free(seen), free(map);
    return OR_ENOMEM;
  }
  for (uint64_t i = 0; i < used; ++i) seen[tok[i]]++;
  uint32_t k = 0, nq = 0, np = 0;
  for (uint32_t i = 0; i < a->nq; ++i)
    if (seen[i]) map[i] = k++, a->quads[nq++] = a->quads[i];
  for (uint32_t i = 0; i < a->np; ++i)
    if (seen[a->nq + i]) map[a->nq + i] = k++, a->pairs[np++] = a->pairs[i];
  a->ns = 0;
  for (uint32_t c = 0; c < 256; ++c)
    if (seen[base + c]) map[base + c] = k++, a->singles[a->ns++] = (uint8_t)c;
  a->nq = nq, a->np = np, a->n_sym = k;
  if (a->n_sym > (1u << R)) {
    free(seen), free(map);
    return OR_EINVAL;
  }
  a->cnt = (uint64_t *)calloc(a->n_sym, sizeof(uint64_t));
  a->freq = (uint16_t *)malloc(sizeof(uint16_t) * a->n_sym);
  if (!a->cnt || !a->freq) {
    free(seen), free(map);
    return OR_ENOMEM;
  }
  for (uint64_t i = 0; i < used; ++i) {
    tok[i] = map[tok[i]];
    a->cnt[tok[i]]++;
  }
  free(seen), free(map);
  rc = or_freq_norm(a->cnt, a->n_sym, R, a->freq);
  if (rc != OR_OK) return rc;
  a->bits = 0.0;
  for (uint32_t k = 0; k < a->n_sym; ++k)
    a->bits += (double)a->cnt[k] * log2((double)(1u << R) / (double)a->freq[k]);
  return OR_OK;
}

/* ------------------------------------------------------------------ */
/* rANS at M = 2^16 over one chunk's states                           */
/* ------------------------------------------------------------------ */

/* tok[s][0..len[s]) are the symbols of state s (stored at tok + off[s]).
 * F_k = freq_k << (16 - R); a stored frequency 0 stands for 2^R. */
int or_prans_encode(const uint32_t *tok, const uint64_t *off, const uint32_t *len, uint32_t W,
                    const uint16_t *freq, uint32_t n_sym, uint32_t R, uint16_t *words,
                    uint64_t max_words, uint64_t *n_words, uint32_t *states) {
  if (W == 0 || R < 1 || R > 16 || n_sym == 0) return OR_EINVAL;
  uint64_t *F = (uint64_t *)malloc(sizeof(uint64_t) * n_sym);
  uint64_t *CUM = (uint64_t *)malloc(sizeof(uint64_t) * n_sym);
  uint64_t *x = (uint64_t *)malloc(sizeof(uint64_t) * W);
  if (!F || !CUM || !x) {
    free(F), free(CUM), free(x);
    return OR_ENOMEM;
  }
  uint64_t acc = 0;
  for (uint32_t k = 0; k < n_sym; ++k) {
    uint64_t f = freq[k] ? freq[k] : (1ull << R);
    F[k] = f << (16 - R);
    CUM[k] = acc;
    acc += F[k];
  }
  int rc = OR_OK;
  if (acc != 65536) rc = OR_EINVAL;
  uint32_t T = 0;
  for (uint32_t s = 0; s < W; ++s) {
    x[s] = V2_L;
    if (len[s] > T) T = len[s];
  }
  uint64_t pushed = 0;
  for (uint32_t t = T; rc == OR_OK && t-- > 0;)
    for (uint32_t s = W; s-- > 0;) {
      if (t >= len[s]) continue;
      uint32_t k = tok[off[s] + t];
      if (k >= n_sym) {
        rc = OR_EINVAL;
        break;
      }
      if (x[s] >= (F[k] << 16)) {
        if (pushed >= max_words) {
          rc = OR_ENOMEM;
          break;
        }
        words[pushed++] = (uint16_t)(x[s] & 0xFFFF);
        x[s] >>= 16;
      }
      x[s] = (x[s] / F[k]) * 65536 + (x[s] % F[k]) + CUM[k];
    }
  if (rc == OR_OK) {
    for (uint64_t a = 0, b = pushed; a + 1 < b; ++a, --b) {
      uint16_t tmp = words[a];
      words[a] = words[b - 1];
      words[b - 1] = tmp;
    }
    for (uint32_t s = 0; s < W; ++s) states[s] = (uint32_t)x[s];
    *n_words = pushed;
  }
  free(F), free(CUM), free(x);
  return rc;
}

/* Decode: state s produces symbols until the lengths of its phrases reach
 * need[s] codes; plen[k] is the number of codes of symbol k.  Symbols go to
 * tok + off[s] (at most need[s] of them), their count to *got. */
int or_prans_decode(const uint16_t *words, uint64_t n_words, const uint32_t *states,
                    const uint32_t *need, uint32_t W, const uint16_t *freq, const uint8_t *plen,
                    uint32_t n_sym, uint32_t R, uint32_t *tok, const uint64_t *off,
                    uint32_t *got) {
  if (W == 0 || R < 1 || R > 16 || n_sym == 0) return OR_EINVAL;
  uint64_t *F = (uint64_t *)malloc(sizeof(uint64_t) * n_sym);
  uint64_t *CUM = (uint64_t *)malloc(sizeof(uint64_t) * (n_sym + 1));
  uint64_t *x = (uint64_t *)malloc(sizeof(uint64_t) * W);
  uint32_t *pos = (uint32_t *)calloc(W, sizeof(uint32_t));
  uint8_t *act = (uint8_t *)malloc(W);
  if (!F || !CUM || !x || !pos || !act) {
    free(F), free(CUM), free(x), free(pos), free(act);
    return OR_ENOMEM;
  }
  CUM[0] = 0;
  for (uint32_t k = 0; k < n_sym; ++k) {
    uint64_t f = freq[k] ? freq[k] : (1ull << R);
    F[k] = f << (16 - R);
    CUM[k + 1] = CUM[k] + F[k];
  }
  int rc = CUM[n_sym] == 65536 ? OR_OK : OR_EINVAL;
  for (uint32_t s = 0; s < W; ++s) {
    x[s] = states[s];
    got[s] = 0;
  }
  uint64_t p = 0;
  for (;;) {
    int any = 0;
    for (uint32_t s = 0; s < W; ++s) {
      act[s] = pos[s] < need[s];
      any |= act[s];
    }
    if (!any || rc != OR_OK) break;
    for (uint32_t s = 0; s < W; ++s) {
      if (!act[s]) continue;
      uint64_t slot = x[s] & 0xFFFF;
      uint32_t k = 0; /* the symbol whose interval [CUM_k, CUM_k + F_k) holds slot */
      while (CUM[k + 1] <= slot) ++k;
      x[s] = F[k] * (x[s] >> 16) + slot - CUM[k];
      tok[off[s] + got[s]] = k;
      got[s] += 1;
      pos[s] += plen[k];
    }
    for (uint32_t s = 0; s < W; ++s) {
      if (!act[s] || x[s] >= V2_L) continue;
      uint16_t wv = 0;
      if (p < n_words) wv = words[p];
      else rc = OR_ECORRUPT;
      ++p;
      x[s] = (x[s] << 16) | wv;
    }
  }
  for (uint32_t s = 0; s < W; ++s)
    if (x[s] != V2_L || pos[s] != need[s]) rc = (rc == OR_OK ? OR_ECORRUPT : rc);
  if (p != n_words && rc == OR_OK) rc = OR_ECORRUPT;
  free(F), free(CUM), free(x), free(pos), free(act);
  return rc;
}

/* ------------------------------------------------------------------ */
/* Container version 2                                                */
/* ------------------------------------------------------------------ */
enum {
  H_MAGIC = 0, H_VERSION = 4, H_HEADER_BYTES = 8, H_FORMAT = 12, H_ROWS = 16, H_COLS = 20,
  H_CHUNK = 24, H_NCHUNKS = 28, H_LANES = 32, H_PBITS = 36, H_NSYMS = 40, H_FLAGS = 44,
  H_TOTAL_WORDS = 48, H_PADDED_WORDS = 56, H_SEED = 64, H_ALPHA = 72, H_TARGET = 76,
  H_ENTROPY = 80, H_TILE_COLS = 84, H_OFF_SCALE = 88, H_OFF_PHR = 96, H_OFF_FREQ = 104,
  H_OFF_CHUNK_OFF = 112, H_OFF_CHUNK_STATE = 120, H_OFF_WORDS = 128, H_FILE_BYTES = 136,
  H_NQUAD = 144, H_NPAIR = 148, H_NSINGLE = 152, H_TAU = 156, H_OFF_ORDER = 160,
  HEADER_BYTES = 256
};
enum { FLAG_ROW_ORDER = 1u };

static uint64_t padded_words_for(uint64_t total) { return (total + 1024 + 127) & ~(uint64_t)127; }

/* rows by ascending phrase count, ties by lower row index (item 4) */
typedef struct {
  uint64_t cost;
  uint32_t row;
} row_cost_t;
static int row_cost_cmp(const void *pa, const void *pb) {
  const row_cost_t *a = (const row_cost_t *)pa, *b = (const row_cost_t *)pb;
  if (a->cost != b->cost) return a->cost < b->cost ? -1 : 1;
  return a->row < b->row ? -1 : (a->row > b->row);
}

int or_container2_build(const uint16_t *w, uint32_t M, uint32_t N, float alpha,
                        const uint16_t *given_scale, uint32_t fmt, uint32_t R, uint32_t TR,
                        uint32_t TC, uint32_t row_order, uint64_t seed, float target_bits,
                        uint8_t **blob_out, uint64_t *blob_bytes) {
  if (!w || M == 0 || N == 0 || R < 10 || R > 12 || (TR != 64 && TR != 128 && TR != 256) ||
      TC == 0 || TC % 4 || (fmt != OR_FMT_E4M3 && fmt != OR_FMT_INT8) || row_order > 1)
    return OR_EINVAL;
  uint64_t n = (uint64_t)M * N;
  if (n >= (1ull << 32) || (uint64_t)TR * TC >= (1ull << 32)) return OR_EINVAL;
  uint32_t NT = (N + TC - 1) / TC, NB = (M + TR - 1) / TR;
  uint64_t n_chunks64 = (uint64_t)NT * NB;
  if (n_chunks64 >= (1ull << 32)) return OR_EINVAL;
  uint32_t n_chunks = (uint32_t)n_chunks64;
  uint16_t *scale = (uint16_t *)malloc(sizeof(uint16_t) * M);
  uint8_t *q = (uint8_t *)malloc((size_t)n);
  uint32_t *tok = (uint32_t *)malloc(sizeof(uint32_t) * (size_t)n);  /* all symbols, by chunk */
  uint64_t *tok_off = (uint64_t *)malloc(sizeof(uint64_t) * (size_t)n_chunks * TR);
  uint32_t *tok_len = (uint32_t *)malloc(sizeof(uint32_t) * (size_t)n_chunks * TR);
  uint16_t *words = (uint16_t *)malloc(sizeof(uint16_t) * ((size_t)n + 16));
  uint32_t *chunk_off = (uint32_t *)malloc(sizeof(uint32_t) * ((size_t)n_chunks + 1));
  uint32_t *states = (uint32_t *)malloc(sizeof(uint32_t) * (size_t)n_chunks * TR);
  uint32_t *order = NULL;
  uint8_t *qs = NULL;
  row_cost_t *rc_rows = NULL;
  alphabet_t best, cur;
  memset(&best, 0, sizeof best);
  memset(&cur, 0, sizeof cur);
  uint32_t best_tau = 0;
  int rc = OR_OK;
  if (!scale || !q || !tok || !tok_off || !tok_len || !words || !chunk_off || !states) {
    rc = OR_ENOMEM;
    goto done;
  }
  if (given_scale) memcpy(scale, given_scale, sizeof(uint16_t) * M);
  else or_row_scales(w, M, N, alpha, fmt, scale);
  or_quantize(w, M, N, scale, fmt, q);
  /* the alphabet that codes the layer in the fewest bits (ties: larger tau) */
  for (uint32_t tau = 8; tau >= 1; tau /= 2) {
    rc = build_alphabet(q, M, N, TR, TC, R, tau, n_chunks, tok, tok_off, tok_len, &cur);
    if (rc != OR_OK) goto done;
    if (best_tau == 0 || cur.bits < best.bits) {
      alphabet_free(&best);
      best = cur;
      best_tau = tau;
      memset(&cur, 0, sizeof cur);
    } else {
      alphabet_free(&cur);
    }
  }
  /* the parse of the chosen alphabet */
  if (best_tau != 1) {
    alphabet_free(&cur);
    rc = build_alphabet(q, M, N, TR, TC, R, best_tau, n_chunks, tok, tok_off, tok_len, &cur);
    if (rc != OR_OK) goto done;
    alphabet_free(&cur);
  }
  if (row_order) {
    /* item 4: each row's phrase count over its segments, the rows sorted by
     * it, and the parse of the codes with their rows in that order (the
     * same alphabet: its counts do not depend on the order of the rows) */
    order = (uint32_t *)malloc(sizeof(uint32_t) * M);
    qs = (uint8_t *)malloc((size_t)n);
    rc_rows = (row_cost_t *)malloc(sizeof(row_cost_t) * M);
    if (!order || !qs || !rc_rows) {
      rc = OR_ENOMEM;
      goto done;
    }
    for (uint32_t i = 0; i < M; ++i) {
      uint64_t cost = 0;
      for (uint32_t t = 0; t < NT; ++t) cost += tok_len[((uint64_t)(i / TR) * NT + t) * TR + i % TR];
      rc_rows[i].cost = cost;
      rc_rows[i].row = i;
    }
    qsort(rc_rows, M, sizeof(row_cost_t), row_cost_cmp);
    for (uint32_t k = 0; k < M; ++k) {
      order[k] = rc_rows[k].row;
      memcpy(qs + (uint64_t)k * N, q + (uint64_t)order[k] * N, N);
    }
    rc = build_alphabet(qs, M, N, TR, TC, R, best_tau, n_chunks, tok, tok_off, tok_len, &cur);
    if (rc != OR_OK) goto done;
    int same = cur.n_sym == best.n_sym && cur.nq == best.nq && cur.np == best.np &&
               cur.ns == best.ns;
    for (uint32_t k = 0; same && k < best.n_sym; ++k) same = cur.freq[k] == best.freq[k];
    alphabet_free(&cur);
    if (!same) {
      rc = OR_EINVAL;
      goto done;
    }
  }
  uint32_t nq = best.nq, np = best.np, ns = best.ns, n_sym = best.n_sym;
  uint64_t total = 0;
  for (uint32_t c = 0; c < n_chunks; ++c) {
    uint64_t nw = 0;
    chunk_off[c] = (uint32_t)total;
    rc = or_prans_encode(tok, tok_off + (uint64_t)c * TR, tok_len + (uint64_t)c * TR, TR,
                         best.freq, n_sym, R, words + total, (uint64_t)n + 16 - total, &nw,
                         states + (uint64_t)c * TR);
    if (rc != OR_OK) goto done;
    total += nw;
    if (total >= (1ull << 32)) {
      rc = OR_EINVAL;
      goto done;
    }
  }
  chunk_off[n_chunks] = (uint32_t)total;

  uint64_t counts[256] = {0};
  for (uint64_t k = 0; k < n; ++k) counts[q[k]]++;
  uint64_t padded = padded_words_for(total);
  uint64_t o_scale = HEADER_BYTES;
  uint64_t o_phr = align256(o_scale + 2ull * M);
  uint64_t o_freq = align256(o_phr + 4ull * n_sym);
  uint64_t o_coff = align256(o_freq + 2ull * n_sym);
  uint64_t o_cst = align256(o_coff + 4ull * (n_chunks + 1));
  uint64_t o_order = row_order ? align256(o_cst + 4ull * n_chunks * TR) : 0;
  uint64_t o_words = row_order ? align256(o_order + 4ull * M) : align256(o_cst + 4ull * n_chunks * TR);
  uint64_t bytes = align256(o_words + 2ull * padded);
  uint8_t *b = (uint8_t *)calloc(1, bytes);
  if (!b) {
    rc = OR_ENOMEM;
    goto done;
  }
  memcpy(b + H_MAGIC, "EQC1", 4);
  put32(b, H_VERSION, 2);
  put32(b, H_HEADER_BYTES, HEADER_BYTES);
  put32(b, H_FORMAT, fmt);
  put32(b, H_ROWS, M);
  put32(b, H_COLS, N);
  put32(b, H_CHUNK, TR * TC);
  put32(b, H_NCHUNKS, n_chunks);
  put32(b, H_LANES, TR);
  put32(b, H_PBITS, R);
  put32(b, H_NSYMS, n_sym);
  put32(b, H_FLAGS, row_order ? FLAG_ROW_ORDER : 0);
  put64(b, H_TOTAL_WORDS, total);
  put64(b, H_PADDED_WORDS, padded);
  put64(b, H_SEED, seed);
  {
    float av = given_scale ? 0.0f : alpha, e = (float)or_entropy_counts(counts, 256);
    uint32_t u;
    memcpy(&u, &av, 4);
    put32(b, H_ALPHA, u);
    memcpy(&u, &target_bits, 4);
    put32(b, H_TARGET, u);
    memcpy(&u, &e, 4);
    put32(b, H_ENTROPY, u);
  }
  put32(b, H_TILE_COLS, TC);
  put64(b, H_OFF_SCALE, o_scale);
  put64(b, H_OFF_PHR, o_phr);
  put64(b, H_OFF_FREQ, o_freq);
  put64(b, H_OFF_CHUNK_OFF, o_coff);
  put64(b, H_OFF_CHUNK_STATE, o_cst);
  put64(b, H_OFF_WORDS, o_words);
  put64(b, H_FILE_BYTES, bytes);
  put32(b, H_NQUAD, nq);
  put32(b, H_NPAIR, np);
  put32(b, H_NSINGLE, ns);
  put32(b, H_TAU, best_tau);
  put64(b, H_OFF_ORDER, o_order);
  if (row_order)
    for (uint32_t k = 0; k < M; ++k) put32(b, o_order + 4ull * k, order[k]);
  for (uint32_t i = 0; i < M; ++i) {
    b[o_scale + 2ull * i] = (uint8_t)scale[i];
    b[o_scale + 2ull * i + 1] = (uint8_t)(scale[i] >> 8);
  }
  for (uint32_t k = 0; k < nq; ++k) put32(b, o_phr + 4ull * k, best.quads[k]);
  for (uint32_t k = 0; k < np; ++k) put32(b, o_phr + 4ull * (nq + k), best.pairs[k]);
  for (uint32_t k = 0; k < ns; ++k) b[o_phr + 4ull * (nq + np + k)] = best.singles[k];
  for (uint32_t k = 0; k < n_sym; ++k) {
    b[o_freq + 2ull * k] = (uint8_t)best.freq[k];
    b[o_freq + 2ull * k + 1] = (uint8_t)(best.freq[k] >> 8);
  }
  for (uint32_t c = 0; c <= n_chunks; ++c) put32(b, o_coff + 4ull * c, chunk_off[c]);
  for (uint64_t s = 0; s < (uint64_t)n_chunks * TR; ++s) put32(b, o_cst + 4 * s, states[s]);
  for (uint64_t k = 0; k < total; ++k) {
    b[o_words + 2 * k] = (uint8_t)words[k];
    b[o_words + 2 * k + 1] = (uint8_t)(words[k] >> 8);
  }
  *blob_out = b;
  *blob_bytes = bytes;
done:
  alphabet_free(&best);
  alphabet_free(&cur);
  free(scale), free(q), free(tok), free(tok_off), free(tok_len);
  free(words), free(chunk_off), free(states), free(order), free(qs), free(rc_rows);
  return rc;
}

int or_container2_info(const uint8_t *b, uint64_t bytes, or_info2 *h) {
  if (!b || bytes < HEADER_BYTES || memcmp(b, "EQC1", 4) != 0) return OR_EFORMAT;
  if (get32(b, H_VERSION) != 2 || get32(b, H_HEADER_BYTES) != HEADER_BYTES) return OR_EFORMAT;
  h->base_format = get32(b, H_FORMAT);
  h->rows = get32(b, H_ROWS);
  h->cols = get32(b, H_COLS);
  h->chunk_syms = get32(b, H_CHUNK);
  h->n_chunks = get32(b, H_NCHUNKS);
  h->lanes = get32(b, H_LANES);
  h->prob_bits = get32(b, H_PBITS);
  h->n_syms = get32(b, H_NSYMS);
  h->tile_cols = get32(b, H_TILE_COLS);
  h->n_quads = get32(b, H_NQUAD);
  h->n_pairs = get32(b, H_NPAIR);
  h->n_singles = get32(b, H_NSINGLE);
  h->tau = get32(b, H_TAU);
  h->total_words = get64(b, H_TOTAL_WORDS);
  h->padded_words = get64(b, H_PADDED_WORDS);
  h->seed = get64(b, H_SEED);
  uint32_t u;
  u = get32(b, H_ALPHA), memcpy(&h->alpha, &u, 4);
  u = get32(b, H_TARGET), memcpy(&h->target_bits, &u, 4);
  u = get32(b, H_ENTROPY), memcpy(&h->entropy_bits, &u, 4);
  h->off_scale = get64(b, H_OFF_SCALE);
  h->off_phr = get64(b, H_OFF_PHR);
  h->off_freq = get64(b, H_OFF_FREQ);
  h->off_chunk_off = get64(b, H_OFF_CHUNK_OFF);
  h->off_chunk_state = get64(b, H_OFF_CHUNK_STATE);
  h->off_words = get64(b, H_OFF_WORDS);
  h->file_bytes = get64(b, H_FILE_BYTES);
  h->flags = get32(b, H_FLAGS);
  h->off_order = get64(b, H_OFF_ORDER);
  uint64_t n = (uint64_t)h->rows * h->cols;
  uint32_t TR = h->lanes, TC = h->tile_cols;
  if ((h->base_format != OR_FMT_E4M3 && h->base_format != OR_FMT_INT8) || n == 0 ||
      n >= (1ull << 32) || (TR != 64 && TR != 128 && TR != 256) || TC == 0 || TC % 4 ||
      (uint64_t)TR * TC != h->chunk_syms || h->prob_bits < 10 || h->prob_bits > 12 ||
      h->n_syms < 1 || h->n_syms > (1u << h->prob_bits) ||
      (uint64_t)h->n_quads + h->n_pairs + h->n_singles != h->n_syms || h->n_singles > 256 ||
      h->n_chunks != (uint64_t)((h->rows + TR - 1) / TR) * ((h->cols + TC - 1) / TC) ||
      h->padded_words < h->total_words || h->file_bytes > bytes)
    return OR_EFORMAT;
  if (h->off_scale + 2ull * h->rows > h->file_bytes ||
      h->off_phr + 4ull * h->n_syms > h->file_bytes ||
      h->off_freq + 2ull * h->n_syms > h->file_bytes ||
      h->off_chunk_off + 4ull * (h->n_chunks + 1) > h->file_bytes ||
      h->off_chunk_state + 4ull * h->n_chunks * TR > h->file_bytes ||
      h->off_words + 2ull * h->padded_words > h->file_bytes)
    return OR_EFORMAT;
  /* item 4: the order section, a permutation of the rows */
  if (h->flags & ~(uint32_t)FLAG_ROW_ORDER) return OR_EFORMAT;
  if (!(h->flags & FLAG_ROW_ORDER)) return h->off_order == 0 ? OR_OK : OR_EFORMAT;
  if (h->off_order < HEADER_BYTES || h->off_order > h->file_bytes ||
      4ull * h->rows > h->file_bytes - h->off_order)
    return OR_EFORMAT;
  uint8_t *seen = (uint8_t *)calloc(h->rows, 1);
  if (!seen) return OR_ENOMEM;
  int rc = OR_OK;
  for (uint32_t k = 0; k < h->rows && rc == OR_OK; ++k) {
    uint32_t r = get32(b, h->off_order + 4ull * k);
    if (r >= h->rows || seen[r]) rc = OR_EFORMAT;
    else seen[r] = 1;
  }
  free(seen);
  return rc;
}

/* Matrix row of stored row k (item 4; the identity without a row order). */
uint32_t or_container2_row(const uint8_t *b, const or_info2 *h, uint32_t k) {
  return (h->flags & FLAG_ROW_ORDER) ? get32(b, h->off_order + 4ull * k) : k;
}

/* Alg. 2, entropy decoding for one chunk: the tile's codes, row-major (rows x cols of
 * the tile as or_tile_geometry gives them; tile row s is stored row r0 + s, which
 * or_container2_row maps to its matrix row). */
int or_container2_decode_chunk(const uint8_t *b, uint64_t bytes, uint32_t c, uint8_t *tile) {
  or_info2 h;
  int rc = or_container2_info(b, bytes, &h);
  if (rc != OR_OK) return rc;
  if (c >= h.n_chunks) return OR_EINVAL;
  uint32_t TR = h.lanes, TC = h.tile_cols, n_sym = h.n_syms;
  uint32_t r0, c0, rows, cols;
  or_tile_geometry(h.rows, h.cols, TR, TC, c, &r0, &c0, &rows, &cols);
  uint32_t w0 = get32(b, h.off_chunk_off + 4ull * c);
  uint32_t w1 = get32(b, h.off_chunk_off + 4ull * (c + 1));
  if (w1 < w0 || w1 > h.total_words) return OR_EFORMAT;
  uint16_t *freq = (uint16_t *)malloc(sizeof(uint16_t) * n_sym);
  uint8_t *plen = (uint8_t *)malloc(n_sym);
  uint32_t *states = (uint32_t *)malloc(sizeof(uint32_t) * TR);
  uint32_t *need = (uint32_t *)malloc(sizeof(uint32_t) * TR);
  uint32_t *got = (uint32_t *)malloc(sizeof(uint32_t) * TR);
  uint64_t *off = (uint64_t *)malloc(sizeof(uint64_t) * TR);
  uint32_t *tok = (uint32_t *)malloc(sizeof(uint32_t) * ((size_t)TR * TC + 1));
  uint16_t *words = (uint16_t *)malloc(sizeof(uint16_t) * ((size_t)(w1 - w0) + 1));
  if (!freq || !plen || !states || !need || !got || !off || !tok || !words) {
    rc = OR_ENOMEM;
    goto done;
  }
  for (uint32_t k = 0; k < n_sym; ++k) {
    freq[k] = (uint16_t)(b[h.off_freq + 2 * k] | (b[h.off_freq + 2 * k + 1] << 8));
    plen[k] = k < h.n_quads ? 4 : (k < h.n_quads + h.n_pairs ? 2 : 1);
  }
  for (uint32_t s = 0; s < TR; ++s) {
    states[s] = get32(b, h.off_chunk_state + 4ull * ((uint64_t)c * TR + s));
    need[s] = s < rows ? cols : 0;
    off[s] = (uint64_t)s * TC;
  }
  for (uint32_t k = 0; k < w1 - w0; ++k) {
    uint64_t o = h.off_words + 2ull * (w0 + k);
    words[k] = (uint16_t)(b[o] | (b[o + 1] << 8));
  }
  rc = or_prans_decode(words, w1 - w0, states, need, TR, freq, plen, n_sym, h.prob_bits, tok,
                       off, got);
  /* expand the phrases of each row (as far as they were decoded) */
  for (uint32_t s = 0; s < rows; ++s) {
    uint32_t j = 0;
    for (uint32_t i = 0; i < got[s] && j < cols; ++i) {
      uint32_t k = tok[off[s] + i];
      for (uint32_t e = 0; e < plen[k] && j < cols; ++e)
        tile[(uint64_t)s * cols + j++] = b[h.off_phr + 4ull * k + e];
    }
    for (; j < cols; ++j) tile[(uint64_t)s * cols + j] = 0;
  }
done:
  free(freq), free(plen), free(states), free(need), free(got), free(off), free(tok), free(words);
  return rc;
}

int or_container2_decode(const uint8_t *b, uint64_t bytes, uint8_t *q) {
  or_info2 h;
  int rc = or_container2_info(b, bytes, &h);
  if (rc != OR_OK) return rc;
  uint8_t *tile = (uint8_t *)malloc((size_t)h.lanes * h.tile_cols);
  if (!tile) return OR_ENOMEM;
  int worst = OR_OK;
  for (uint32_t c = 0; c < h.n_chunks; ++c) {
    uint32_t r0, c0, rows, cols;
    or_tile_geometry(h.rows, h.cols, h.lanes, h.tile_cols, c, &r0, &c0, &rows, &cols);
    rc = or_container2_decode_chunk(b, bytes, c, tile);
    if (rc != OR_OK && worst == OR_OK) worst = rc;
    for (uint32_t s = 0; s < rows; ++s)
      memcpy(q + (uint64_t)or_container2_row(b, &h, r0 + s) * h.cols + c0,
             tile + (uint64_t)s * cols, cols);
  }
  free(tile);
  return worst;
}
