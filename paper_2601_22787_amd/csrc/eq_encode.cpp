// Host encoder for the compressed-layer container (declared in eq_encode.h).
//
// Alg. 1 of the paper (Sec. 2.2): AbsMax-based per-row scales (eq. absmax,
// channel-wise as in Sec. 2.1), quantisation Q to the base format (Float8
// E4M3FN, or Int8 as in the ablation of Sec. 3.5), row-major vec, ANS entropy
// coding per chunk (App. A.1).  The coder is interleaved rANS
// with a 32-bit state in [2^16, 2^32), 16-bit stream words and W lanes per
// chunk; symbol k of a chunk is coded by lane k mod W at step k div W.
#include "eq_encode.h"

#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstdlib>
#include <cstring>
#include <thread>
#include <vector>

namespace {

constexpr uint32_t kStateLow = 1u << 16;  // lower end of the state interval
constexpr uint64_t kHeaderBytes = 256;

// Default worker count: one per hardware thread, at most 16.
unsigned worker_count(uint32_t requested) {
  if (requested) return requested;
  unsigned n = std::thread::hardware_concurrency();
  return n ? std::min(n, 16u) : 1;
}

// Run fn(i) for i in [0, n) on up to `threads` workers (dynamic schedule).
template <class Fn>
void parallel_for(uint64_t n, unsigned threads, Fn fn) {
  threads = static_cast<unsigned>(std::min<uint64_t>(threads, n));
  if (threads <= 1) {
    for (uint64_t i = 0; i < n; ++i) fn(i);
    return;
  }
  std::atomic<uint64_t> next{0};
  auto body = [&] {
    for (uint64_t i; (i = next.fetch_add(1)) < n;) fn(i);
  };
  std::vector<std::thread> pool;
  pool.reserve(threads - 1);
  for (unsigned t = 1; t < threads; ++t) pool.emplace_back(body);
  body();
  for (auto &t : pool) t.join();
}

inline float bf16_to_float(uint16_t b) {
  uint32_t u = static_cast<uint32_t>(b) << 16;
  float f;
  std::memcpy(&f, &u, 4);
  return f;
}

// Nearest BF16 of a double (ties to even): scale the binade to an integer
// significand of 8 bits and round it with the current (nearest-even) mode.
uint16_t double_to_bf16(double v) {
  if (v == 0.0) return std::signbit(v) ? 0x8000 : 0;
  int e;
  double m = std::frexp(v, &e);
  int shift = 8;
  if (e - 1 < -126) shift = 8 - (-126 - (e - 1));  // BF16 subnormal range
  double r = std::nearbyint(std::ldexp(m, shift));
  float f = static_cast<float>(std::ldexp(r, e - shift));
  uint32_t u;
  std::memcpy(&u, &f, 4);
  return static_cast<uint16_t>(u >> 16);
}

// E4M3FN code of v: clamp |v| to 448, round to nearest (ties to even) on the
// E4M3 grid, -0 -> +0.  Normal range: round the fp32 significand from 23 to
// 3 bits in place (a carry moves into the exponent); subnormal range
// (|v| < 2^-6): the grid is k * 2^-9, so round |v| * 2^9 to an integer.
uint8_t quantize_e4m3(float v) {
  float a = std::fabs(v);
  if (a > 448.0f) a = 448.0f;
  uint32_t mag;
  if (a < 0.015625f) {
    mag = static_cast<uint32_t>(std::nearbyint(a * 512.0f));  // exact scaling
  } else {
    uint32_t b;
    std::memcpy(&b, &a, 4);
    uint32_t r = (b + 0x7FFFFu + ((b >> 20) & 1u)) >> 20;  // exponent:8 | mantissa:3
    mag = r - ((127u - 7u) << 3);
  }
  if (mag == 0) return 0;
  return static_cast<uint8_t>(mag | (std::signbit(v) ? 0x80u : 0u));
}

// Int8 code of v: clamp to [-127, 127] (symmetric, so 0x80 never occurs),
// then the nearest integer with ties to even (the default rounding mode).
uint8_t quantize_int8(float v) {
  const float c = std::min(127.0f, std::max(-127.0f, v));
  return static_cast<uint8_t>(static_cast<int8_t>(std::nearbyint(c)));
}

constexpr uint32_t kFmtE4M3 = 1, kFmtInt8 = 2;

double qmax(uint32_t fmt) { return fmt == kFmtInt8 ? 127.0 : 448.0; }

uint16_t row_scale(const uint16_t *row, uint32_t N, float alpha, uint32_t fmt) {
  float amax = 0.0f;
  for (uint32_t j = 0; j < N; ++j) amax = std::max(amax, std::fabs(bf16_to_float(row[j])));
  if (amax == 0.0f) return 0x3F80;
  return double_to_bf16(static_cast<double>(alpha) * static_cast<double>(amax) / qmax(fmt));
}

// Quantise the listed rows; codes are written only if `codes` is non-null.
// Row i's scale is given[i] when `given` is non-null, else the AbsMax scale
// times alpha.
void quantize_rows(const uint16_t *w, uint32_t N, float alpha, uint32_t fmt,
                   const std::vector<uint32_t> &rows, unsigned threads, uint16_t *scale,
                   uint8_t *codes, uint64_t hist[256], const uint16_t *given = nullptr) {
  uint8_t (*const quantize)(float) = fmt == kFmtInt8 ? quantize_int8 : quantize_e4m3;
  const uint64_t n_rows = rows.size();
  const uint64_t per = 16;  // rows per task
  const uint64_t tasks = (n_rows + per - 1) / per;
  std::vector<std::vector<uint64_t>> part(tasks, std::vector<uint64_t>(256, 0));
  parallel_for(tasks, threads, [&](uint64_t t) {
    uint64_t *h = part[t].data();
    for (uint64_t r = t * per; r < std::min(n_rows, (t + 1) * per); ++r) {
      const uint32_t i = rows[r];
      const uint16_t *src = w + static_cast<uint64_t>(i) * N;
      uint16_t s = given ? given[i] : row_scale(src, N, alpha, fmt);
      if (scale) scale[i] = s;
      const float sf = bf16_to_float(s);
      uint8_t *dst = codes ? codes + static_cast<uint64_t>(i) * N : nullptr;
      for (uint32_t j = 0; j < N; ++j) {
        uint8_t q = quantize(bf16_to_float(src[j]) / sf);
        ++h[q];
        if (dst) dst[j] = q;
      }
    }
  });
  for (int c = 0; c < 256; ++c) {
    uint64_t acc = 0;
    for (auto &p : part) acc += p[c];
    hist[c] = acc;
  }
}

// eq. emp_entropy over a 256-bin histogram, summed in ascending code order.
double entropy_bits(const uint64_t hist[256]) {
  uint64_t n = 0;
  for (int c = 0; c < 256; ++c) n += hist[c];
  if (!n) return 0.0;
  double h = 0.0;
  for (int c = 0; c < 256; ++c) {
    if (!hist[c]) continue;
    double p = static_cast<double>(hist[c]) / static_cast<double>(n);
    h -= p * std::log2(p);
  }
  return h;
}

// ANS metadata: frequencies summing to 2^P over the present symbols (ascending
// code): f = max(1, floor(n_k 2^P / n)); surplus units by largest remainder
// (ties: lower code), cycling; excess units removed one at a time from the
// largest f > 1 (ties: lower code).
bool normalise(const uint64_t hist[256], uint32_t P, std::vector<uint8_t> &sym,
               std::vector<uint16_t> &freq) {
  const int64_t M = int64_t(1) << P;
  uint64_t n = 0;
  sym.clear();
  for (int c = 0; c < 256; ++c)
    if (hist[c]) {
      sym.push_back(static_cast<uint8_t>(c));
      n += hist[c];
    }
  const size_t K = sym.size();
  if (K == 0 || static_cast<int64_t>(K) > M) return false;
  std::vector<int64_t> f(K);
  std::vector<uint64_t> rem(K);
  if (K == 1) {
    freq.assign(1, static_cast<uint16_t>(M));
    return true;
  }
  int64_t sum = 0;
  for (size_t k = 0; k < K; ++k) {
    uint64_t num = hist[sym[k]] * static_cast<uint64_t>(M);
    f[k] = std::max<int64_t>(1, static_cast<int64_t>(num / n));
    rem[k] = num % n;
    sum += f[k];
  }
  int64_t deficit = M - sum;
  if (deficit > 0) {
    std::vector<size_t> order(K);
    for (size_t k = 0; k < K; ++k) order[k] = k;
    std::stable_sort(order.begin(), order.end(),
                     [&](size_t a, size_t b) { return rem[a] > rem[b]; });
    for (size_t i = 0; deficit > 0; i = (i + 1) % K, --deficit) ++f[order[i]];
  }
  while (deficit < 0) {
    size_t best = K;
    for (size_t k = 0; k < K; ++k)
      if (f[k] > 1 && (best == K || f[k] > f[best])) best = k;
    if (best == K) return false;
    --f[best];
    ++deficit;
  }
  freq.resize(K);
  for (size_t k = 0; k < K; ++k) freq[k] = static_cast<uint16_t>(f[k]);
  return true;
}

struct SymbolCoder {
  uint32_t freq = 0, cum = 0;
  uint64_t push_at = 0;  // push a word first when x >= freq * 2^(32-P)
};

// Encode one chunk of n symbols.  Words are produced back to front into
// `out` (capacity n), so the decoder reads them front to back; returns the
// number of words, which end at out + n.
uint32_t encode_chunk(const uint8_t *q, uint32_t n, uint32_t W, uint32_t P,
                      const SymbolCoder *coder, uint16_t *out_end, uint32_t *states) {
  std::vector<uint64_t> x(W, kStateLow);
  uint16_t *w = out_end;
  const uint32_t T = (n + W - 1) / W;
  for (uint32_t t = T; t-- > 0;) {
    const uint32_t base = t * W;
    const uint32_t last = std::min(W, n - base);
    for (uint32_t l = last; l-- > 0;) {
      const SymbolCoder &c = coder[q[base + l]];
      uint64_t s = x[l];
      if (s >= c.push_at) {
        *--w = static_cast<uint16_t>(s & 0xFFFF);
        s >>= 16;
      }
      x[l] = ((s / c.freq) << P) + (s % c.freq) + c.cum;
    }
  }
  for (uint32_t l = 0; l < W; ++l) states[l] = static_cast<uint32_t>(x[l]);
  return static_cast<uint32_t>(out_end - w);
}

template <class T>
void put(uint8_t *b, uint64_t off, T v) {
  std::memcpy(b + off, &v, sizeof v);  // little-endian host
}

uint64_t round_up(uint64_t v, uint64_t a) { return (v + a - 1) / a * a; }

}  // namespace

extern "C" float eqe_alpha_search(const uint16_t *w, uint32_t M, uint32_t N, double target_bits,
                                  uint32_t sample_rows, uint32_t threads, uint32_t base_format,
                                  double *h_out) {
  if (base_format == 0) base_format = kFmtE4M3;
  if (!w || !M || !N || (base_format != kFmtE4M3 && base_format != kFmtInt8)) return -1.0f;
  std::vector<uint32_t> rows;
  if (sample_rows && sample_rows < M) {
    for (uint32_t r = 0; r < sample_rows; ++r)
      rows.push_back(static_cast<uint32_t>(static_cast<uint64_t>(r) * M / sample_rows));
  } else {
    for (uint32_t r = 0; r < M; ++r) rows.push_back(r);
  }
  const unsigned nt = worker_count(threads);
  double lo = -4.0, hi = 24.0, best_err = INFINITY, best_h = 0.0;
  float best = 1.0f;
  for (int it = 0; it < 40; ++it) {
    const double mid = 0.5 * (lo + hi);
    const float alpha = static_cast<float>(std::exp2(mid));
    uint64_t hist[256];
    quantize_rows(w, N, alpha, base_format, rows, nt, nullptr, nullptr, hist);
    const double h = entropy_bits(hist);
    if (std::fabs(h - target_bits) < best_err) {
      best_err = std::fabs(h - target_bits);
      best = alpha;
      best_h = h;
    }
    (h > target_bits ? lo : hi) = mid;
  }
  if (h_out) *h_out = best_h;
  return best;
}

namespace {

// Scale usable by the decoder (finite, normal, 2^-117 <= s < 2^120, so
// every dequantised product is exact in fp32) and positive.
bool scale_usable(uint16_t s) {
  const int e = (s >> 7) & 0xFF;
  return !(s & 0x8000) && e >= 127 - 117 && e <= 127 + 119;
}

// Alg. 1: quantise with the AbsMax scales times alpha, or with the given
// scales when `given` is non-null (alpha is then recorded as 0), and encode.
int encode_impl(const uint16_t *w, uint32_t M, uint32_t N, float alpha, const uint16_t *given,
                const eqe_params *p, uint8_t **blob_out, uint64_t *bytes_out) {
  if (!w || !p || !blob_out || !bytes_out || !M || !N) return -1;
  const uint64_t n = static_cast<uint64_t>(M) * N;
  const uint32_t W = p->lanes, C = p->chunk_syms, P = p->prob_bits;
  const uint32_t fmt = p->base_format ? p->base_format : kFmtE4M3;
  if (n >= (uint64_t(1) << 32) || (W != 64 && W != 128 && W != 256) || C == 0 || C % W ||
      P < 8 || P > 12 || (!given && !(alpha > 0.0f)) || (fmt != kFmtE4M3 && fmt != kFmtInt8))
    return -1;
  if (given)
    for (uint32_t i = 0; i < M; ++i)
      if (!scale_usable(given[i])) return -1;
  const unsigned nt = worker_count(p->threads);
  try {
    std::vector<uint16_t> scale(M);
    std::vector<uint8_t> codes(n);
    std::vector<uint32_t> rows(M);
    for (uint32_t i = 0; i < M; ++i) rows[i] = i;
    uint64_t hist[256];
    quantize_rows(w, N, alpha, fmt, rows, nt, scale.data(), codes.data(), hist, given);

    std::vector<uint8_t> sym;
    std::vector<uint16_t> freq;
    if (!normalise(hist, P, sym, freq)) return -1;
    SymbolCoder coder[256];
    uint32_t cum = 0;
    for (size_t k = 0; k < sym.size(); ++k) {
      coder[sym[k]].freq = freq[k];
      coder[sym[k]].cum = cum;
      coder[sym[k]].push_at = static_cast<uint64_t>(freq[k]) << (32 - P);
      cum += freq[k];
    }

    const uint32_t n_chunks = static_cast<uint32_t>((n + C - 1) / C);
    std::vector<uint16_t> scratch(static_cast<uint64_t>(n_chunks) * C);
    std::vector<uint32_t> count(n_chunks);
    std::vector<uint32_t> states(static_cast<uint64_t>(n_chunks) * W);
    parallel_for(n_chunks, nt, [&](uint64_t c) {
      const uint64_t k0 = c * C;
      const uint32_t nc = static_cast<uint32_t>(std::min<uint64_t>(C, n - k0));
      count[c] = encode_chunk(codes.data() + k0, nc, W, P, coder, scratch.data() + k0 + C,
                              states.data() + c * W);
    });
    std::vector<uint32_t> off(n_chunks + 1, 0);
    for (uint32_t c = 0; c < n_chunks; ++c) off[c + 1] = off[c] + count[c];
    const uint64_t total = off[n_chunks];
    const uint64_t padded = round_up(total + 1024, 128);
    const uint32_t K = static_cast<uint32_t>(sym.size());

    const uint64_t o_scale = kHeaderBytes;
    const uint64_t o_sym = round_up(o_scale + 2ull * M, 256);
    const uint64_t o_freq = round_up(o_sym + K, 256);
    const uint64_t o_off = round_up(o_freq + 2ull * K, 256);
    const uint64_t o_state = round_up(o_off + 4ull * (n_chunks + 1), 256);
    const uint64_t o_words = round_up(o_state + 4ull * n_chunks * W, 256);
    const uint64_t bytes = round_up(o_words + 2 * padded, 256);
    uint8_t *b = static_cast<uint8_t *>(std::calloc(1, bytes));
    if (!b) return -5;
    std::memcpy(b, "EQC1", 4);
    put<uint32_t>(b, 4, 1);                  // version
    put<uint32_t>(b, 8, kHeaderBytes);
    put<uint32_t>(b, 12, fmt);               // base format: 1 E4M3FN, 2 Int8
    put<uint32_t>(b, 16, M);
    put<uint32_t>(b, 20, N);
    put<uint32_t>(b, 24, C);
    put<uint32_t>(b, 28, n_chunks);
    put<uint32_t>(b, 32, W);
    put<uint32_t>(b, 36, P);
    put<uint32_t>(b, 40, K);
    put<uint32_t>(b, 44, 0);                 // flags
    put<uint64_t>(b, 48, total);
    put<uint64_t>(b, 56, padded);
    put<uint64_t>(b, 64, p->seed);
    put<float>(b, 72, given ? 0.0f : alpha);
    put<float>(b, 76, p->target_bits);
    put<float>(b, 80, static_cast<float>(entropy_bits(hist)));
    put<uint64_t>(b, 88, o_scale);
    put<uint64_t>(b, 96, o_sym);
    put<uint64_t>(b, 104, o_freq);
    put<uint64_t>(b, 112, o_off);
    put<uint64_t>(b, 120, o_state);
    put<uint64_t>(b, 128, o_words);
    put<uint64_t>(b, 136, bytes);
    std::memcpy(b + o_scale, scale.data(), 2ull * M);
    std::memcpy(b + o_sym, sym.data(), K);
    std::memcpy(b + o_freq, freq.data(), 2ull * K);
    std::memcpy(b + o_off, off.data(), 4ull * (n_chunks + 1));
    std::memcpy(b + o_state, states.data(), 4ull * n_chunks * W);
    parallel_for(n_chunks, nt, [&](uint64_t c) {
      const uint64_t end = c * C + C;
      std::memcpy(b + o_words + 2ull * off[c], scratch.data() + end - count[c], 2ull * count[c]);
    });
    *blob_out = b;
    *bytes_out = bytes;
    return 0;
  } catch (const std::bad_alloc &) {
    return -5;
  }
}

}  // namespace

extern "C" int eqe_encode(const uint16_t *w, uint32_t M, uint32_t N, float alpha,
                          const eqe_params *p, uint8_t **blob_out, uint64_t *bytes_out) {
  return encode_impl(w, M, N, alpha, nullptr, p, blob_out, bytes_out);
}

extern "C" int eqe_encode_scaled(const uint16_t *w, uint32_t M, uint32_t N,
                                 const uint16_t *scale_bf16, const eqe_params *p,
                                 uint8_t **blob_out, uint64_t *bytes_out) {
  if (!scale_bf16) return -1;
  return encode_impl(w, M, N, 0.0f, scale_bf16, p, blob_out, bytes_out);
}

extern "C" int eqe_rd_lambda_search(const uint16_t *w, uint32_t M, uint32_t N,
                                    double target_bits, uint32_t sample_rows,
                                    const eqe_rd_params *prm, double *lambda_out, double *h_out) {
  if (!w || !M || !N || !prm || !lambda_out) return -1;
  const uint32_t fmt = prm->base_format ? prm->base_format : kFmtE4M3;
  if (fmt != kFmtE4M3 && fmt != kFmtInt8) return -1;
  try {
    // the rows searched, copied contiguously
    const uint32_t R = (sample_rows && sample_rows < M) ? sample_rows : M;
    std::vector<uint16_t> sub(static_cast<uint64_t>(R) * N);
    for (uint32_t r = 0; r < R; ++r) {
      const uint64_t i = R == M ? r : static_cast<uint64_t>(r) * M / R;
      std::memcpy(sub.data() + static_cast<uint64_t>(r) * N, w + i * N, 2ull * N);
    }
    std::vector<uint32_t> rows(R);
    for (uint32_t r = 0; r < R; ++r) rows[r] = r;
    std::vector<uint16_t> sb(R);
    const unsigned nt = worker_count(prm->threads);
    double lo = -8.0, hi = 16.0, best_err = INFINITY, best_h = 0.0, best = 1.0;
    for (int it = 0; it < 14; ++it) {
      const double mid = 0.5 * (lo + hi);
      eqe_rd_params q = *prm;
      q.lambda = std::exp2(mid);
      q.base_format = fmt;
      const int rc = eqe_rd_scales(sub.data(), R, N, &q, nullptr, sb.data(), nullptr);
      if (rc != 0) return rc;
      uint64_t hist[256];
      quantize_rows(sub.data(), N, 0.0f, fmt, rows, nt, nullptr, nullptr, hist, sb.data());
      const double h = entropy_bits(hist);
      if (std::fabs(h - target_bits) < best_err) {
        best_err = std::fabs(h - target_bits);
        best = q.lambda;
        best_h = h;
      }
      (h > target_bits ? lo : hi) = mid;  // larger lambda -> lower entropy
    }
    *lambda_out = best;
    if (h_out) *h_out = best_h;
    return 0;
  } catch (const std::bad_alloc &) {
    return -5;
  }
}

extern "C" void eqe_free(void *ptr) { std::free(ptr); }

// ---------------------------------------------------------------------------
// Container version 2: tiles of TR rows x TC columns are the chunks (row s of
// a tile is the segment of coder state s), each segment coded as a greedy
// parse into quads, pairs and single codes from a per-layer dictionary, with
// rANS at M = 2^16 and frequencies in multiples of 2^(16-R).  The rules
// (dictionary shares, the choice among tau = 8, 4, 2, 1, the normalisation)
// are stated in eq_encode.h.
// ---------------------------------------------------------------------------
namespace {

constexpr uint32_t kNoEntry = 0xFFFFFFFFu;

// Open-addressing counter keyed by a 32-bit value.
class Counter {
 public:
  Counter() : keys_(1024, 0), counts_(1024, 0), used_(1024, 0) {}
  void add(uint32_t key, uint64_t n = 1) {
    if (2 * (size_ + 1) > keys_.size()) grow();
    size_t i = slot(key);
    if (!used_[i]) {
      used_[i] = 1;
      keys_[i] = key;
      ++size_;
    }
    counts_[i] += n;
  }
  void merge(const Counter &o) {
    for (size_t i = 0; i < o.keys_.size(); ++i)
      if (o.used_[i]) add(o.keys_[i], o.counts_[i]);
  }
  template <class Fn>
  void each(Fn fn) const {
    for (size_t i = 0; i < keys_.size(); ++i)
      if (used_[i]) fn(keys_[i], counts_[i]);
  }

 private:
  size_t slot(uint32_t key) const {
    const size_t mask = keys_.size() - 1;
    size_t i = (key * 0x9E3779B1u) & mask;
    while (used_[i] && keys_[i] != key) i = (i + 1) & mask;
    return i;
  }
  void grow() {
    std::vector<uint32_t> k;
    std::vector<uint64_t> c;
    std::vector<uint8_t> u;
    k.swap(keys_), c.swap(counts_), u.swap(used_);
    keys_.assign(2 * k.size(), 0), counts_.assign(2 * k.size(), 0), used_.assign(2 * k.size(), 0);
    size_ = 0;
    for (size_t i = 0; i < k.size(); ++i)
      if (u[i]) add(k[i], c[i]);
  }
  std::vector<uint32_t> keys_;
  std::vector<uint64_t> counts_;
  std::vector<uint8_t> used_;
  size_t size_ = 0;
};

// Sorted set of dictionary values with their indices, looked up by hashing.
class Lookup {
 public:
  explicit Lookup(const std::vector<uint32_t> &vals) {
    size_t cap = 16;
    while (cap < 4 * vals.size()) cap *= 2;
    keys_.assign(cap, 0);
    idx_.assign(cap, kNoEntry);
    for (uint32_t k = 0; k < vals.size(); ++k) {
      size_t i = (vals[k] * 0x9E3779B1u) & (cap - 1);
      while (idx_[i] != kNoEntry) i = (i + 1) & (cap - 1);
      keys_[i] = vals[k];
      idx_[i] = k;
    }
  }
  uint32_t find(uint32_t v) const {
    const size_t mask = keys_.size() - 1;
    for (size_t i = (v * 0x9E3779B1u) & mask;; i = (i + 1) & mask) {
      if (idx_[i] == kNoEntry) return kNoEntry;
      if (keys_[i] == v) return idx_[i];
    }
  }

 private:
  std::vector<uint32_t> keys_, idx_;
};

inline uint32_t quad_at(const uint8_t *u) {
  uint32_t v;
  std::memcpy(&v, u, 4);  // little-endian host: codes in position order
  return v;
}
inline uint32_t pair_at(const uint8_t *u) { return uint32_t(u[0]) | uint32_t(u[1]) << 8; }

struct Geometry {
  uint32_t M, N, TR, TC, NT, n_chunks;
  void tile(uint32_t c, uint32_t &r0, uint32_t &c0, uint32_t &rows, uint32_t &cols) const {
    r0 = (c / NT) * TR;
    c0 = (c % NT) * TC;
    rows = std::min(TR, M - r0);
    cols = std::min(TC, N - c0);
  }
};

// Values passing count * 2^(R+2) >= tau * units, at most cap of them by
// (count desc, value asc), returned ascending.
std::vector<uint32_t> select_values(const Counter &h, uint64_t units, uint32_t R, uint32_t tau,
                                    uint32_t cap) {
  std::vector<std::pair<uint64_t, uint32_t>> cand;
  h.each([&](uint32_t v, uint64_t c) {
    if ((c << (R + 2)) >= uint64_t(tau) * units) cand.emplace_back(c, v);
  });
  std::sort(cand.begin(), cand.end(), [](const auto &a, const auto &b) {
    return a.first != b.first ? a.first > b.first : a.second < b.second;
  });
  if (cand.size() > cap) cand.resize(cap);
  std::vector<uint32_t> out;
  for (auto &p : cand) out.push_back(p.second);
  std::sort(out.begin(), out.end());
  return out;
}

// Counts of the units of width 4 (positions 0, 4, ...) or 2 (0, 2, ...) of
// every segment.
Counter unit_counts(const uint8_t *q, const Geometry &g, uint32_t width, unsigned nt,
                    uint64_t &units) {
  std::vector<Counter> part(nt);
  std::atomic<uint32_t> next_task{0};
  const uint32_t tasks = g.M;  // one row at a time, all its tiles
  auto body = [&](unsigned id) {
    Counter &h = part[id];
    for (uint32_t r; (r = next_task.fetch_add(1)) < tasks;) {
      const uint8_t *row = q + uint64_t(r) * g.N;
      for (uint32_t t = 0; t < g.NT; ++t) {
        const uint32_t c0 = t * g.TC, w = std::min(g.TC, g.N - c0);
        for (uint32_t j = 0; j + width <= w; j += width)
          h.add(width == 4 ? quad_at(row + c0 + j) : pair_at(row + c0 + j));
      }
    }
  };
  std::vector<std::thread> pool;
  for (unsigned t = 1; t < nt; ++t) pool.emplace_back(body, t);
  body(0);
  for (auto &t : pool) t.join();
  units = 0;
  for (uint32_t t = 0; t < g.NT; ++t) units += uint64_t(g.M) * (std::min(g.TC, g.N - t * g.TC) / width);
  Counter all;
  for (auto &p : part) all.merge(p);
  return all;
}

// Greedy parse of one segment; emits raw symbol ids: quad k, pair nq + k,
// single nq + np + code.
template <class Emit>
void parse(const uint8_t *u, uint32_t w, const Lookup &dq, const Lookup &dp, uint32_t nq,
           uint32_t np, Emit emit) {
  uint32_t j = 0;
  while (j < w) {
    if (j + 4 <= w) {
      const uint32_t k = dq.find(quad_at(u + j));
      if (k != kNoEntry) {
        emit(k);
        j += 4;
        continue;
      }
    }
    if (j + 2 <= w) {
      const uint32_t k = dp.find(pair_at(u + j));
      if (k != kNoEntry) {
        emit(nq + k);
        j += 2;
        continue;
      }
    }
    emit(nq + np + u[j]);
    j += 1;
  }
}

// Counts to frequencies >= 1 summing to 2^R: the rule of normalise() above
// over an arbitrary alphabet (ties by lower index).
bool normalise_counts(const std::vector<uint64_t> &cnt, uint32_t R, std::vector<uint16_t> &freq) {
  const size_t K = cnt.size();
  const int64_t M = int64_t(1) << R;
  if (K == 0 || int64_t(K) > M) return false;
  uint64_t n = 0;
  for (uint64_t c : cnt) {
    if (!c) return false;
    n += c;
  }
  std::vector<int64_t> f(K);
  std::vector<uint64_t> rem(K);
  int64_t sum = 0;
  for (size_t k = 0; k < K; ++k) {
    const uint64_t num = cnt[k] * uint64_t(M);
    f[k] = std::max<int64_t>(1, int64_t(num / n));
    rem[k] = num % n;
    sum += f[k];
  }
  int64_t deficit = M - sum;
  if (deficit > 0) {
    std::vector<size_t> order(K);
    for (size_t k = 0; k < K; ++k) order[k] = k;
    std::stable_sort(order.begin(), order.end(),
                     [&](size_t a, size_t b) { return rem[a] > rem[b]; });
    for (size_t i = 0; deficit > 0; i = (i + 1) % K, --deficit) ++f[order[i]];
  }
  while (deficit < 0) {
    size_t best = K;
    for (size_t k = 0; k < K; ++k)
      if (f[k] > 1 && (best == K || f[k] > f[best])) best = k;
    if (best == K) return false;
    --f[best];
    ++deficit;
  }
  freq.resize(K);
  for (size_t k = 0; k < K; ++k) freq[k] = static_cast<uint16_t>(f[k]);
  return true;
}

// One candidate alphabet: its dictionaries after dropping unused entries,
// the renumbering of raw symbol ids, counts, frequencies and coded bits.
struct Alphabet {
  std::vector<uint32_t> quads, pairs;  // as selected (before dropping)
  std::vector<uint32_t> map;           // raw id -> final index
  std::vector<uint32_t> phr;           // final phrases: codes as a little-endian u32
  uint32_t nq = 0, np = 0, ns = 0;
  std::vector<uint64_t> cnt;
  std::vector<uint16_t> freq;
  double bits = 0.0;
};

bool make_alphabet(const uint8_t *q, const Geometry &g, uint32_t R, uint32_t tau,
                   const Counter &quad_h, uint64_t quad_units, const std::vector<uint32_t> &pairs,
                   unsigned nt, Alphabet &a) {
  a.quads = select_values(quad_h, quad_units, R, tau, 1u << (R - 1));
  a.pairs = pairs;
  const uint32_t nq = uint32_t(a.quads.size()), np = uint32_t(a.pairs.size());
  const uint32_t raw = nq + np + 256;
  const Lookup dq(a.quads), dp(a.pairs);
  std::vector<std::vector<uint64_t>> part(nt, std::vector<uint64_t>(raw, 0));
  std::atomic<uint32_t> next_task{0};
  auto body = [&](unsigned id) {
    uint64_t *h = part[id].data();
    for (uint32_t r; (r = next_task.fetch_add(1)) < g.M;) {
      const uint8_t *row = q + uint64_t(r) * g.N;
      for (uint32_t t = 0; t < g.NT; ++t) {
        const uint32_t c0 = t * g.TC, w = std::min(g.TC, g.N - c0);
        parse(row + c0, w, dq, dp, nq, np, [&](uint32_t s) { ++h[s]; });
      }
    }
  };
  std::vector<std::thread> pool;
  for (unsigned t = 1; t < nt; ++t) pool.emplace_back(body, t);
  body(0);
  for (auto &t : pool) t.join();
  std::vector<uint64_t> seen(raw, 0);
  for (auto &p : part)
    for (uint32_t s = 0; s < raw; ++s) seen[s] += p[s];
  a.map.assign(raw, kNoEntry);
  a.phr.clear();
  a.cnt.clear();
  a.nq = a.np = a.ns = 0;
  for (uint32_t k = 0; k < nq; ++k)
    if (seen[k]) a.map[k] = uint32_t(a.phr.size()), a.phr.push_back(a.quads[k]),
                 a.cnt.push_back(seen[k]), ++a.nq;
  for (uint32_t k = 0; k < np; ++k)
    if (seen[nq + k]) a.map[nq + k] = uint32_t(a.phr.size()), a.phr.push_back(a.pairs[k]),
                      a.cnt.push_back(seen[nq + k]), ++a.np;
  for (uint32_t c = 0; c < 256; ++c)
    if (seen[nq + np + c]) a.map[nq + np + c] = uint32_t(a.phr.size()), a.phr.push_back(c),
                           a.cnt.push_back(seen[nq + np + c]), ++a.ns;
  if (a.phr.size() > (size_t(1) << R)) return false;
  if (!normalise_counts(a.cnt, R, a.freq)) return false;
  a.bits = 0.0;
  for (size_t k = 0; k < a.cnt.size(); ++k)
    a.bits += double(a.cnt[k]) * std::log2(double(1u << R) / double(a.freq[k]));
  return true;
}

// Encode one chunk: the states' symbol sequences (sym[off[s] .. off[s] +
// len[s])) back to front; words are produced into `out_end` backwards.
uint64_t encode_chunk2(const uint16_t *sym, const uint32_t *off, const uint32_t *len, uint32_t W,
                       const uint64_t *F, const uint64_t *CUM, uint16_t *out_end,
                       uint32_t *states) {
  std::vector<uint64_t> x(W, kStateLow);
  uint32_t T = 0;
  for (uint32_t s = 0; s < W; ++s) T = std::max(T, len[s]);
  uint16_t *w = out_end;
  for (uint32_t t = T; t-- > 0;)
    for (uint32_t s = W; s-- > 0;) {
      if (t >= len[s]) continue;
      const uint32_t k = sym[off[s] + t];
      uint64_t v = x[s];
      if (v >= (F[k] << 16)) {
        *--w = static_cast<uint16_t>(v & 0xFFFF);
        v >>= 16;
      }
      x[s] = (v / F[k]) * 65536 + (v % F[k]) + CUM[k];
    }
  for (uint32_t s = 0; s < W; ++s) states[s] = static_cast<uint32_t>(x[s]);
  return static_cast<uint64_t>(out_end - w);
}

int encode2_impl(const uint16_t *w, uint32_t M, uint32_t N, float alpha, const uint16_t *given,
                 const eqe_params2 *p, uint8_t **blob_out, uint64_t *bytes_out) {
  if (!w || !p || !blob_out || !bytes_out || !M || !N) return -1;
  const uint64_t n = static_cast<uint64_t>(M) * N;
  const uint32_t R = p->res_bits, TR = p->tile_rows, TC = p->tile_cols;
  const uint32_t fmt = p->base_format ? p->base_format : kFmtE4M3;
  if (n >= (uint64_t(1) << 32) || (TR != 64 && TR != 128 && TR != 256) || TC == 0 || TC % 4 ||
      uint64_t(TR) * TC >= (uint64_t(1) << 32) || R < 10 || R > 12 ||
      (!given && !(alpha > 0.0f)) || (fmt != kFmtE4M3 && fmt != kFmtInt8) || p->row_order > 1)
    return -1;
  if (given)
    for (uint32_t i = 0; i < M; ++i)
      if (!scale_usable(given[i])) return -1;
  Geometry g{M, N, TR, TC, (N + TC - 1) / TC, 0};
  const uint64_t nchunks64 = uint64_t(g.NT) * ((M + TR - 1) / TR);
  if (nchunks64 >= (uint64_t(1) << 32)) return -1;
  g.n_chunks = uint32_t(nchunks64);
  const unsigned nt = worker_count(p->threads);
  try {
    std::vector<uint16_t> scale(M);
    std::vector<uint8_t> codes(n);
    std::vector<uint32_t> rows(M);
    for (uint32_t i = 0; i < M; ++i) rows[i] = i;
    uint64_t hist[256];
    quantize_rows(w, N, alpha, fmt, rows, nt, scale.data(), codes.data(), hist, given);

    uint64_t quad_units = 0, pair_units = 0;
    const Counter quad_h = unit_counts(codes.data(), g, 4, nt, quad_units);
    const Counter pair_h = unit_counts(codes.data(), g, 2, nt, pair_units);
    const std::vector<uint32_t> pairs = select_values(pair_h, pair_units, R, 1, 1u << (R - 2));
    Alphabet best, cur;
    uint32_t best_tau = 0;
    for (uint32_t tau = 8; tau >= 1; tau /= 2) {
      if (!make_alphabet(codes.data(), g, R, tau, quad_h, quad_units, pairs, nt, cur)) return -1;
      if (best_tau == 0 || cur.bits < best.bits) {
        best = cur;
        best_tau = tau;
      }
    }
    const uint32_t n_sym = uint32_t(best.phr.size());
    std::vector<uint64_t> F(n_sym), CUM(n_sym);
    for (uint32_t k = 0, acc = 0; k < n_sym; ++k) {
      F[k] = uint64_t(best.freq[k]) << (16 - R);
      CUM[k] = acc;
      acc += uint32_t(F[k]);
    }

    // parse and encode every chunk
    const Lookup dq(best.quads), dp(best.pairs);
    const uint32_t nq_raw = uint32_t(best.quads.size()), np_raw = uint32_t(best.pairs.size());

    // Row order: the rows by ascending phrase count over their segments
    // (ties: lower row), so that a tile's rows, which it takes as many steps
    // to decode as its longest one needs, are alike.  The alphabet does not
    // depend on it.
    std::vector<uint32_t> order(M);
    for (uint32_t i = 0; i < M; ++i) order[i] = i;
    if (p->row_order) {
      std::vector<uint64_t> cost(M, 0);
      parallel_for(M, nt, [&](uint64_t r) {
        uint64_t k = 0;
        for (uint32_t t = 0; t < g.NT; ++t) {
          const uint32_t c0 = t * g.TC, w = std::min(g.TC, N - c0);
          parse(codes.data() + r * N + c0, w, dq, dp, nq_raw, np_raw, [&](uint32_t) { ++k; });
        }
        cost[r] = k;
      });
      std::stable_sort(order.begin(), order.end(),
                       [&](uint32_t a, uint32_t b) { return cost[a] < cost[b]; });
    }
    std::vector<std::vector<uint16_t>> words(g.n_chunks);
    std::vector<uint32_t> states(uint64_t(g.n_chunks) * TR);
    parallel_for(g.n_chunks, nt, [&](uint64_t c) {
      uint32_t r0, c0, rws, cols;
      g.tile(uint32_t(c), r0, c0, rws, cols);
      std::vector<uint16_t> sym;
      sym.reserve(uint64_t(rws) * cols / 2);
      std::vector<uint32_t> off(TR, 0), len(TR, 0);
      for (uint32_t s = 0; s < rws; ++s) {
        off[s] = uint32_t(sym.size());
        parse(codes.data() + uint64_t(order[r0 + s]) * N + c0, cols, dq, dp, nq_raw, np_raw,
              [&](uint32_t raw) { sym.push_back(static_cast<uint16_t>(best.map[raw])); });
        len[s] = uint32_t(sym.size()) - off[s];
      }
      for (uint32_t s = rws; s < TR; ++s) off[s] = uint32_t(sym.size());
      std::vector<uint16_t> buf(sym.size() + 16);
      const uint64_t nw = encode_chunk2(sym.data(), off.data(), len.data(), TR, F.data(),
                                        CUM.data(), buf.data() + buf.size(),
                                        states.data() + c * TR);
      words[c].assign(buf.end() - nw, buf.end());
    });
    std::vector<uint64_t> off(uint64_t(g.n_chunks) + 1, 0);
    for (uint32_t c = 0; c < g.n_chunks; ++c) off[c + 1] = off[c] + words[c].size();
    const uint64_t total = off[g.n_chunks];
    if (total >= (uint64_t(1) << 32)) return -1;
    const uint64_t padded = round_up(total + 1024, 128);

    const uint64_t o_scale = kHeaderBytes;
    const uint64_t o_phr = round_up(o_scale + 2ull * M, 256);
    const uint64_t o_freq = round_up(o_phr + 4ull * n_sym, 256);
    const uint64_t o_off = round_up(o_freq + 2ull * n_sym, 256);
    const uint64_t o_state = round_up(o_off + 4ull * (g.n_chunks + 1), 256);
    const uint64_t o_order = p->row_order ? round_up(o_state + 4ull * g.n_chunks * TR, 256) : 0;
    const uint64_t o_words = p->row_order ? round_up(o_order + 4ull * M, 256)
                                          : round_up(o_state + 4ull * g.n_chunks * TR, 256);
    const uint64_t bytes = round_up(o_words + 2 * padded, 256);
    uint8_t *b = static_cast<uint8_t *>(std::calloc(1, bytes));
    if (!b) return -5;
    std::memcpy(b, "EQC1", 4);
    put<uint32_t>(b, 4, 2);                  // version
    put<uint32_t>(b, 8, kHeaderBytes);
    put<uint32_t>(b, 12, fmt);
    put<uint32_t>(b, 16, M);
    put<uint32_t>(b, 20, N);
    put<uint32_t>(b, 24, TR * TC);
    put<uint32_t>(b, 28, g.n_chunks);
    put<uint32_t>(b, 32, TR);
    put<uint32_t>(b, 36, R);
    put<uint32_t>(b, 40, n_sym);
    put<uint32_t>(b, 44, p->row_order ? 1u : 0u);  // flags: bit 0, row order
    put<uint64_t>(b, 48, total);
    put<uint64_t>(b, 56, padded);
    put<uint64_t>(b, 64, p->seed);
    put<float>(b, 72, given ? 0.0f : alpha);
    put<float>(b, 76, p->target_bits);
    put<float>(b, 80, static_cast<float>(entropy_bits(hist)));
    put<uint32_t>(b, 84, TC);
    put<uint64_t>(b, 88, o_scale);
    put<uint64_t>(b, 96, o_phr);
    put<uint64_t>(b, 104, o_freq);
    put<uint64_t>(b, 112, o_off);
    put<uint64_t>(b, 120, o_state);
    put<uint64_t>(b, 128, o_words);
    put<uint64_t>(b, 136, bytes);
    put<uint32_t>(b, 144, best.nq);
    put<uint32_t>(b, 148, best.np);
    put<uint32_t>(b, 152, best.ns);
    put<uint32_t>(b, 156, best_tau);
    put<uint64_t>(b, 160, o_order);
    if (p->row_order) std::memcpy(b + o_order, order.data(), 4ull * M);
    std::memcpy(b + o_scale, scale.data(), 2ull * M);
    std::memcpy(b + o_phr, best.phr.data(), 4ull * n_sym);
    std::memcpy(b + o_freq, best.freq.data(), 2ull * n_sym);
    for (uint32_t c = 0; c <= g.n_chunks; ++c) put<uint32_t>(b, o_off + 4ull * c, uint32_t(off[c]));
    std::memcpy(b + o_state, states.data(), 4ull * g.n_chunks * TR);
    parallel_for(g.n_chunks, nt, [&](uint64_t c) {
      if (!words[c].empty())
        std::memcpy(b + o_words + 2 * off[c], words[c].data(), 2 * words[c].size());
    });
    *blob_out = b;
    *bytes_out = bytes;
    return 0;
  } catch (const std::bad_alloc &) {
    return -5;
  }
}

}  // namespace

extern "C" int eqe_encode2(const uint16_t *w, uint32_t M, uint32_t N, float alpha,
                           const uint16_t *scale_bf16, const eqe_params2 *p, uint8_t **blob_out,
                           uint64_t *bytes_out) {
  return encode2_impl(w, M, N, scale_bf16 ? 0.0f : alpha, scale_bf16, p, blob_out, bytes_out);
}
