// Scale optimisation of the encoder (declared in eq_encode.h).
//
// Sec. 2.2 of the paper, eq. optimization: per layer, minimise over the
// channel-wise scales S
//   F(S) = ||W - W_hat||_1 / ||W||_1 + lambda * R(W_q),
//   W_q = Q(W / S),  W_hat = S * W_q,
// with R the entry-wise l1 norm of the quantised values (taken per entry,
// i.e. divided by M*N, so that lambda is independent of the layer size),
// starting from the AbsMax scales (eq. absmax), with L-BFGS and the
// straight-through estimator for the rounding of Q (Alg. 1, the scale optimisation).  The
// objective separates over rows, so one evaluation is one pass over W with
// rows spread over threads.
#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstring>
#include <thread>
#include <vector>

#include "eq_encode.h"

namespace {

constexpr uint32_t kFmtE4M3 = 1, kFmtInt8 = 2;

unsigned workers(uint32_t requested) {
  if (requested) return requested;
  unsigned n = std::thread::hardware_concurrency();
  return n ? std::min(n, 16u) : 1;
}

template <class Fn>
void parallel_rows(uint32_t M, unsigned threads, Fn fn) {
  threads = std::min<unsigned>(threads, M);
  if (threads <= 1) {
    for (uint32_t i = 0; i < M; ++i) fn(i);
    return;
  }
  std::atomic<uint32_t> next{0};
  auto body = [&] {
    for (uint32_t i; (i = next.fetch_add(1)) < M;) fn(i);
  };
  std::vector<std::thread> pool;
  for (unsigned t = 1; t < threads; ++t) pool.emplace_back(body);
  body();
  for (auto &t : pool) t.join();
}

float bf16_value(uint16_t b) {
  const uint32_t u = static_cast<uint32_t>(b) << 16;
  float f;
  std::memcpy(&f, &u, 4);
  return f;
}

// Nearest integer of |x| < 2^22, ties to even: adding and subtracting
// 1.5 * 2^23 rounds in the default (nearest-even) mode without a libm call.
inline float round_even(float x) {
  const volatile float big = 12582912.0f;  // kept out of constant folding
  return (x + big) - big;
}

// Value of the nearest E4M3FN number to v after clamping to +-448 (ties to
// even), computed on the float bit pattern: normal range by rounding the
// significand to 3 bits in place, subnormal range (|v| < 2^-6) on the grid
// k * 2^-9.
// Both candidates are formed and one is selected, so that the loop over a
// row stays free of data-dependent branches.
float q_e4m3(float v) {
  const float a = std::min(std::fabs(v), 448.0f);
  const float sub = round_even(a * 512.0f) * 0.001953125f;
  uint32_t b;
  std::memcpy(&b, &a, 4);
  b = (b + 0x7FFFFu + ((b >> 20) & 1u)) & ~0xFFFFFu;
  float nrm;
  std::memcpy(&nrm, &b, 4);
  const float r = a < 0.015625f ? sub : nrm;
  return std::copysign(r, v);
}

float q_int8(float v) { return round_even(std::min(127.0f, std::max(-127.0f, v))); }

double sgn(double v) { return static_cast<double>(int(v > 0.0) - int(v < 0.0)); }

struct Problem {
  const uint16_t *w;
  uint32_t M, N, fmt;
  double lambda, wl1, qmax;
  unsigned threads;
};

// F(S) and its straight-through gradient.  For row i with scale s and entry
// w: u = w / s in fp32 (one division, as the quantiser does), v = Q(u),
// w_hat = s * v.  The estimator takes dQ/du = 1 inside [-Qmax, Qmax] and 0
// where the clamp is active, so dv/ds = -w / s^2 there and dw_hat/ds =
// v + s dv/ds.  Rows that are all zero keep their scale (zero gradient).
double evaluate(const Problem &p, const double *s, double *grad, double *dist) {
  std::vector<double> d_row(p.M), r_row(p.M);
  float (*const quant)(float) = p.fmt == kFmtInt8 ? q_int8 : q_e4m3;
  const double inv_wl1 = p.wl1 > 0.0 ? 1.0 / p.wl1 : 0.0;
  const double inv_n = 1.0 / (static_cast<double>(p.M) * p.N);
  parallel_rows(p.M, p.threads, [&](uint32_t i) {
    const uint16_t *row = p.w + static_cast<uint64_t>(i) * p.N;
    const double si = s[i];
    const double inv_s2 = 1.0 / (si * si);
    const float sf = static_cast<float>(si);
    double d = 0.0, r = 0.0, gd = 0.0, gr = 0.0;
    for (uint32_t j = 0; j < p.N; ++j) {
      const float wf = bf16_value(row[j]);
      const float u = wf / sf;
      const double v = quant(u);
      const double diff = si * v - wf;
      d += std::fabs(diff);
      r += std::fabs(v);
      if (grad) {
        const double dv = (std::fabs(u) <= p.qmax) * (-static_cast<double>(wf) * inv_s2);
        gd += sgn(diff) * (v + si * dv);
        gr += sgn(v) * dv;
      }
    }
    d_row[i] = d;
    r_row[i] = r;
    if (grad) grad[i] = gd * inv_wl1 + p.lambda * gr * inv_n;
  });
  double d = 0.0, r = 0.0;
  for (uint32_t i = 0; i < p.M; ++i) {
    d += d_row[i];
    r += r_row[i];
  }
  if (dist) *dist = d * inv_wl1;
  return d * inv_wl1 + p.lambda * r * inv_n;
}

bool setup(const uint16_t *w, uint32_t M, uint32_t N, uint32_t fmt, double lambda,
           uint32_t threads, Problem &p, std::vector<double> *s0) {
  if (fmt == 0) fmt = kFmtE4M3;
  if (!w || !M || !N || (fmt != kFmtE4M3 && fmt != kFmtInt8) || !(lambda >= 0.0) ||
      static_cast<uint64_t>(M) * N >= (uint64_t(1) << 32))
    return false;
  p = Problem{w, M, N, fmt, lambda, 0.0, fmt == kFmtInt8 ? 127.0 : 448.0, workers(threads)};
  std::vector<double> amax(M), l1(M);
  parallel_rows(M, p.threads, [&](uint32_t i) {
    double a = 0.0, t = 0.0;
    for (uint32_t j = 0; j < N; ++j) {
      const double v = std::fabs(bf16_value(w[static_cast<uint64_t>(i) * N + j]));
      a = std::max(a, v);
      t += v;
    }
    amax[i] = a;
    l1[i] = t;
  });
  for (uint32_t i = 0; i < M; ++i) p.wl1 += l1[i];
  if (s0) {
    s0->resize(M);
    for (uint32_t i = 0; i < M; ++i) (*s0)[i] = amax[i] > 0.0 ? amax[i] / p.qmax : 1.0;
  }
  return true;
}

double dot(const std::vector<double> &a, const std::vector<double> &b) {
  double t = 0.0;
  for (size_t i = 0; i < a.size(); ++i) t += a[i] * b[i];
  return t;
}

// L-BFGS (Liu and Nocedal 1989) with a fixed step length: the search
// direction comes from the two-loop recursion over the last `history`
// curvature pairs (a pair is kept only if y.s > 1e-10), scaled by
// s.y / y.y of the newest pair; the first step is lr * min(1, 1/|g|_1)
// along -g.  Scales are kept at or above 1e-6 of their start.  Stops after
// `iters` steps, or when |g|_inf <= 1e-12 or F changes by less than 1e-10.
// The quantised objective is piecewise, so the iterate with the lowest F is
// returned.
double lbfgs(const Problem &p, std::vector<double> &x, uint32_t iters, uint32_t history,
             double lr) {
  const uint32_t M = p.M;
  const std::vector<double> floor_s = [&] {
    std::vector<double> f(x);
    for (auto &v : f) v *= 1e-6;
    return f;
  }();
  std::vector<double> g(M), gn(M), xn(M), q(M);
  double f = evaluate(p, x.data(), g.data(), nullptr);
  std::vector<double> best = x;
  double fbest = f;
  std::vector<std::vector<double>> S, Y;
  std::vector<double> rho;
  for (uint32_t it = 0; it < iters; ++it) {
    double ginf = 0.0, g1 = 0.0;
    for (double v : g) {
      ginf = std::max(ginf, std::fabs(v));
      g1 += std::fabs(v);
    }
    if (ginf <= 1e-12) break;
    q = g;
    const size_t k = S.size();
    std::vector<double> alpha(k);
    for (size_t a = k; a-- > 0;) {
      alpha[a] = rho[a] * dot(S[a], q);
      for (uint32_t i = 0; i < M; ++i) q[i] -= alpha[a] * Y[a][i];
    }
    const double gamma = k ? dot(S[k - 1], Y[k - 1]) / dot(Y[k - 1], Y[k - 1]) : 1.0;
    for (uint32_t i = 0; i < M; ++i) q[i] *= gamma;
    for (size_t a = 0; a < k; ++a) {
      const double b = rho[a] * dot(Y[a], q);
      for (uint32_t i = 0; i < M; ++i) q[i] += S[a][i] * (alpha[a] - b);
    }
    const double t = it == 0 ? lr * std::min(1.0, 1.0 / g1) : lr;
    for (uint32_t i = 0; i < M; ++i) xn[i] = std::max(x[i] - t * q[i], floor_s[i]);
    const double fn = evaluate(p, xn.data(), gn.data(), nullptr);
    std::vector<double> sk(M), yk(M);
    for (uint32_t i = 0; i < M; ++i) {
      sk[i] = xn[i] - x[i];
      yk[i] = gn[i] - g[i];
    }
    const double ys = dot(yk, sk);
    if (ys > 1e-10) {
      if (S.size() == history) {
        S.erase(S.begin());
        Y.erase(Y.begin());
        rho.erase(rho.begin());
      }
      S.push_back(std::move(sk));
      Y.push_back(std::move(yk));
      rho.push_back(1.0 / ys);
    }
    const bool flat = std::fabs(fn - f) < 1e-10;
    x.swap(xn);
    g.swap(gn);
    f = fn;
    if (f < fbest) {
      fbest = f;
      best = x;
    }
    if (flat) break;
  }
  x = best;
  return fbest;
}

// Nearest BF16 (ties to even) of a positive double.
uint16_t to_bf16(double v) {
  int e;
  const double m = std::frexp(v, &e);
  int shift = 8;
  if (e - 1 < -126) shift = 8 - (-126 - (e - 1));
  const float f = static_cast<float>(std::ldexp(std::nearbyint(std::ldexp(m, shift)), e - shift));
  uint32_t u;
  std::memcpy(&u, &f, 4);
  return static_cast<uint16_t>(u >> 16);
}

void defaults(const eqe_rd_params &in, uint32_t &iters, uint32_t &hist, double &lr) {
  iters = in.iters ? in.iters : 200;
  hist = in.history ? in.history : 20;
  lr = in.lr > 0.0 ? in.lr : (in.lambda > 30.0 ? 0.25 : 1.0);
}

}  // namespace

extern "C" double eqe_rd_objective(const uint16_t *w, uint32_t M, uint32_t N,
                                   uint32_t base_format, double lambda, const double *scale,
                                   uint32_t threads, double *grad, double *distortion) {
  Problem p;
  if (!scale || !setup(w, M, N, base_format, lambda, threads, p, nullptr)) return NAN;
  for (uint32_t i = 0; i < M; ++i)
    if (!(scale[i] > 0.0)) return NAN;
  return evaluate(p, scale, grad, distortion);
}

extern "C" int eqe_rd_scales(const uint16_t *w, uint32_t M, uint32_t N, const eqe_rd_params *prm,
                             double *scale_out, uint16_t *scale_bf16_out, double *objective_out) {
  Problem p;
  std::vector<double> x;
  if (!prm || !(prm->lambda >= 0.0) ||
      !setup(w, M, N, prm->base_format, prm->lambda, prm->threads, p, &x))
    return -1;
  uint32_t iters, hist;
  double lr;
  defaults(*prm, iters, hist, lr);
  try {
    const double f = lbfgs(p, x, iters, hist, lr);
    if (objective_out) *objective_out = f;
  } catch (const std::bad_alloc &) {
    return -5;
  }
  for (uint32_t i = 0; i < M; ++i) {
    if (scale_out) scale_out[i] = x[i];
    if (scale_bf16_out) scale_bf16_out[i] = to_bf16(x[i]);
  }
  return 0;
}
