// Host code under AddressSanitizer and UndefinedBehaviorSanitizer: the
// oracle (plain C) and the library's host parts (encoders, container
// validation, the scale optimiser) on small seeded matrices, on damaged
// containers (random byte flips and truncation) and on the RD optimiser.
// Built and run by tests/test_sanitize.py; any sanitizer report aborts the
// program with a non-zero status.  Compares only what the two sides must
// agree on: the oracle's decode of a product container against the codes the
// oracle's own quantiser gives for the container's scales.
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <vector>

#include "eq.h"
#include "eq_encode.h"
extern "C" {
#include "eq_oracle.h"
}

namespace {

uint64_t g_state = 0x9E3779B97F4A7C15ull;
uint64_t next_u64() {  // splitmix64
  uint64_t z = (g_state += 0x9E3779B97F4A7C15ull);
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}
double uniform01() { return (next_u64() >> 11) * (1.0 / 9007199254740992.0); }

// heavy-tailed values times a per-row scale, rounded to BF16 (truncation of
// the float bits is enough for test data)
std::vector<uint16_t> matrix(uint32_t M, uint32_t N) {
  std::vector<uint16_t> w(size_t(M) * N);
  for (uint32_t i = 0; i < M; ++i) {
    const double rs = std::exp(0.5 * (uniform01() - 0.5));
    for (uint32_t j = 0; j < N; ++j) {
      const double u1 = uniform01() + 1e-12, u2 = uniform01();
      double v = std::sqrt(-2.0 * std::log(u1)) * std::cos(6.283185307179586 * u2);
      if (uniform01() < 0.01) v *= 8.0;
      const float f = static_cast<float>(v * rs * 0.02);
      uint32_t b;
      std::memcpy(&b, &f, 4);
      w[size_t(i) * N + j] = static_cast<uint16_t>(b >> 16);
    }
  }
  return w;
}

int fails = 0;
#define CHECK(c)                                                        \
  do {                                                                  \
    if (!(c)) {                                                         \
      std::fprintf(stderr, "check failed: %s (line %d)\n", #c, __LINE__); \
      ++fails;                                                          \
    }                                                                   \
  } while (0)

// device pointers for eq_layer_init, which never dereferences them
alignas(256) uint8_t g_fake_dev[4096];

int layer_init(const std::vector<uint8_t> &blob, uint64_t bytes) {
  eq_layer L;
  void *dev = reinterpret_cast<void *>(
      (reinterpret_cast<uintptr_t>(g_fake_dev) + 255) / 256 * 256);
  return eq_layer_init(&L, blob.data(), bytes, dev, dev, reinterpret_cast<int32_t *>(dev));
}

// Oracle decode of a container against the oracle's quantiser at the
// container's scales.
void check_roundtrip(const std::vector<uint8_t> &blob, const std::vector<uint16_t> &w,
                     uint32_t M, uint32_t N, uint32_t fmt, bool v2) {
  std::vector<uint8_t> q(size_t(M) * N), q_ref(size_t(M) * N);
  std::vector<uint16_t> scale(M);
  uint64_t off_scale;
  if (v2) {
    or_info2 info;
    CHECK(or_container2_info(blob.data(), blob.size(), &info) == 0);
    off_scale = info.off_scale;
    CHECK(or_container2_decode(blob.data(), blob.size(), q.data()) == 0);
  } else {
    or_info info;
    CHECK(or_container_info(blob.data(), blob.size(), &info) == 0);
    off_scale = info.off_scale;
    CHECK(or_container_decode(blob.data(), blob.size(), q.data()) == 0);
  }
  std::memcpy(scale.data(), blob.data() + off_scale, 2 * size_t(M));
  or_quantize(w.data(), M, N, scale.data(), fmt, q_ref.data());
  CHECK(std::memcmp(q.data(), q_ref.data(), q.size()) == 0);
  CHECK(layer_init(blob, blob.size()) == EQ_OK);
}

// Damaged copies: the validators return an error or accept; the decoders
// return OK or an error; nothing reads or writes out of bounds.
void fuzz(const std::vector<uint8_t> &blob, uint32_t M, uint32_t N, bool v2, int trials) {
  std::vector<uint8_t> q(size_t(M) * N + 64);
  for (int t = 0; t < trials; ++t) {
    std::vector<uint8_t> bad = blob;
    const int flips = 1 + static_cast<int>(next_u64() % 4);
    for (int f = 0; f < flips; ++f) {
      // half of the flips in the header and section tables
      const uint64_t span = (next_u64() & 1) ? std::min<uint64_t>(bad.size(), 256) : bad.size();
      bad[next_u64() % span] ^= static_cast<uint8_t>(1u << (next_u64() % 8));
    }
    uint64_t bytes = bad.size();
    if (t % 7 == 0) bytes = next_u64() % bad.size();  // truncated
    (void)layer_init(bad, bytes);
    if (v2) {
      or_info2 info;
      if (or_container2_info(bad.data(), bytes, &info) == 0 &&
          uint64_t(info.rows) * info.cols <= uint64_t(M) * N)
        (void)or_container2_decode(bad.data(), bytes, q.data());
    } else {
      or_info info;
      if (or_container_info(bad.data(), bytes, &info) == 0 &&
          uint64_t(info.rows) * info.cols <= uint64_t(M) * N)
        (void)or_container_decode(bad.data(), bytes, q.data());
    }
  }
}

std::vector<uint8_t> take(uint8_t *p, uint64_t n, bool oracle_owned) {
  std::vector<uint8_t> v(p, p + n);
  if (oracle_owned) or_free(p);
  else eqe_free(p);
  return v;
}

}  // namespace

int main() {
  const uint32_t shapes[][2] = {{37, 1283}, {130, 512}, {300, 1000}, {5, 4}};
  for (const auto &s : shapes) {
    const uint32_t M = s[0], N = s[1];
    const std::vector<uint16_t> w = matrix(M, N);
    for (uint32_t fmt = 1; fmt <= 2; ++fmt) {
      double h = 0;
      const float alpha = eqe_alpha_search(w.data(), M, N, 2.5, 0, 2, fmt, &h);
      CHECK(alpha > 0 && std::isfinite(h));
      // version 1, product encoder and oracle encoder
      eqe_params p{12, 1024, 64, 2, 7, 2.5f, fmt};
      uint8_t *raw = nullptr;
      uint64_t n = 0;
      CHECK(eqe_encode(w.data(), M, N, alpha, &p, &raw, &n) == EQ_OK);
      const std::vector<uint8_t> b1 = take(raw, n, false);
      check_roundtrip(b1, w, M, N, fmt, false);
      CHECK(or_container_build(w.data(), M, N, alpha, fmt, 11, 512, 64, 7, 2.5f, &raw, &n) == 0);
      const std::vector<uint8_t> o1 = take(raw, n, true);
      check_roundtrip(o1, w, M, N, fmt, false);
      // version 2 at two tile shapes, in matrix order and with a row order
      for (const uint32_t tr : {64u, 256u})
        for (const uint32_t ro : {0u, 1u}) {
          eqe_params2 p2{12, tr, tr == 64 ? 64u : 32u, 2, 7, 2.5f, fmt, ro};
          CHECK(eqe_encode2(w.data(), M, N, alpha, nullptr, &p2, &raw, &n) == EQ_OK);
          const std::vector<uint8_t> b2 = take(raw, n, false);
          check_roundtrip(b2, w, M, N, fmt, true);
          fuzz(b2, M, N, true, 150);
        }
      for (const uint32_t ro : {0u, 1u}) {
        CHECK(or_container2_build(w.data(), M, N, alpha, nullptr, fmt, 11, 128, 16, ro, 7, 2.5f,
                                  &raw, &n) == 0);
        const std::vector<uint8_t> o2 = take(raw, n, true);
        check_roundtrip(o2, w, M, N, fmt, true);
      }
      fuzz(b1, M, N, false, 150);
      fuzz(o1, M, N, false, 50);
    }
    // the l1 rate-distortion scale optimisation, product and oracle
    if (M * N <= 200000) {
      eqe_rd_params rp{0.5, 0.0, 15, 5, 2, 1};
      std::vector<double> sc(M);
      std::vector<uint16_t> sb(M);
      double obj = 0;
      CHECK(eqe_rd_scales(w.data(), M, N, &rp, sc.data(), sb.data(), &obj) == EQ_OK);
      CHECK(std::isfinite(obj));
      eqe_params p{12, 1024, 64, 2, 7, 0.0f, 1};
      uint8_t *raw = nullptr;
      uint64_t n = 0;
      CHECK(eqe_encode_scaled(w.data(), M, N, sb.data(), &p, &raw, &n) == EQ_OK);
      const std::vector<uint8_t> b = take(raw, n, false);
      check_roundtrip(b, w, M, N, 1, false);
      std::vector<double> so(M);
      double oo = 0;
      CHECK(or_rd_scales(w.data(), M, N, 1, 0.5, 15, 5, 1.0, so.data(), &oo) == 0);
      CHECK(std::isfinite(oo));
    }
    // the oracle's GEMV on decoded weights
    std::vector<uint16_t> x(2 * size_t(N), 0x3F80), bias(M, 0x3F80);
    std::vector<double> y(2 * size_t(M));
    or_gemv(w.data(), M, N, x.data(), 2, bias.data(), y.data());
    for (double v : y) CHECK(std::isfinite(v));
  }
  if (fails) {
    std::fprintf(stderr, "%d checks failed\n", fails);
    return 1;
  }
  std::printf("sanitized host run ok\n");
  return 0;
}
