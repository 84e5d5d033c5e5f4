// Host side of libeq: container validation (eq_layer_init), error strings.
// The container layout and the checks are documented in eq.h.
#include <cmath>
#include <cstring>
#include <vector>

#include "eq.h"
#include "eq_internal.h"

namespace {

template <class T>
T rd(const uint8_t *b, uint64_t off) {
  T v;
  std::memcpy(&v, b + off, sizeof v);  // little-endian host
  return v;
}

bool section_ok(uint64_t off, uint64_t len, uint64_t file_bytes) {
  return off % 256 == 0 && off >= 256 && off <= file_bytes && len <= file_bytes - off;
}

// BF16 scale usable by the dequantiser: finite, normal, 2^-117 <= |s| < 2^120,
// so s * v(q) is an exact, normal fp32 product for every E4M3 value and every
// Int8 value v(q).
bool scale_ok(uint16_t s) {
  const int e = (s >> 7) & 0xFF;
  return e >= 127 - 117 && e <= 127 + 119;
}

// A code valid in the base format: E4M3FN never NaN, Int8 never -128.
bool code_ok(uint32_t fmt, uint8_t c) {
  return fmt == eq_detail::kFmtE4M3 ? (c & 0x7F) != 0x7F : c != 0x80;
}

// Version 2: tile-ordered chunks and the phrase alphabet (layout in eq.h).
int init_v2(eq_layer *L, const uint8_t *b, uint64_t bytes, const uint8_t *d) {
  const uint32_t fmt = rd<uint32_t>(b, 12);
  const uint32_t M = rd<uint32_t>(b, 16), N = rd<uint32_t>(b, 20), C = rd<uint32_t>(b, 24);
  const uint32_t n_chunks = rd<uint32_t>(b, 28), TR = rd<uint32_t>(b, 32);
  const uint32_t R = rd<uint32_t>(b, 36), K = rd<uint32_t>(b, 40), TC = rd<uint32_t>(b, 84);
  const uint32_t nq = rd<uint32_t>(b, 144), np = rd<uint32_t>(b, 148), ns = rd<uint32_t>(b, 152);
  const uint64_t total = rd<uint64_t>(b, 48), padded = rd<uint64_t>(b, 56);
  const uint64_t o_scale = rd<uint64_t>(b, 88), o_phr = rd<uint64_t>(b, 96);
  const uint64_t o_freq = rd<uint64_t>(b, 104), o_off = rd<uint64_t>(b, 112);
  const uint64_t o_state = rd<uint64_t>(b, 120), o_words = rd<uint64_t>(b, 128);
  const uint64_t file_bytes = rd<uint64_t>(b, 136);
  const uint64_t n = static_cast<uint64_t>(M) * N;
  if (file_bytes > bytes || n == 0 || n >= (uint64_t(1) << 32)) return EQ_EFORMAT;
  if ((TR != 64 && TR != 128 && TR != 256) || TC == 0 || TC % 4 ||
      uint64_t(TR) * TC != C || R < 10 || R > 12)
    return EQ_EFORMAT;
  if (uint64_t(n_chunks) != uint64_t((M + TR - 1) / TR) * ((N + TC - 1) / TC)) return EQ_EFORMAT;
  if (K < 1 || K > (1u << R) || uint64_t(nq) + np + ns != K || ns > 256) return EQ_EFORMAT;
  if (padded < total + 1024 || padded % 128 != 0 || padded + C >= (uint64_t(1) << 32))
    return EQ_EFORMAT;
  if (!section_ok(o_scale, 2ull * M, file_bytes) || !section_ok(o_phr, 4ull * K, file_bytes) ||
      !section_ok(o_freq, 2ull * K, file_bytes) ||
      !section_ok(o_off, 4ull * (n_chunks + 1), file_bytes) ||
      !section_ok(o_state, 4ull * n_chunks * TR, file_bytes) ||
      !section_ok(o_words, 2 * padded, file_bytes))
    return EQ_EFORMAT;
  // phrases: valid codes, unused bytes zero, each part strictly ascending
  uint32_t fsum = 0;
  for (uint32_t k = 0; k < K; ++k) {
    const uint32_t len = k < nq ? 4 : (k < nq + np ? 2 : 1);
    const uint32_t v = rd<uint32_t>(b, o_phr + 4ull * k);
    for (uint32_t e = 0; e < 4; ++e) {
      const uint8_t c = static_cast<uint8_t>(v >> (8 * e));
      if (e < len ? !code_ok(fmt, c) : c != 0) return EQ_EFORMAT;
    }
    const bool part_start = k == 0 || k == nq || k == nq + np;
    if (!part_start && v <= rd<uint32_t>(b, o_phr + 4ull * (k - 1))) return EQ_EFORMAT;
    const uint16_t f = rd<uint16_t>(b, o_freq + 2ull * k);
    if (f == 0) return EQ_EFORMAT;
    fsum += f;
  }
  if (fsum != (1u << R)) return EQ_EFORMAT;
  uint32_t prev = 0;
  for (uint32_t c = 0; c <= n_chunks; ++c) {
    const uint32_t o = rd<uint32_t>(b, o_off + 4ull * c);
    if ((c == 0 && o != 0) || o < prev) return EQ_EFORMAT;
    prev = o;
  }
  if (prev != total) return EQ_EFORMAT;
  for (uint64_t s = 0; s < static_cast<uint64_t>(n_chunks) * TR; ++s)
    if (rd<uint32_t>(b, o_state + 4 * s) < (1u << 16)) return EQ_EFORMAT;
  for (uint32_t i = 0; i < M; ++i)
    if (!scale_ok(rd<uint16_t>(b, o_scale + 2ull * i))) return EQ_EFORMAT;
  // row order (flag bit 0): a permutation of the M rows
  const uint32_t flags = rd<uint32_t>(b, 44);
  const uint64_t o_order = rd<uint64_t>(b, 160);
  if (flags & ~1u) return EQ_EFORMAT;
  if (flags & 1u) {
    if (!section_ok(o_order, 4ull * M, file_bytes)) return EQ_EFORMAT;
    std::vector<uint8_t> seen(M, 0);
    for (uint32_t k = 0; k < M; ++k) {
      const uint32_t r = rd<uint32_t>(b, o_order + 4ull * k);
      if (r >= M || seen[r]) return EQ_EFORMAT;
      seen[r] = 1;
    }
  } else if (o_order != 0) {
    return EQ_EFORMAT;
  }
  L->rows = M;
  L->cols = N;
  L->chunk_syms = C;
  L->n_chunks = n_chunks;
  L->lanes = TR;
  L->prob_bits = R;
  L->n_syms = K;
  L->base_format = fmt;
  L->total_words = total;
  L->padded_words = padded;
  L->scale = reinterpret_cast<const uint16_t *>(d + o_scale);
  L->sym = d + o_phr;
  L->freq = reinterpret_cast<const uint16_t *>(d + o_freq);
  L->chunk_off = reinterpret_cast<const uint32_t *>(d + o_off);
  L->chunk_state = reinterpret_cast<const uint32_t *>(d + o_state);
  L->words = reinterpret_cast<const uint16_t *>(d + o_words);
  L->version = 2;
  L->tile_cols = TC;
  L->n_quads = nq;
  L->n_pairs = np;
  L->n_singles = ns;
  L->row_order = (flags & 1u) ? reinterpret_cast<const uint32_t *>(d + o_order) : nullptr;
  return EQ_OK;
}

}  // namespace

extern "C" size_t eq_lut_bytes(void) { return eq_detail::kLutBytes; }

extern "C" int eq_layer_init(eq_layer *L, const void *host_blob, uint64_t bytes,
                             const void *dev_blob, void *dev_lut, int32_t *dev_status) {
  if (!L || !host_blob || !dev_blob || !dev_lut || !dev_status) return EQ_EINVAL;
  // sections are 256-byte aligned within the blob; the kernels read them with
  // dword (and wider) loads
  if ((reinterpret_cast<uintptr_t>(dev_blob) | reinterpret_cast<uintptr_t>(dev_lut)) & 255)
    return EQ_EINVAL;
  const uint8_t *b = static_cast<const uint8_t *>(host_blob);
  if (bytes < 256 || std::memcmp(b, "EQC1", 4) != 0) return EQ_EFORMAT;
  const uint32_t fmt = rd<uint32_t>(b, 12), version = rd<uint32_t>(b, 4);
  if ((version != 1 && version != 2) || rd<uint32_t>(b, 8) != 256 ||
      (fmt != eq_detail::kFmtE4M3 && fmt != eq_detail::kFmtInt8))
    return EQ_EFORMAT;
  if (version == 2) {
    eq_layer v;
    std::memset(&v, 0, sizeof v);
    const int rc = init_v2(&v, b, bytes, static_cast<const uint8_t *>(dev_blob));
    if (rc != EQ_OK) return rc;
    v.lut = static_cast<uint32_t *>(dev_lut);
    v.status = dev_status;
    *L = v;
    return EQ_OK;
  }
  const uint32_t M = rd<uint32_t>(b, 16), N = rd<uint32_t>(b, 20), C = rd<uint32_t>(b, 24);
  const uint32_t n_chunks = rd<uint32_t>(b, 28), W = rd<uint32_t>(b, 32);
  const uint32_t P = rd<uint32_t>(b, 36), K = rd<uint32_t>(b, 40);
  const uint64_t total = rd<uint64_t>(b, 48), padded = rd<uint64_t>(b, 56);
  const uint64_t o_scale = rd<uint64_t>(b, 88), o_sym = rd<uint64_t>(b, 96);
  const uint64_t o_freq = rd<uint64_t>(b, 104), o_off = rd<uint64_t>(b, 112);
  const uint64_t o_state = rd<uint64_t>(b, 120), o_words = rd<uint64_t>(b, 128);
  const uint64_t file_bytes = rd<uint64_t>(b, 136);
  const uint64_t n = static_cast<uint64_t>(M) * N;
  if (file_bytes > bytes || n == 0 || n >= (uint64_t(1) << 32)) return EQ_EFORMAT;
  if ((W != 64 && W != 128 && W != 256) || C == 0 || C % W != 0) return EQ_EFORMAT;
  if (n_chunks != (n + C - 1) / C || P < eq_detail::kMinProbBits || P > 12 || K < 1 || K > 256 ||
      K > (1u << P))
    return EQ_EFORMAT;
  // word indices (including a chunk's worth of overrun on a corrupt stream)
  // stay below 2^32
  if (padded < total + 1024 || padded % 128 != 0 || padded + C >= (uint64_t(1) << 32))
    return EQ_EFORMAT;
  if (!section_ok(o_scale, 2ull * M, file_bytes) || !section_ok(o_sym, K, file_bytes) ||
      !section_ok(o_freq, 2ull * K, file_bytes) ||
      !section_ok(o_off, 4ull * (n_chunks + 1), file_bytes) ||
      !section_ok(o_state, 4ull * n_chunks * W, file_bytes) ||
      !section_ok(o_words, 2 * padded, file_bytes))
    return EQ_EFORMAT;

  uint32_t fsum = 0;
  for (uint32_t k = 0; k < K; ++k) {
    const uint8_t s = b[o_sym + k];
    if (fmt == eq_detail::kFmtE4M3 ? (s & 0x7F) == 0x7F : s == 0x80)
      return EQ_EFORMAT;                                // E4M3 NaN / Int8 -128
    if (k && s <= b[o_sym + k - 1]) return EQ_EFORMAT;  // strictly ascending
    const uint16_t f = rd<uint16_t>(b, o_freq + 2ull * k);
    if (f == 0) return EQ_EFORMAT;
    fsum += f;
  }
  if (fsum != (1u << P)) return EQ_EFORMAT;
  uint32_t prev = 0;
  for (uint32_t c = 0; c <= n_chunks; ++c) {
    const uint32_t o = rd<uint32_t>(b, o_off + 4ull * c);
    if ((c == 0 && o != 0) || o < prev) return EQ_EFORMAT;
    prev = o;
  }
  if (prev != total) return EQ_EFORMAT;
  for (uint64_t s = 0; s < static_cast<uint64_t>(n_chunks) * W; ++s)
    if (rd<uint32_t>(b, o_state + 4 * s) < (1u << 16)) return EQ_EFORMAT;
  for (uint32_t i = 0; i < M; ++i)
    if (!scale_ok(rd<uint16_t>(b, o_scale + 2ull * i))) return EQ_EFORMAT;

  const uint8_t *d = static_cast<const uint8_t *>(dev_blob);
  eq_layer v;
  std::memset(&v, 0, sizeof v);
  v.rows = M;
  v.cols = N;
  v.chunk_syms = C;
  v.n_chunks = n_chunks;
  v.lanes = W;
  v.prob_bits = P;
  v.n_syms = K;
  v.base_format = fmt;
  v.total_words = total;
  v.padded_words = padded;
  v.scale = reinterpret_cast<const uint16_t *>(d + o_scale);
  v.sym = d + o_sym;
  v.freq = reinterpret_cast<const uint16_t *>(d + o_freq);
  v.chunk_off = reinterpret_cast<const uint32_t *>(d + o_off);
  v.chunk_state = reinterpret_cast<const uint32_t *>(d + o_state);
  v.words = reinterpret_cast<const uint16_t *>(d + o_words);
  v.lut = static_cast<uint32_t *>(dev_lut);
  v.status = dev_status;
  v.version = 1;
  *L = v;
  return EQ_OK;
}

extern "C" const char *eq_strerror(int code) {
  switch (code) {
    case EQ_OK: return "ok";
    case EQ_EINVAL: return "invalid argument (null pointer, size or range)";
    case EQ_EFORMAT: return "container header or sections inconsistent";
    case EQ_EHIP: return "HIP launch or runtime call failed";
    case EQ_ECORRUPT: return "entropy-coded stream failed its end-of-chunk check";
    case EQ_ESCRATCH: return "workspace needed exceeds the static scratch (EQ_NOALLOC_SCRATCH_BYTES)";
    default: return "unknown error code";
  }
}
