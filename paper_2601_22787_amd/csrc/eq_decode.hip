// gfx950 kernels and C-ABI launchers of libeq (declared in include/eq.h).
//
// Alg. 2 of the paper: ANS decoding of the per-layer bitstream, view as the
// row-major weight matrix, and the product with the per-row-scaled weights
// (Sec. 2.1 dequantiser and linear layer).  One wavefront owns one chunk:
// each of its 64 lanes holds W/64 interleaved coder states, the slot and
// value tables sit in LDS, and the stream words of a step are handed out
// with a wavefront ballot and a masked bit count, which reproduces the
// coder's ascending-lane read order exactly.
#include <hip/hip_runtime.h>

#include <atomic>
#include <type_traits>

#include "eq.h"
#include "eq_internal.h"

namespace {

using namespace eq_detail;

constexpr int kWave = 64;
constexpr int kBlock = 512;              // 8 wavefronts, one chunk each
constexpr int kWavesPerBlock = kBlock / kWave;
constexpr int kMaxBatch = 8;
constexpr uint32_t kHalf = 512;          // stream words per window half (1 KiB)
constexpr uint32_t kWin = 2 * kHalf;     // per-wave LDS window of stream words

enum Mode { kCodes = 0, kBf16 = 1, kGemv = 2 };

struct Args {
  const uint32_t *lut;          // slot table (2 x u32 per slot), then E4M3 value table
  const uint16_t *scale;
  const uint32_t *chunk_off;
  const uint32_t *chunk_state;
  const uint16_t *words;
  int32_t *status;
  uint32_t rows, cols, chunk_syms, n_chunks, lanes, prob_bits;
  uint32_t padded_words;
  uint32_t n;                   // rows * cols (< 2^32)
  uint8_t *codes;
  uint16_t *wout;
  const uint16_t *x;
  uint32_t batch;
  const uint16_t *bias;
  float *y;
  float *ws;
};

__device__ inline float bf16_to_f32(uint16_t b) { return __uint_as_float(uint32_t(b) << 16); }

// Round a finite fp32 value to nearest-even BF16.
__device__ inline uint16_t f32_to_bf16(float f) {
  const uint32_t u = __float_as_uint(f);
  return static_cast<uint16_t>((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
}

// E4M3FN value of a code: sign | exponent (bias 7) | 3-bit mantissa;
// exponent 0 is subnormal (m * 2^-9).
__device__ inline float e4m3_value(uint32_t c) {
  const uint32_t e = (c >> 3) & 15u, m = c & 7u;
  float mag;
  if (e == 0) mag = static_cast<float>(m) * 0.001953125f;  // 2^-9, exact
  else mag = __uint_as_float(((e + 120u) << 23) | (m << 20));
  if ((c & 0x7Fu) == 0x7Fu) mag = __uint_as_float(0x7FC00000u);
  return (c & 0x80u) ? -mag : mag;
}

__device__ inline float wave_sum(float v) {
#pragma unroll
  for (int o = kWave / 2; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

__device__ inline uint32_t uniform(uint32_t v) { return __builtin_amdgcn_readfirstlane(v); }

// 16 stream words starting at word index i (a multiple of 8), clamped to the
// padded section so that a read ahead never leaves the container.
__device__ inline uint4 load_words(const uint16_t *words, uint32_t i, uint32_t last8) {
  return *reinterpret_cast<const uint4 *>(words + min(i, last8));
}

// Decode tables.  Slot s of symbol k (cum_k <= s < cum_k + f_k):
//   lut[2s]   = f_k | code_k << 24     (low 24 bits feed a 24-bit multiply-add)
//   lut[2s+1] = s - cum_k
// then lut[2 * kMaxSlots + c] = bits of the E4M3 value of code c.
__global__ void prepare_kernel(const uint8_t *sym, const uint16_t *freq, uint32_t K,
                               uint32_t *lut, int32_t *status) {
  const uint32_t t = threadIdx.x;
  if (t < K) {
    uint32_t cum = 0;
    for (uint32_t k = 0; k < t; ++k) cum += freq[k];
    const uint32_t f = freq[t];
    for (uint32_t s = 0; s < f; ++s) {
      lut[2 * (cum + s)] = f | (uint32_t(sym[t]) << 24);
      lut[2 * (cum + s) + 1] = s;
    }
  }
  lut[2 * kMaxSlots + t] = __float_as_uint(e4m3_value(t));
  if (t == 0) *status = 0;
}

// One wavefront decodes one chunk.  G = W / 64 coder states per lane (state
// g * 64 + lane); MODE selects what is done with each decoded symbol;
// UNIFORM means every step of W symbols lies inside one matrix row (N is a
// multiple of W); XLDS means the activations are staged in LDS.
template <int G, int MODE, bool UNIFORM, bool XLDS>
__global__ __launch_bounds__(kBlock) void decode_kernel(Args a) {
  extern __shared__ uint16_t x_s[];  // [batch][cols] BF16 when XLDS
  __shared__ uint2 slot_s[kMaxSlots];
  __shared__ float val_s[256];
  __shared__ uint4 win_s[kWavesPerBlock][kWin / 8];
  const uint32_t nslots = 1u << a.prob_bits;
  const uint32_t N = a.cols;
  {
    const uint2 *src = reinterpret_cast<const uint2 *>(a.lut);
    for (uint32_t i = threadIdx.x; i < nslots; i += kBlock) slot_s[i] = src[i];
    if (threadIdx.x < 256) val_s[threadIdx.x] = __uint_as_float(a.lut[2 * kMaxSlots + threadIdx.x]);
    if (XLDS) {
      const uint32_t nx = a.batch * N;
      for (uint32_t i = threadIdx.x; i < nx; i += kBlock) x_s[i] = a.x[i];
    }
  }
  __syncthreads();

  const uint32_t lane = threadIdx.x & (kWave - 1);
  const uint32_t wave = uniform(threadIdx.x / kWave);
  const uint32_t c = uniform(blockIdx.x * kWavesPerBlock + wave);
  if (c >= a.n_chunks) return;

  constexpr uint32_t W = G * kWave;
  const uint32_t k0 = c * a.chunk_syms;
  const uint32_t nc = min(a.chunk_syms, a.n - k0);
  const uint32_t mask = nslots - 1;
  const uint32_t P = a.prob_bits;
  const uint32_t last8 = a.padded_words - 8;

  uint32_t x[G];
#pragma unroll
  for (int g = 0; g < G; ++g) x[g] = a.chunk_state[c * W + g * kWave + lane];
  uint32_t p = a.chunk_off[c];
  const uint32_t p_end = a.chunk_off[c + 1];

  // Stream words [wb, wb + kWin) live in this wave's LDS window and the next
  // half is in flight in registers.  A step reads at most W words and the
  // window slides by a half whenever p passes its middle, so every word a
  // step can read is in LDS.
  const uint16_t *win = reinterpret_cast<const uint16_t *>(win_s[wave]);
  uint32_t wb = p & ~7u;
  {
    const uint4 h0 = load_words(a.words, wb + 8 * lane, last8);
    const uint4 h1 = load_words(a.words, wb + kHalf + 8 * lane, last8);
    win_s[wave][lane] = h0;
    win_s[wave][kHalf / 8 + lane] = h1;
  }
  __builtin_amdgcn_s_waitcnt(0);  // states, offsets and window are in
  uint4 next = load_words(a.words, wb + kWin + 8 * lane, last8);

  // uniform-row bookkeeping (every step lies inside one row)
  uint32_t row = k0 / N;
  const uint32_t first_row = row;
  uint32_t row_end = (row + 1) * N;  // <= n < 2^32
  float srow = 0.0f;
  if (MODE == kBf16 && UNIFORM) srow = bf16_to_f32(a.scale[row]);
  // per-state row/column (general shapes)
  uint32_t prow[G], pcol[G];
  if (!UNIFORM) {
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const uint32_t pos = k0 + g * kWave + lane;
      prow[g] = pos / N;
      pcol[g] = pos - prow[g] * N;
    }
  }
  float acc[UNIFORM ? 1 : G][kMaxBatch];
#pragma unroll
  for (int g = 0; g < (UNIFORM ? 1 : G); ++g)
#pragma unroll
    for (int b = 0; b < kMaxBatch; ++b) acc[g][b] = 0.0f;
  bool pending[G];
#pragma unroll
  for (int g = 0; g < G; ++g) pending[g] = false;

  auto xval = [&](uint32_t b, uint32_t col) -> float {
    return bf16_to_f32(XLDS ? x_s[b * N + col] : a.x[b * N + col]);
  };

  auto flush_uniform = [&](uint32_t r) {
    const bool owned = r * N >= k0 && (r + 1) * N <= k0 + nc;
    const float s = bf16_to_f32(a.scale[r]);
    const float bb = a.bias ? bf16_to_f32(a.bias[r]) : 0.0f;
#pragma unroll
    for (int b = 0; b < kMaxBatch; ++b) {
      if (b < (int)a.batch) {
        const float sum = wave_sum(acc[0][b]);
        if (lane == 0) {
          if (owned) a.y[b * a.rows + r] = s * sum + bb;
          else a.ws[(2 * c + (r == first_row ? 0 : 1)) * a.batch + b] = sum;
        }
      }
      acc[0][b] = 0.0f;
    }
  };

  // One step: W symbols at chunk offset t * W.  TAIL: the last, partial step.
  auto step = [&](auto tail_tag, uint32_t t) {
    constexpr bool TAIL = decltype(tail_tag)::value;
    if (p - wb >= kHalf) {  // slide the window by one half
      const uint4 keep = win_s[wave][kHalf / 8 + lane];
      win_s[wave][lane] = keep;
      win_s[wave][kHalf / 8 + lane] = next;
      wb += kHalf;
      next = load_words(a.words, wb + kWin + 8 * lane, last8);
    }
    const uint32_t kk = t * W;  // offset of this step inside the chunk
    if (UNIFORM && MODE != kCodes && k0 + kk >= row_end) {
      if (MODE == kGemv) flush_uniform(row);
      ++row;
      row_end += N;
      if (MODE == kBf16) srow = bf16_to_f32(a.scale[row]);
    }
    // decode every active state of the step
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const uint32_t pos = kk + g * kWave + lane;
      if (!TAIL || pos < nc) {
        const uint2 e = slot_s[x[g] & mask];
        x[g] = __umul24(e.x, x[g] >> P) + e.y;
        if (MODE == kCodes) {
          uint8_t *out = a.codes + (k0 + kk + g * kWave);
          out[lane] = static_cast<uint8_t>(e.x >> 24);
        } else if (MODE == kBf16) {
          const float s = UNIFORM ? srow : bf16_to_f32(a.scale[prow[g]]);
          uint16_t *out = a.wout + (k0 + kk + g * kWave);
          out[lane] = f32_to_bf16(s * val_s[e.x >> 24]);
        } else {
          const float v = val_s[e.x >> 24];
          const uint32_t col = UNIFORM ? (k0 + kk + N - row_end) + g * kWave + lane : pcol[g];
#pragma unroll
          for (int b = 0; b < kMaxBatch; ++b)
            if (b < (int)a.batch) acc[UNIFORM ? 0 : g][b] += v * xval(b, col);
          if (!UNIFORM) pending[g] = true;
        }
      }
      if (!UNIFORM && MODE != kCodes) {
        // advance this state's position by one step (W symbols)
        pcol[g] += W;
        if (pcol[g] >= N) {
          if (MODE == kGemv && pending[g]) {
#pragma unroll
            for (int b = 0; b < kMaxBatch; ++b) {
              if (b < (int)a.batch) atomicAdd(&a.ws[b * a.rows + prow[g]], acc[g][b]);
              acc[g][b] = 0.0f;
            }
            pending[g] = false;
          }
          prow[g] += pcol[g] / N;
          pcol[g] %= N;
        }
      }
    }
    // renormalise in ascending state order: state g*64 + lane
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const bool need = (!TAIL || kk + g * kWave + lane < nc) && x[g] < kStateLow;
      const uint64_t m = __builtin_amdgcn_ballot_w64(need);
      const uint32_t below = __builtin_amdgcn_mbcnt_hi(uint32_t(m >> 32),
                                                       __builtin_amdgcn_mbcnt_lo(uint32_t(m), 0u));
      const uint16_t *wp = win + (p - wb);
      if (need) x[g] = (x[g] << 16) | wp[below];
      p += static_cast<uint32_t>(__popcll(m));
    }
  };

  const uint32_t full = nc / W;
  for (uint32_t t = 0; t < full; ++t) step(std::false_type{}, t);
  if (nc % W) step(std::true_type{}, full);

  if (MODE == kGemv) {
    if (UNIFORM) {
      flush_uniform(row);
    } else {
#pragma unroll
      for (int g = 0; g < G; ++g)
        if (pending[g])
#pragma unroll
          for (int b = 0; b < kMaxBatch; ++b)
            if (b < (int)a.batch) atomicAdd(&a.ws[b * a.rows + prow[g]], acc[g][b]);
    }
  }

  // end-of-chunk check: every state back at 2^16, stream used up exactly
  bool bad = p != p_end;
#pragma unroll
  for (int g = 0; g < G; ++g) bad |= x[g] != kStateLow;
  if (__builtin_amdgcn_ballot_w64(bad) != 0 && lane == 0) atomicOr(a.status, 1);
}

// Rows split between chunks (whole-row steps): y = s * (sum of the chunks'
// partial sums, in chunk order) + bias.  One thread per chunk boundary; the
// first boundary inside a row does the merge.
__global__ void merge_rows_kernel(Args a) {
  const uint32_t c = blockIdx.x * blockDim.x + threadIdx.x + 1;
  if (c >= a.n_chunks) return;
  const uint32_t N = a.cols, C = a.chunk_syms;
  const uint32_t kb = c * C;
  if (kb % N == 0) return;
  const uint32_t r = kb / N;
  const uint32_t c_first = (r * N) / C;
  if (c - 1 != c_first) return;
  const uint32_t c_last = min((r + 1) * N - 1, a.n - 1) / C;
  const float s = bf16_to_f32(a.scale[r]);
  const float bb = a.bias ? bf16_to_f32(a.bias[r]) : 0.0f;
  for (uint32_t b = 0; b < a.batch; ++b) {
    float sum = 0.0f;
    for (uint32_t cc = c_first; cc <= c_last; ++cc) {
      const uint32_t slot = ((cc * C) / N == r) ? 0u : 1u;
      sum += a.ws[(2 * cc + slot) * a.batch + b];
    }
    a.y[b * a.rows + r] = s * sum + bb;
  }
}

__global__ void fill_zero_kernel(float *p, uint32_t n) {
  const uint32_t i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = 0.0f;
}

// General shapes: y = s * (atomically accumulated row sums) + bias.
__global__ void finalize_rows_kernel(Args a) {
  const uint32_t i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= a.rows * a.batch) return;
  const uint32_t r = i % a.rows;
  const float bb = a.bias ? bf16_to_f32(a.bias[r]) : 0.0f;
  a.y[i] = bf16_to_f32(a.scale[r]) * a.ws[i] + bb;
}

Args make_args(const eq_layer *L) {
  Args a{};
  a.lut = L->lut;
  a.scale = L->scale;
  a.chunk_off = L->chunk_off;
  a.chunk_state = L->chunk_state;
  a.words = L->words;
  a.status = L->status;
  a.rows = L->rows;
  a.cols = L->cols;
  a.chunk_syms = L->chunk_syms;
  a.n_chunks = L->n_chunks;
  a.lanes = L->lanes;
  a.prob_bits = L->prob_bits;
  a.padded_words = static_cast<uint32_t>(L->padded_words);
  a.n = L->rows * L->cols;
  return a;
}

bool layer_ok(const eq_layer *L) {
  return L && L->lut && L->status && L->words && L->chunk_off && L->chunk_state && L->scale &&
         (L->lanes == 64 || L->lanes == 128 || L->lanes == 256) && L->prob_bits >= 8 &&
         L->prob_bits <= 12 && L->n_chunks > 0 && L->cols > 0 && L->rows > 0;
}

constexpr uint32_t kMaxXLdsBytes = 64 * 1024;
constexpr size_t kStaticLds =
    kMaxSlots * sizeof(uint2) + 256 * sizeof(float) + kWavesPerBlock * kWin * sizeof(uint16_t);

// LDS bytes one workgroup may use on the current device (cached per device).
size_t lds_per_block() {
  static std::atomic<int> cache[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 64 * 1024;
  int v = cache[dev].load(std::memory_order_relaxed);
  if (v == 0) {
    if (hipDeviceGetAttribute(&v, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) != hipSuccess ||
        v <= 0)
      v = 64 * 1024;
    cache[dev].store(v, std::memory_order_relaxed);
  }
  return static_cast<size_t>(v);
}

template <int MODE, bool UNIFORM, bool XLDS>
void launch_mode(const Args &a, hipStream_t s) {
  const dim3 grid((a.n_chunks + kWavesPerBlock - 1) / kWavesPerBlock), block(kBlock);
  const size_t shm = XLDS ? size_t(a.batch) * a.cols * sizeof(uint16_t) : 0;
  switch (a.lanes) {
    case 64:
      hipLaunchKernelGGL((decode_kernel<1, MODE, UNIFORM, XLDS>), grid, block, shm, s, a);
      break;
    case 128:
      hipLaunchKernelGGL((decode_kernel<2, MODE, UNIFORM, XLDS>), grid, block, shm, s, a);
      break;
    default:
      hipLaunchKernelGGL((decode_kernel<4, MODE, UNIFORM, XLDS>), grid, block, shm, s, a);
      break;
  }
}

template <int MODE>
int launch_decode(const Args &a, hipStream_t s) {
  const bool uniform = a.cols % a.lanes == 0;
  const size_t xbytes = size_t(a.batch) * a.cols * sizeof(uint16_t);
  const bool xlds = MODE == kGemv && xbytes <= kMaxXLdsBytes && kStaticLds + xbytes <= lds_per_block();
  if (uniform) {
    if (xlds) launch_mode<MODE, true, true>(a, s);
    else launch_mode<MODE, true, false>(a, s);
  } else {
    if (xlds) launch_mode<MODE, false, true>(a, s);
    else launch_mode<MODE, false, false>(a, s);
  }
  return hipGetLastError() == hipSuccess ? EQ_OK : EQ_EHIP;
}

}  // namespace

extern "C" int eq_layer_prepare(const eq_layer *L, hipStream_t stream) {
  if (!layer_ok(L) || !L->sym || !L->freq || L->n_syms < 1 || L->n_syms > 256) return EQ_EINVAL;
  hipLaunchKernelGGL(prepare_kernel, dim3(1), dim3(256), 0, stream, L->sym, L->freq, L->n_syms,
                     L->lut, L->status);
  return hipGetLastError() == hipSuccess ? EQ_OK : EQ_EHIP;
}

extern "C" int eq_decode_codes(const eq_layer *L, uint8_t *codes, hipStream_t stream) {
  if (!layer_ok(L) || !codes) return EQ_EINVAL;
  Args a = make_args(L);
  a.codes = codes;
  return launch_decode<kCodes>(a, stream);
}

extern "C" int eq_decode_bf16(const eq_layer *L, uint16_t *w, hipStream_t stream) {
  if (!layer_ok(L) || !w) return EQ_EINVAL;
  Args a = make_args(L);
  a.wout = w;
  return launch_decode<kBf16>(a, stream);
}

extern "C" size_t eq_gemv_workspace_bytes(const eq_layer *L, uint32_t B) {
  if (!layer_ok(L) || B < 1 || B > kMaxBatch) return 0;
  size_t floats = (L->cols % L->lanes == 0) ? size_t(2) * L->n_chunks * B : size_t(L->rows) * B;
  return (floats * sizeof(float) + 255) / 256 * 256;
}

extern "C" int eq_decode_gemv(const eq_layer *L, const uint16_t *x, uint32_t B,
                              const uint16_t *bias, float *y, void *ws, size_t ws_bytes,
                              hipStream_t stream) {
  if (!layer_ok(L) || !x || !y || !ws || B < 1 || B > kMaxBatch) return EQ_EINVAL;
  if (ws_bytes < eq_gemv_workspace_bytes(L, B)) return EQ_EINVAL;
  if (uint64_t(B) * L->cols >= (uint64_t(1) << 32) || uint64_t(B) * L->rows >= (uint64_t(1) << 32))
    return EQ_EINVAL;
  Args a = make_args(L);
  a.x = x;
  a.batch = B;
  a.bias = bias;
  a.y = y;
  a.ws = static_cast<float *>(ws);
  const bool uniform = L->cols % L->lanes == 0;
  if (!uniform) {
    const uint32_t n = L->rows * B;
    hipLaunchKernelGGL(fill_zero_kernel, dim3((n + 255) / 256), dim3(256), 0, stream, a.ws, n);
  }
  int rc = launch_decode<kGemv>(a, stream);
  if (rc != EQ_OK) return rc;
  if (uniform) {
    if (L->n_chunks > 1)
      hipLaunchKernelGGL(merge_rows_kernel, dim3((L->n_chunks + 254) / 256), dim3(256), 0, stream,
                         a);
  } else {
    const uint32_t n = L->rows * B;
    hipLaunchKernelGGL(finalize_rows_kernel, dim3((n + 255) / 256), dim3(256), 0, stream, a);
  }
  return hipGetLastError() == hipSuccess ? EQ_OK : EQ_EHIP;
}

extern "C" int eq_get_status(const eq_layer *L, hipStream_t stream) {
  if (!L || !L->status) return EQ_EINVAL;
  int32_t h = 0;
  if (hipMemcpyAsync(&h, L->status, sizeof h, hipMemcpyDeviceToHost, stream) != hipSuccess)
    return EQ_EHIP;
  if (hipStreamSynchronize(stream) != hipSuccess) return EQ_EHIP;
  return h ? EQ_ECORRUPT : EQ_OK;
}
