// gfx950 kernels and C-ABI launchers of libeq (declared in include/eq.h).
//
// Alg. 2 of the paper: ANS decoding of the per-layer bitstream, view as the
// row-major weight matrix, and the product with the per-row-scaled weights
// (Sec. 2.1 dequantiser and linear layer).  One wavefront owns one chunk:
// each of its 64 lanes holds W/64 interleaved coder states, the slot table
// sits in LDS, and the stream words of a step are handed out with a
// wavefront ballot and a masked bit count, which reproduces the coder's
// ascending-lane read order exactly.
#include <hip/hip_runtime.h>

#include <atomic>
#include <mutex>
#include <type_traits>

#include "eq.h"
#include "eq_device.h"
#include "eq_internal.h"
#include "eq_v2.h"

namespace {

using namespace eq_detail;
using namespace eq_dev;

constexpr int kMaxWaves = 16;                 // wavefronts per block (one chunk each at a time)
constexpr int kMaxBlock = kWave * kMaxWaves;
constexpr int kMaxBatch = 8;
constexpr uint32_t kHalf = 512;               // stream words per window half (1 KiB)
constexpr uint32_t kWin = 2 * kHalf;          // per-wave LDS window of stream words
constexpr uint32_t kMaxXLdsBytes = 64 * 1024; // activations staged whole up to this size
constexpr uint32_t kTileBytes = 48 * 1024;    // one activation tile at most (two are in LDS)
constexpr uint32_t kMinTileBytes = 32 * 1024; // tiles at least this large, or no tiling
constexpr uint32_t kStageRegs = 4;            // 16-byte registers per thread to stage a tile

enum Mode { kCodes = 0, kBf16 = 1, kGemv = 2 };

// Where the GEMV reads activations from.
enum XSrc {
  kXGlobal = 0,  // device memory, [batch][cols]
  kXLds = 1,     // whole in LDS (column pairs when W >= 128 and rows are whole steps)
  kXTile = 2     // tiles shared by a block of same-column chunks (see gemv_tiled_kernel)
};

struct Args {
  const uint32_t *lut;          // slot table, f32 value table, bf16 value table
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
  float *ws;                    // row partials (uniform) or row sums (general shapes)
  const uint32_t *xp;           // activations in column-pair layout (tiled GEMV)
  uint32_t fmt;                 // base format of the codes (kFmtE4M3 / kFmtInt8)
  uint32_t ncls;                // chunk classes sharing a start column (tiled GEMV)
  uint32_t tile_steps;          // steps per activation tile (tiled GEMV)
};

// One v_mfma_f32_4x4x4_16b_bf16: 16 blocks of 4 lanes, C[i][j] += sum_k
// A[i][k] B[k][j], where lane 4 blk + i holds row i of A (four BF16 in two
// registers, low half first) and lane 4 blk + j holds column j of B and
// column j of C (register i = row i).  The diagonal C[j][j], register
// (lane & 3) of lane 4 blk + j, is therefore the lane's own four-term dot
// product of its A and B values; the other registers hold cross terms.
__device__ inline float4v mfma_dot4(uint32_t a01, uint32_t a23, uint32_t b01, uint32_t b23,
                                    float4v c) {
  typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
  return __builtin_amdgcn_mfma_f32_4x4x4bf16_1k(__builtin_bit_cast(short4v, u32x2{a01, a23}),
                                                __builtin_bit_cast(short4v, u32x2{b01, b23}),
                                                c, 0, 0, 0);
}

// The lane's own entry of an mfma_dot4 accumulator.
__device__ inline float mfma_diag(float4v c, uint32_t lane) {
  const uint32_t j = lane & 3u;
  return j == 0 ? c.x : j == 1 ? c.y : j == 2 ? c.z : c.w;
}

// Byte address of the row-table entry of the code in bits 24..31 of a slot
// entry e (bits 13..23 of e are zero, so e >> 23 is twice the code); tab is
// the table's address over 512.
__device__ inline uint32_t rowtab_addr(uint32_t tab, uint32_t e) {
  return __builtin_amdgcn_alignbit(tab, e, 23);
}

// Two E4M3FN codes (bytes 0 and 1 of c) to the BF16 pair of their values
// (exact: every E4M3 value is a BF16 value).
__device__ inline uint32_t e4m3x2_to_bf16x2(uint32_t c) {
  return __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(c, 1.0f, false));
}

// BF16 pair of the values of the codes in bits 24..31 of two slot entries
// (low half: lo's).  Exact: every E4M3 value and every integer in [-127,
// 127] is a BF16 value.  E4M3: one byte permute and one hardware conversion.
template <int FMT>
__device__ inline uint32_t codes_to_bf16x2(uint32_t lo, uint32_t hi) {
  if (FMT == kFmtInt8)
    return pack_bf16(static_cast<float>(static_cast<int32_t>(lo) >> 24),
                     static_cast<float>(static_cast<int32_t>(hi) >> 24));
  return e4m3x2_to_bf16x2(__builtin_amdgcn_perm(hi, lo, 0x0c0c0703u));
}

// Value of the code in bits 24..31 of a slot entry, exactly (E4M3FN: the
// hardware's conversion of that byte; Int8: the sign-extended byte).
template <int FMT>
__device__ inline float code_f32(uint32_t e) {
  if (FMT == kFmtInt8) return static_cast<float>(static_cast<int32_t>(e) >> 24);
  return __builtin_amdgcn_cvt_f32_fp8(static_cast<int>(e), 3);
}

// Value-table entry of the code in bits 24..31 of a slot entry.  Bits 13..23
// of the entry are zero (f <= 2^12), so e >> 22 is already the byte offset.
__device__ inline uint32_t code_value(const uint32_t *val_s, uint32_t e) {
  return *reinterpret_cast<const uint32_t *>(reinterpret_cast<const char *>(val_s) + (e >> 22));
}

// Decode tables.  Slot s of symbol k (cum_k <= s < cum_k + f_k):
//   lut[2s]   = f_k | code_k << 24     (low 24 bits feed a 24-bit multiply-add)
//   lut[2s+1] = s - cum_k
// then lut[2 kMaxSlots + c] = fp32 bits of the value of code c in the base
// format (E4M3FN, or Int8 two's complement) and lut[2 kMaxSlots + 256 + c] =
// its BF16 bits (exact), zero-extended.
__global__ __launch_bounds__(1024) void prepare_kernel(const uint8_t *sym, const uint16_t *freq,
                                                       uint32_t K, uint32_t nslots, uint32_t fmt,
                                                       uint32_t *lut, int32_t *status) {
  __shared__ uint32_t cum_s[257];
  const uint32_t t = threadIdx.x;
  if (t == 0) {
    uint32_t c = 0;
    for (uint32_t k = 0; k < K; ++k) {
      cum_s[k] = c;
      c += freq[k];
    }
    cum_s[K] = c;
  }
  __syncthreads();
  for (uint32_t s = t; s < nslots; s += blockDim.x) {
    uint32_t lo = 0, hi = K - 1;  // largest k with cum_k <= s
    while (lo < hi) {
      const uint32_t mid = (lo + hi + 1) / 2;
      if (cum_s[mid] <= s) lo = mid;
      else hi = mid - 1;
    }
    lut[2 * s] = uint32_t(freq[lo]) | (uint32_t(sym[lo]) << 24);
    lut[2 * s + 1] = s - cum_s[lo];
  }
  if (t < 256) {
    const float v = fmt == kFmtInt8 ? static_cast<float>(static_cast<int8_t>(t)) : e4m3_value(t);
    const uint32_t bits = __float_as_uint(v);
    lut[2 * kMaxSlots + t] = bits;
    lut[2 * kMaxSlots + 256 + t] = bits >> 16;
  }
  if (t == 0) *status = 0;
}

// Column-pair layout of the activations (whole-row steps, W >= 128, so N is
// a multiple of 128).  A pair is (x[b][128 m + l], x[b][128 m + 64 + l]) as
// two BF16; batch rows go in groups of bw = 4 (bw = 1 when B = 1), padded
// with zeros, and u32 entry ((m * BG + bg) * 64 + l) * bw + bb holds the pair
// of batch row b = bg * bw + bb.  One lane then reads the pairs of four batch
// rows with one 16-byte load.
__host__ __device__ inline uint32_t pair_width(uint32_t B) { return B == 1 ? 1u : 4u; }
__host__ __device__ inline uint32_t pair_groups(uint32_t B) {
  return (B + pair_width(B) - 1) / pair_width(B);
}
__host__ __device__ inline size_t pair_bytes(uint32_t B, uint32_t N) {
  return size_t(N / 2) * pair_groups(B) * pair_width(B) * sizeof(uint32_t);
}

// Entry i = ((m * BG + bg) * 64 + l) * bw + bb of the column-paired layout:
// x[b][128 m + l] | x[b][128 m + l + 64] << 16 with b = bg * bw + bb (zero
// beyond the batch).  bw is 1 or 4 and BG is 1 or 2 (B <= 8), so the index
// splits with shifts.
__device__ inline uint32_t pair_entry(const uint16_t *x, uint32_t N, uint32_t B, uint32_t i) {
  const uint32_t lbw = B == 1 ? 0u : 2u;  // log2 bw
  const uint32_t lbg = B > 4 ? 1u : 0u;   // log2 BG
  const uint32_t bb = i & ((1u << lbw) - 1), l = (i >> lbw) & 63u;
  const uint32_t bg = (i >> (lbw + 6)) & ((1u << lbg) - 1), m = i >> (lbw + 6 + lbg);
  const uint32_t b = (bg << lbw) + bb;
  if (b >= B) return 0;
  const uint16_t *row = x + size_t(b) * N + 128 * m + l;
  return uint32_t(row[0]) | (uint32_t(row[64]) << 16);
}

// Batch 1: entries 4 j .. 4 j + 3 of the paired layout (N % 128 == 0, x
// 8-byte aligned): two 8-byte loads and one 16-byte result.
__device__ inline uint4 pair_entries4(const uint16_t *x, uint32_t j) {
  const uint32_t m = j >> 4, l = (j & 15) * 4;
  const uint2 lo = *reinterpret_cast<const uint2 *>(x + 128 * m + l);
  const uint2 hi = *reinterpret_cast<const uint2 *>(x + 128 * m + l + 64);
  return make_uint4(__builtin_amdgcn_perm(hi.x, lo.x, 0x05040100u),
                    __builtin_amdgcn_perm(hi.x, lo.x, 0x07060302u),
                    __builtin_amdgcn_perm(hi.y, lo.y, 0x05040100u),
                    __builtin_amdgcn_perm(hi.y, lo.y, 0x07060302u));
}

// Batch 8 with W = 256 (the matrix-core GEMV, N a multiple of 256): the same
// pairs, ordered so that one 16-byte load holds both pairs of a lane's step
// for two batch rows.  Entry i = ((m * 4 + r) * 64 + l) * 4 + e holds the
// pair (x[b][c], x[b][c + 64]) with c = 256 m + 128 (e & 1) + l and
// b = 2 r + (e >> 1).
__device__ inline uint32_t quad_entry(const uint16_t *x, uint32_t N, uint32_t i) {
  const uint32_t e = i & 3u, l = (i >> 2) & 63u, r = (i >> 8) & 3u, m = i >> 10;
  const uint32_t b = 2 * r + (e >> 1);
  const uint16_t *row = x + size_t(b) * N + 256 * m + 128 * (e & 1u) + l;
  return uint32_t(row[0]) | (uint32_t(row[64]) << 16);
}

__global__ void pair_layout_kernel(const uint16_t *x, uint32_t N, uint32_t B, uint32_t quad,
                                   uint32_t *xp) {
  const uint32_t i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < pair_bytes(B, N) / sizeof(uint32_t))
    xp[i] = quad ? quad_entry(x, N, i) : pair_entry(x, N, B, i);
}

// Static LDS of a decode block: the value table first, so that its byte
// offsets fit the 16-bit immediate of LDS instructions, then the slot table
// (33 KiB, a multiple of 512 bytes).
struct DecodeLds {
  uint32_t val[256];
  uint2 slot[kMaxSlots];
};

// Dynamic LDS of a decode block, sized for its wavefronts: one stream window
// per wavefront, then the activations (GEMV: whole, or two tiles), then, for
// BF16 output on whole-row steps, one 512-byte row table per wavefront at a
// 512-byte aligned address, so that the byte address of an entry is
// (table address) | (2 * code).
constexpr uint32_t kWinBytes = kWin * sizeof(uint16_t);
constexpr uint32_t kRowTabBytes = 256 * sizeof(uint16_t);
// BF16 output (uniform rows): per wavefront a row table and a staging area
// of one step's values (at most 256 BF16 values, the size of a row table).
__host__ __device__ inline size_t dyn_lds_bytes(uint32_t waves, size_t xbytes, bool rowtabs) {
  return size_t(waves) * kWinBytes + xbytes + (rowtabs ? kRowTabBytes * (2 * waves + 1) : 0);
}

// Stage the decode tables (and nothing else) into LDS.
template <int MODE>
__device__ inline void stage_tables(const Args &a, DecodeLds &sm) {
  const uint32_t nthreads = blockDim.x;
  const uint32_t nslots = 1u << a.prob_bits;
  const uint4 *src = reinterpret_cast<const uint4 *>(a.lut);
  uint4 *dst = reinterpret_cast<uint4 *>(sm.slot);
  for (uint32_t i = threadIdx.x; i < nslots / 2; i += nthreads) dst[i] = src[i];
  const uint32_t *vsrc = a.lut + 2 * kMaxSlots + (MODE == kGemv ? 256 : 0);
  for (uint32_t i = threadIdx.x; i < 256; i += nthreads) sm.val[i] = vsrc[i];
}

// Decoder of one chunk by one wavefront.  G = W / 64 coder states per lane
// (state g * 64 + lane); MODE selects what is done with each decoded symbol;
// UNIFORM means every step of W symbols lies inside one matrix row (N is a
// multiple of W); XS says where the GEMV reads activations; NB is the GEMV
// batch when fixed at compile time (0: the runtime batch, up to 8); FMT is
// the base format of the codes where the GEMV converts them in registers
// (PAIR); every other path reads the layer's value table.
template <int G, int MODE, bool UNIFORM, int XS, int NB, int FMT = kFmtE4M3>
struct Decoder {
  static constexpr uint32_t W = G * kWave;
  // GEMV on pairs of states (2q, 2q+1) of a lane: columns j and j + 64
  static constexpr bool PAIR = MODE == kGemv && UNIFORM && G >= 2 && XS != kXGlobal;

  const Args &a;
  const uint2 *slot;
  const uint32_t *val;
  uint4 *win4;
  const uint16_t *win;
  const void *xl;  // activations in LDS (kXLds)
  uint32_t lane, c, N, k0, nc, P, mask, last8, full;
  int nb;
  uint32_t x[G];
  // Stream position: wb is the word index of the window's first word, ra
  // the LDS byte address of the next unread word (wa: of the window start).
  uint32_t p_end, wb, wa, ra;
  uint4 next;
  __amdgpu_buffer_rsrc_t out_rsrc;
  uint32_t row, first_row, row_end;
  uint16_t *rowtab;  // this wavefront's row table (BF16 output, uniform rows)
  float srow;        // its row's scale
  // BF16 output of the pipelined steps: a step's values are written to the
  // staging area in column order, then each lane reads back its G adjacent
  // columns and stores them with one store (instead of one per state).

  uint32_t tab;      // its LDS address over 512
  uint32_t prow[G], pcol[G];
  float acc[1][kMaxBatch];

  // Software pipeline over the states of a lane (full steps, see prun): a
  // state's slot entry is read while the states issued before it are
  // processed, and its renormalisation word while later states are.
  static constexpr bool PIPE =
      G >= 2 && (MODE == kCodes || (UNIFORM && (MODE == kBf16 || PAIR)));
  static constexpr int LAG = G / 2;  // processing trails issue by LAG states
  static constexpr bool STAGED = PIPE && MODE == kBf16;
  // BF16 values of the pipelined steps computed on the VALU from the code and
  // the row's scale (two per pack), not looked up in the row table: the row
  // table's scattered two-byte reads were the LDS's busiest traffic.
  static constexpr bool VBF16 = PIPE && MODE == kBf16;
  // Batch-8 GEMV of the pipelined steps on the matrix cores: once both state
  // pairs of a lane are converted, one 4x4x4 MFMA per batch row adds the
  // lane's four products (its diagonal entry, see mfma_dot4) where eight
  // v_dot2 would.  The MFMA shares the VALU's issue port, so this halves the
  // issue slots of the products.
  static constexpr bool MFMA8 = PAIR && PIPE && G == 4 && NB == 8;
  float4v macc[MFMA8 ? kMaxBatch : 1];
  uint32_t w01;      // BF16 weights of state pair 0 (MFMA8), waiting for pair 1
  uint4 xq8[MFMA8 ? 4 : 1];  // a step's activation pairs for batch rows 2 r, 2 r + 1 (MFMA8)
  uint2 ent[G];      // slot entries in flight
  uint32_t qv[G];    // x >> P of the state whose entry is in flight
  uint64_t nd[G];    // renormalisation masks of the last processed step
  uint32_t wd[G];    // renormalisation words in flight
  uint32_t sym[G];   // slot entry .x of the last processed step (code in bits 24..31)
  uint32_t outv[G];  // BF16 values in flight, stored at step offset okk[g]
  uint32_t okk[G];
  uint32_t stg;                // staging area (LDS byte address) + 2 * lane
  bool staged;                 // output through the staging area (wave-uniform)
  uint32_t pend[G > 1 ? G / 2 : 1];  // a step's G values of this lane, read back
  uint32_t pkk;                // their step offset
  bool pend_valid;
  uint32_t xv1[G / 2 > 0 ? G / 2 : 1];    // activation pairs of a state pair (batch 1)
  uint4 xv8[G / 2 > 0 ? G / 2 : 1][2];     // (batch > 1), per 4-row batch group
  uint32_t icol;     // column of the first symbol of the step being issued
  // Issue priority of the pipelined steps: 3 until step prio_at[0], then 2,
  // 1 and from prio_at[2] on 0.  The wave arbiter prefers higher priority
  // and, among equals, older waves; at one priority the waves started first
  // run ahead and the last ones finish alone on a compute unit, with nothing
  // to hide their latencies.  Lowering a wave's priority as it passes these
  // points lets the waves behind it catch up; the last stage is short, so
  // the waves of a compute unit finish close together.
  // The tiled GEMV's waves meet at a barrier every tile: there the points
  // divide each tile's steps the same way.
  static constexpr bool PRIO = true;
  uint32_t prio_at[3];

  __device__ __forceinline__ Decoder(const Args &a_, uint32_t c_, uint32_t lane_,
                                     const DecodeLds &sm, uint4 *win4_, uint16_t *rowtab_,
                                     const void *xl_, uint16_t *stage_ = nullptr)
      : a(a_), slot(sm.slot), val(sm.val), win4(win4_),
        win(reinterpret_cast<const uint16_t *>(win4_)), xl(xl_), lane(lane_), c(c_),
        rowtab(rowtab_) {
    staged = uniform(stage_ != nullptr ? 1u : 0u) != 0;
    stg = stage_ ? uniform(lds_addr(stage_)) + 2 * lane_ : 0;
    N = a.cols;
    k0 = c * a.chunk_syms;
    nc = min(a.chunk_syms, a.n - k0);
    P = a.prob_bits;
    mask = (1u << P) - 1;
    full = nc / W;
    prio_at[0] = full / 2;
    prio_at[1] = full - full / 4;
    prio_at[2] = full - full / 16;
    nb = NB ? NB : static_cast<int>(a.batch);
#pragma unroll
    for (int g = 0; g < G; ++g) x[g] = a.chunk_state[c * W + g * kWave + lane];
    const uint32_t p = as_const(a.chunk_off)[c];
    p_end = as_const(a.chunk_off)[c + 1];
    // Window loads stop at the 8-word group holding the chunk's last word
    // (words past it are never consumed); later groups repeat it from cache.
    last8 = min(a.padded_words - 8, p_end & ~7u);
    // Stream words [wb, wb + kWin) live in this wave's LDS window and the
    // next half is in flight in registers.  A step reads at most W words and
    // the window slides by a half whenever p passes its middle, so every word
    // a step can read is in LDS.
    wb = p & ~7u;
    wa = uniform(lds_addr(win));
    ra = wa + 2 * (p - wb);
    {
      const uint4 h0 = load_words(a.words, wb + 8 * lane, last8);
      const uint4 h1 = load_words(a.words, wb + kHalf + 8 * lane, last8);
      win4[lane] = h0;
      win4[kHalf / 8 + lane] = h1;
    }
    __builtin_amdgcn_s_waitcnt(0);  // states, offsets and window are in
    next = load_words(a.words, wb + kWin + 8 * lane, last8);
    // Outputs of this chunk go through buffer resources: the address is the
    // chunk's base plus a scalar step offset plus the lane's offset.  Stores
    // of the partial last step are predicated per lane.
    if (MODE == kCodes)
      out_rsrc = __builtin_amdgcn_make_buffer_rsrc(a.codes + k0, 0, int(nc), kBufferFlags);
    if (MODE == kBf16)
      out_rsrc = __builtin_amdgcn_make_buffer_rsrc(a.wout + k0, 0, int(2 * nc), kBufferFlags);
    row = k0 / N;
    first_row = row;
    row_end = (row + 1) * N;  // <= n < 2^32
    if (MODE == kBf16 && UNIFORM) {
      tab = uniform(lds_addr(rowtab) >> 9);
      fill_rowtab(row);
    }
    if (!UNIFORM) {
#pragma unroll
      for (int g = 0; g < G; ++g) {
        const uint32_t pos = k0 + g * kWave + lane;
        prow[g] = pos / N;
        pcol[g] = pos - prow[g] * N;
      }
    }
#pragma unroll
    for (int b = 0; b < kMaxBatch; ++b) acc[0][b] = 0.0f;
#pragma unroll
    for (int b = 0; b < (MFMA8 ? kMaxBatch : 1); ++b) macc[b] = float4v{0.0f, 0.0f, 0.0f, 0.0f};
  }

  __device__ __forceinline__ uint32_t xbits(uint32_t b, uint32_t col) const {
    return XS == kXLds ? reinterpret_cast<const uint16_t *>(xl)[b * N + col] : a.x[b * N + col];
  }

  // Finished row r of a uniform chunk: y directly if the chunk holds the whole
  // row, else the partial sum (slot 0: first row, slot 1: last row).
  __device__ __forceinline__ void flush_uniform(uint32_t r) {
    const bool owned = r * N >= k0 && (r + 1) * N <= k0 + nc;
    const float s = bf16_at(a.scale, r);
    const float bb = a.bias ? bf16_at(a.bias, r) : 0.0f;
#pragma unroll
    for (int b = 0; b < kMaxBatch; ++b) {
      if (MFMA8) {
        acc[0][b] += mfma_diag(macc[b], lane);
        macc[b] = float4v{0.0f, 0.0f, 0.0f, 0.0f};
      }
      if (b < nb) {
        const float sum = wave_sum(acc[0][b]);
        if (lane == 0) {
          if (owned) a.y[b * a.rows + r] = s * sum + bb;
          else a.ws[(2 * c + (r == first_row ? 0 : 1)) * a.batch + b] = sum;
        }
      }
      acc[0][b] = 0.0f;
    }
  }

  // Row table of row r: bf16(s_r * v(code)) for every code, the exact
  // product rounded once (codes outside the base format never occur in a
  // valid container).  v comes from the fp32 value table.
  __device__ __forceinline__ void fill_rowtab(uint32_t r) {
    const float s = bf16_at(a.scale, r);
    srow = s;
    const uint32_t c = 4 * lane;
    const uint32_t lo = pack_bf16(s * __uint_as_float(val[c]), s * __uint_as_float(val[c + 1]));
    const uint32_t hi =
        pack_bf16(s * __uint_as_float(val[c + 2]), s * __uint_as_float(val[c + 3]));
    reinterpret_cast<uint2 *>(rowtab)[lane] = make_uint2(lo, hi);
  }

  // Whole-row steps: move to the next row when step t starts it.
  __device__ __forceinline__ void row_check(uint32_t t) {
    if (UNIFORM && MODE != kCodes && k0 + t * W >= row_end) {
      if (MODE == kGemv) flush_uniform(row);
      ++row;
      row_end += N;
      if (MODE == kBf16) fill_rowtab(row);
    }
  }

  // Slide the stream window by one half once the position has passed its
  // middle.
  __device__ __forceinline__ void slide() {
    if (ra - wa >= 2 * kHalf) {
      const uint4 keep = win4[kHalf / 8 + lane];
      win4[lane] = keep;
      win4[kHalf / 8 + lane] = next;
      wb += kHalf;
      ra -= 2 * kHalf;
      next = load_words(a.words, wb + kWin + 8 * lane, last8);
    }
  }

  // One step: W symbols at chunk offset t * W, inside the current row (for
  // whole-row steps the caller has done row_check).  TAIL: the last,
  // partial step.  SLIDE: check the window first (a step reads at most W
  // words, so two steps fit between checks).  xt: this step's activation
  // pairs in LDS (kXTile only), in column-pair layout starting at the step's
  // first 128-column block.
  template <bool TAIL, bool SLIDE = true>
  __device__ __forceinline__ void step(uint32_t t, const uint32_t *xt) {
    if (SLIDE) slide();
    const uint32_t kk = t * W;  // offset of this step inside the chunk
    bool act[G];
#pragma unroll
    for (int g = 0; g < G; ++g) act[g] = !TAIL || kk + g * kWave + lane < nc;

    // decode every active state of the step
    uint32_t e0[G];
#pragma unroll
    for (int g = 0; g < G; ++g) {
      if (act[g]) {
        const uint2 e = slot[x[g] & mask];
        x[g] = __umul24(e.x, x[g] >> P) + e.y;
        e0[g] = e.x;
      } else {
        e0[g] = 0;  // code 0: value +0
      }
    }

    // use the symbols
    uint32_t outv[G];
    if (MODE == kCodes) {
#pragma unroll
      for (int g = 0; g < G; ++g)
        if (!TAIL || act[g])
          __builtin_amdgcn_raw_buffer_store_b8(static_cast<uint8_t>(e0[g] >> 24), out_rsrc,
                                               lane + g * kWave, kk, 0);
    } else if (MODE == kBf16 && UNIFORM) {
      // one row-table read per symbol; stored once the renormalisation has
      // been issued
#pragma unroll
      for (int g = 0; g < G; ++g) outv[g] = lds_read_u16(rowtab_addr(tab, e0[g]));
    } else if (MODE == kBf16) {
#pragma unroll
      for (int g = 0; g < G; g += 2) {
        const float s0 = bf16_at(a.scale, prow[g]);
        const float v0 = s0 * __uint_as_float(val[e0[g] >> 24]);
        float v1 = 0.0f;
        if (g + 1 < G) {
          const float s1 = bf16_at(a.scale, prow[g + 1]);
          v1 = s1 * __uint_as_float(val[e0[g + 1] >> 24]);
        }
        const uint32_t h = pack_bf16(v0, v1);  // exact products, rounded once
        if (!TAIL || act[g])
          __builtin_amdgcn_raw_buffer_store_b16(static_cast<uint16_t>(h), out_rsrc,
                                                2 * (lane + g * kWave), 2 * kk, 0);
        if (g + 1 < G && (!TAIL || act[g + 1]))
          __builtin_amdgcn_raw_buffer_store_b16(static_cast<uint16_t>(h >> 16), out_rsrc,
                                                2 * (lane + (g + 1) * kWave), 2 * kk, 0);
      }
    } else if (MFMA8) {
      // batch 8, quad layout: the step's 256 columns are one block of 1024 entries
      const uint32_t *xq = XS == kXTile
                               ? xt + 4 * lane
                               : reinterpret_cast<const uint32_t *>(xl) +
                                     ((k0 + kk + N - row_end) >> 8) * 1024 + 4 * lane;
      const uint32_t w0 = codes_to_bf16x2<FMT>(e0[0], e0[1]);
      const uint32_t w1 = codes_to_bf16x2<FMT>(e0[2], e0[3]);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const uint4 xv = *reinterpret_cast<const uint4 *>(xq + r * 256);
        acc[0][2 * r] = dot2_bf16(w1, xv.y, dot2_bf16(w0, xv.x, acc[0][2 * r]));
        acc[0][2 * r + 1] = dot2_bf16(w1, xv.w, dot2_bf16(w0, xv.z, acc[0][2 * r + 1]));
      }
    } else if (PAIR) {
      // pairs of this step's 128-column blocks: xq + (q * BG + bg) * 64 * bw
      constexpr uint32_t bw = NB == 1 ? 1 : 4;
      const uint32_t BG = NB == 1 ? 1 : (nb + 3) / 4;
      const uint32_t *xq;
      if (XS == kXTile) {
        xq = xt + lane * bw;
      } else {
        const uint32_t blk = (k0 + kk + N - row_end) >> 7;  // first 128-column block
        xq = reinterpret_cast<const uint32_t *>(xl) + (blk * BG * kWave + lane) * bw;
      }
#pragma unroll
      for (int q = 0; q < G / 2; ++q) {
        const uint32_t w2 = codes_to_bf16x2<FMT>(e0[2 * q], e0[2 * q + 1]);
        if (NB == 1) {
          acc[0][0] = dot2_bf16(w2, xq[q * kWave], acc[0][0]);
        } else {
#pragma unroll
          for (uint32_t bg = 0; bg < 2; ++bg) {
            if (bg < BG) {
              const uint4 xv =
                  *reinterpret_cast<const uint4 *>(xq + (q * BG + bg) * kWave * bw);
              acc[0][4 * bg + 0] = dot2_bf16(w2, xv.x, acc[0][4 * bg + 0]);
              acc[0][4 * bg + 1] = dot2_bf16(w2, xv.y, acc[0][4 * bg + 1]);
              acc[0][4 * bg + 2] = dot2_bf16(w2, xv.z, acc[0][4 * bg + 2]);
              acc[0][4 * bg + 3] = dot2_bf16(w2, xv.w, acc[0][4 * bg + 3]);
            }
          }
        }
      }
    } else if (MODE == kGemv) {
#pragma unroll
      for (int g = 0; g < G; ++g) {
        if (!act[g]) continue;
        const uint32_t v = code_value(val, e0[g]);  // BF16 value in the low half
        const uint32_t col = (k0 + kk + N - row_end) + g * kWave + lane;
#pragma unroll
        for (int b = 0; b < kMaxBatch; ++b)
          if (b < nb) acc[0][b] = dot2_bf16(v, xbits(b, col), acc[0][b]);
      }
    }
    if (!UNIFORM && MODE == kBf16) {
#pragma unroll
      for (int g = 0; g < G; ++g) {
        // advance this state's position by one step (W symbols)
        pcol[g] += W;
        if (pcol[g] >= N) {
          prow[g] += pcol[g] / N;
          pcol[g] %= N;
        }
      }
    }

    // renormalise in ascending state order (state g*64 + lane): all reads of
    // the step are issued before any is used.  A lane's word follows those of
    // the needing lanes below it.
    uint64_t need[G];
    uint32_t word[G];
    uint32_t r = ra;
#pragma unroll
    for (int g = 0; g < G; ++g) {
      need[g] = __builtin_amdgcn_ballot_w64(act[g] && x[g] < kStateLow);
      const uint32_t below = __builtin_amdgcn_mbcnt_hi(
          uint32_t(need[g] >> 32), __builtin_amdgcn_mbcnt_lo(uint32_t(need[g]), 0u));
      word[g] = lds_read_u16(r + 2 * below);
      r = add_twice(r, static_cast<uint32_t>(__popcll(need[g])));
    }
#pragma unroll
    for (int g = 0; g < G; ++g) x[g] = select_by_mask(need[g], x[g], (x[g] << 16) | word[g]);
    ra = r;

    if (MODE == kBf16 && UNIFORM) {
#pragma unroll
      for (int g = 0; g < G; ++g)
        if (!TAIL || act[g])
          __builtin_amdgcn_raw_buffer_store_b16(static_cast<uint16_t>(outv[g]), out_rsrc,
                                                2 * (lane + g * kWave), 2 * kk, 0);
    }
  }

  // Close the chunk: last row sums, end-of-chunk check (every state back at
  // 2^16, stream used up exactly).
  __device__ __forceinline__ void finish() {
    if (MODE == kGemv) flush_uniform(row);
    bool bad = wb + (ra - wa) / 2 != p_end;
#pragma unroll
    for (int g = 0; g < G; ++g) bad |= x[g] != kStateLow;
    if (__builtin_amdgcn_ballot_w64(bad) != 0 && lane == 0) atomicOr(a.status, 1);
  }

  // --- pipelined full steps -------------------------------------------------

  // Activation pairs of state pair q for the step whose first column is col
  // (kXLds) or whose tile is at xt (kXTile).
  __device__ __forceinline__ void load_x(int q, uint32_t col, const uint32_t *xt) {
    if (MFMA8) {
      // all eight batch rows of both pairs at once, after the step's last state
      if (q == G / 2 - 1) {
        const uint32_t *xq = (XS == kXTile ? xt : reinterpret_cast<const uint32_t *>(xl) +
                                                      (col >> 8) * 1024) + 4 * lane;
#pragma unroll
        for (int r = 0; r < 4; ++r) xq8[r] = *reinterpret_cast<const uint4 *>(xq + r * 256);
      }
      return;
    }
    constexpr uint32_t bw = NB == 1 ? 1 : 4;
    const uint32_t BG = NB == 1 ? 1 : (nb + 3) / 4;
    const uint32_t *xq;
    if (XS == kXTile) xq = xt + lane * bw;
    else xq = reinterpret_cast<const uint32_t *>(xl) + ((col >> 7) * BG * kWave + lane) * bw;
    if (NB == 1) {
      xv1[q] = xq[q * kWave];
    } else {
#pragma unroll
      for (uint32_t bg = 0; bg < 2; ++bg)
        if (bg < BG) xv8[q][bg] = *reinterpret_cast<const uint4 *>(xq + (q * BG + bg) * kWave * bw);
    }
  }

  // Staged BF16 output of the pipelined steps: a step's values are written to
  // the wavefront's staging area in column order (state g of lane l at column
  // 64 g + l); then each lane reads back its G adjacent columns (G lane ..)
  // and stores them with one store, when the next step is read back (or at
  // the end of the run).  One store per step instead of one per state.
  __device__ __forceinline__ void stage_put(int g, uint32_t v) {
    lds_write_u16(stg + 2 * kWave * g, v);
  }
  __device__ __forceinline__ void stage_store() {
    typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
    if (G >= 4)
      __builtin_amdgcn_raw_buffer_store_b64(u32x2{pend[0], pend[G >= 4 ? 1 : 0]}, out_rsrc,
                                            2 * G * lane, 2 * pkk, 0);
    else
      __builtin_amdgcn_raw_buffer_store_b32(pend[0], out_rsrc, 2 * G * lane, 2 * pkk, 0);
  }
  // Read back the staged step at chunk offset kk (storing the previous one).
  __device__ __forceinline__ void stage_get(uint32_t kk) {
    if (pend_valid) stage_store();
    const uint32_t addr = stg + 2 * (G - 1) * lane;  // staging area + 2 G lane
    if (G >= 4) {
      const uint64_t v = *lds_ptr<const uint64_t>(addr);
      pend[0] = static_cast<uint32_t>(v);
      pend[G >= 4 ? 1 : 0] = static_cast<uint32_t>(v >> 32);
    } else {
      pend[0] = *lds_ptr<const uint32_t>(addr);
    }
    pkk = kk;
    pend_valid = true;
  }

  // BF16 value of state g for its store: the pair packs of the pipelined
  // steps leave an odd state's value in the high half, which a d16_hi store
  // writes directly.
  __device__ __forceinline__ uint32_t out_half(int g) const {
    return (VBF16 && G >= 4 && (g & 1)) ? outv[g] >> 16 : outv[g];
  }

  // Issue state g of step t: finish its renormalisation from the previous
  // step (unless FIRST), put out its pending BF16 value (STG: into the
  // staging area; after the last state, read the step back), start its slot
  // read.
  template <bool FIRST, bool STG>
  __device__ __forceinline__ void pissue(int g, const uint32_t *xt) {
    if (!FIRST) {
      x[g] = renorm_lanes(nd[g], x[g], wd[g]);
      if (MODE == kBf16) {
        if (STG) {
          stage_put(g, out_half(g));
          if (g == G - 1) stage_get(okk[g]);
        } else {
          __builtin_amdgcn_raw_buffer_store_b16(static_cast<uint16_t>(out_half(g)), out_rsrc,
                                                2 * (lane + g * kWave), 2 * okk[g], 0);
        }
      }
    }
    ent[g] = slot[x[g] & mask];
    qv[g] = x[g] >> P;
    if (PAIR && (g & 1)) load_x(g / 2, icol, xt);
  }

  // Process state h of step t (chunk offset kk): decode, start its
  // renormalisation read, use the symbol.
  __device__ __forceinline__ void pproc(int h, uint32_t kk) {
    x[h] = __umul24(ent[h].x, qv[h]) + ent[h].y;
    sym[h] = ent[h].x;
    nd[h] = __builtin_amdgcn_ballot_w64(x[h] < kStateLow);
    const uint32_t below = __builtin_amdgcn_mbcnt_hi(uint32_t(nd[h] >> 32),
                                                     __builtin_amdgcn_mbcnt_lo(uint32_t(nd[h]), 0u));
    wd[h] = lds_read_u16(ra + 2 * below);
    ra = add_twice(ra, static_cast<uint32_t>(__popcll(nd[h])));
    if (MODE == kCodes) {
      __builtin_amdgcn_raw_buffer_store_b8(static_cast<uint8_t>(sym[h] >> 24), out_rsrc,
                                           lane + h * kWave, kk, 0);
    } else if (MODE == kBf16) {
      if (VBF16) {
        // bf16(s * v): the fp32 product is exact, rounded once, as in the row
        // table.  G = 4: for the pair (h - 1, h), one pack (state h - 1's value
        // is first stored after state h is processed); G = 2: state 0's value
        // is stored before state 1 is processed, so one value at a time.
        if (G >= 4) {
          if (h & 1) {
            const uint32_t pr = pack_bf16(srow * code_f32<FMT>(sym[(h - 1) & (G - 1)]),
                                          srow * code_f32<FMT>(sym[h]));
            outv[(h - 1) & (G - 1)] = pr;
            outv[h] = pr;  // its high half (see out_half)
          }
        } else {
          outv[h] = pack_bf16(srow * code_f32<FMT>(sym[h]), 0.0f);
        }
      } else {
        outv[h] = lds_read_u16(rowtab_addr(tab, sym[h]));
      }
      okk[h] = kk;
    } else if (h & 1) {
      const int q = h / 2;
      const uint32_t w2 = codes_to_bf16x2<FMT>(sym[h - 1], sym[h]);
      if (NB == 1) {
        acc[0][0] = dot2_bf16(w2, xv1[q], acc[0][0]);
      } else if (MFMA8) {
        if (q == 0) {
          w01 = w2;
        } else {
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            macc[2 * r] = mfma_dot4(xq8[r].x, xq8[r].y, w01, w2, macc[2 * r]);
            macc[2 * r + 1] = mfma_dot4(xq8[r].z, xq8[r].w, w01, w2, macc[2 * r + 1]);
          }
        }
      } else {
        const uint32_t BG = (nb + 3) / 4;
#pragma unroll
        for (uint32_t bg = 0; bg < 2; ++bg) {
          if (bg < BG) {
            const uint4 xv = xv8[q][bg];
            acc[0][4 * bg + 0] = dot2_bf16(w2, xv.x, acc[0][4 * bg + 0]);
            acc[0][4 * bg + 1] = dot2_bf16(w2, xv.y, acc[0][4 * bg + 1]);
            acc[0][4 * bg + 2] = dot2_bf16(w2, xv.z, acc[0][4 * bg + 2]);
            acc[0][4 * bg + 3] = dot2_bf16(w2, xv.w, acc[0][4 * bg + 3]);
          }
        }
      }
    }
  }

  // Full steps [t, t_end), software-pipelined: for each step t the states are
  // issued in order g = 0..G-1, and after issuing g the wave processes state
  // g - LAG (of step t, or of step t - 1 when g < LAG).  Processing stays in
  // ascending state order, step by step, which is the order of the stream's
  // words.  Rows change between the last state of step t - 1 and the first
  // of step t.  xt: step t's activation tile (kXTile), stride xs per step.
  __device__ __forceinline__ void prun(uint32_t t, uint32_t t_end, const uint32_t *xt,
                                       uint32_t xs) {
    if (STAGED && staged) prun_impl<true>(t, t_end, xt, xs);
    else prun_impl<false>(t, t_end, xt, xs);
  }
  template <bool STG>
  __device__ __forceinline__ void prun_impl(uint32_t t, uint32_t t_end, const uint32_t *xt,
                                            uint32_t xs) {
    static_assert(2 * W <= kWin - kHalf, "a step and a half must fit the window");
    if (XS == kXTile) {
      const uint32_t n = t_end - t;
      prio_at[0] = t + n / 2;
      prio_at[1] = t + n - n / 4;
      prio_at[2] = t + n - n / 16;
    }
    if (STG) pend_valid = false;
    slide();
    if (MODE != kCodes) {
      row_check(t);
      icol = k0 + t * W + N - row_end;
    }
#pragma unroll
    for (int g = 0; g < G; ++g) pissue<true, STG>(g, xt);
#pragma unroll
    for (int h = 0; h < LAG; ++h) pproc(h, t * W);
    for (++t; t < t_end;) {
      // Issue priority 3 - (stage of the chunk reached, see prio_at).
      uint32_t seg_end = t_end;
      if (PRIO) {
        const uint32_t q = (t >= prio_at[0]) + (t >= prio_at[1]) + (t >= prio_at[2]);
        seg_end =
            min(t_end, q == 0 ? prio_at[0] : q == 1 ? prio_at[1] : q == 2 ? prio_at[2] : t_end);
        set_prio_down(q);
      }
      for (; t < seg_end; ++t) {
      // t stays a plain scalar counter (not rewritten into a vector one)
      asm("" : "+s"(t));
      // words read since the last check: at most one step and a half
      slide();
      xt += xs;
      if (MODE != kCodes) {
        icol += W;
        if (icol >= N) icol -= N;
      }
#pragma unroll
      for (int g = 0; g < G; ++g) {
        pissue<false, STG>(g, xt);
        if (g < LAG) {
          pproc(g + G - LAG, (t - 1) * W);
        } else {
          if (g == LAG) row_check(t);
          pproc(g - LAG, t * W);
        }
      }
      }
    }
#pragma unroll
    for (int h = LAG; h < G; ++h) pproc(h, (t - 1) * W);
#pragma unroll
    for (int g = 0; g < G; ++g) {
      x[g] = renorm_lanes(nd[g], x[g], wd[g]);
      if (MODE == kBf16 && !STG)
        __builtin_amdgcn_raw_buffer_store_b16(static_cast<uint16_t>(out_half(g)), out_rsrc,
                                              2 * (lane + g * kWave), 2 * okk[g], 0);
    }
    if (STG) {
#pragma unroll
      for (int g = 0; g < G; ++g) stage_put(g, out_half(g));
      stage_get(okk[G - 1]);
      stage_store();
    }
  }

  // Full steps [t, t_end), a row segment at a time, two steps per iteration
  // with one window check.  Step t's activation tile is xt + (t - t_first) *
  // xs (kXTile).
  __device__ __forceinline__ void run_steps(uint32_t t, uint32_t t_end, const uint32_t *xt,
                                            uint32_t xs) {
    static_assert(2 * W <= kWin - kHalf, "two steps must fit the window");
    if constexpr (PIPE) {
      if (t < t_end) prun(t, t_end, xt, xs);
      return;
    }
    while (t < t_end) {
      uint32_t seg_end = t_end;
      if (UNIFORM && MODE != kCodes) {
        row_check(t);
        seg_end = min(t_end, (row_end - k0) / W);  // first step of the next row
      }
      for (; t + 1 < seg_end; t += 2, xt += 2 * xs) {
        step<false, true>(t, xt);
        step<false, false>(t + 1, xt + xs);
      }
      if (t < seg_end) {
        step<false, true>(t, xt);
        ++t;
        xt += xs;
      }
    }
  }

  // The partial last step of a chunk, if any.
  __device__ __forceinline__ void tail(const uint32_t *xt) {
    if (nc % W) {
      row_check(full);
      step<true>(full, xt);
    }
  }

  __device__ __forceinline__ void run() {
    run_steps(0, full, nullptr, 0);
    tail(nullptr);
    finish();
  }
};

// One block's share of a layer: block blk of nblk decodes chunks blk * waves
// + wave, + nblk * waves, ...  Dynamic LDS (dyn): the wavefronts' stream
// windows, then the activations (kXLds) or the row tables.
template <int G, int MODE, bool UNIFORM, int XS, int NB, int FMT>
__device__ __forceinline__ void decode_block(const Args &a, uint32_t blk, uint32_t nblk,
                                             DecodeLds &sm, uint4 *dyn) {
  const uint32_t nthreads = blockDim.x;
  const uint32_t waves = uniform(nthreads / kWave);
  uint4 *const xl = dyn + waves * (kWinBytes / sizeof(uint4));
  stage_tables<MODE>(a, sm);
  if (XS == kXLds) {
    const uint32_t nx = a.batch * a.cols;
    if (Decoder<G, MODE, UNIFORM, XS, NB, FMT>::PAIR) {
      uint32_t *xp = reinterpret_cast<uint32_t *>(xl);
      const uint32_t np = pair_bytes(a.batch, a.cols) / sizeof(uint32_t);
      if (Decoder<G, MODE, UNIFORM, XS, NB, FMT>::MFMA8) {
        for (uint32_t i = threadIdx.x; i < np; i += nthreads) xp[i] = quad_entry(a.x, a.cols, i);
      } else if (a.batch == 1 && (reinterpret_cast<uintptr_t>(a.x) & 7) == 0) {
        for (uint32_t j = threadIdx.x; j < np / 4; j += nthreads) xl[j] = pair_entries4(a.x, j);
      } else {
        for (uint32_t i = threadIdx.x; i < np; i += nthreads) xp[i] = pair_entry(a.x, a.cols, a.batch, i);
      }
    } else if (nx % 8 == 0 && (reinterpret_cast<uintptr_t>(a.x) & 15) == 0) {
      const uint4 *xv = reinterpret_cast<const uint4 *>(a.x);
      for (uint32_t i = threadIdx.x; i < nx / 8; i += nthreads) xl[i] = xv[i];
    } else {
      uint16_t *xs = reinterpret_cast<uint16_t *>(xl);
      for (uint32_t i = threadIdx.x; i < nx; i += nthreads) xs[i] = a.x[i];
    }
  }
  __syncthreads();

  const uint32_t lane = threadIdx.x & (kWave - 1);
  const uint32_t wave = uniform(threadIdx.x / kWave);
  uint16_t *rowtab = nullptr, *stage = nullptr;
  if (MODE == kBf16 && UNIFORM) {
    char *base = reinterpret_cast<char *>(xl);
    base += (0u - lds_addr(base)) & (kRowTabBytes - 1);
    rowtab = reinterpret_cast<uint16_t *>(base) + wave * 256;
    // staged output (G values per store) needs the output's steps aligned
    constexpr uintptr_t step_align = 2 * G;
    if (G >= 2 && (reinterpret_cast<uintptr_t>(a.wout) & (step_align - 1)) == 0)
      stage = reinterpret_cast<uint16_t *>(base) + (waves + wave) * 256;
  }
  uint4 *const win = dyn + wave * (kWinBytes / sizeof(uint4));
  for (uint32_t c = uniform(blk * waves + wave); c < a.n_chunks; c += nblk * waves) {
    Decoder<G, MODE, UNIFORM, XS, NB, FMT> d(a, c, lane, sm, win, rowtab, xl, stage);
    d.run();
  }
}

template <int G, int MODE, bool UNIFORM, int XS, int NB, int FMT>
__global__ __launch_bounds__(kMaxBlock) void decode_kernel(Args a) {
  extern __shared__ uint4 dyn[];
  __shared__ DecodeLds sm;
  decode_block<G, MODE, UNIFORM, XS, NB, FMT>(a, blockIdx.x, gridDim.x, sm, dyn);
}

// Several layers in one launch (whole-row steps, one lane count): blocks
// [blk_end[i-1], blk_end[i]) decode layer i.  For the GEMV the layers share
// the activations.
constexpr uint32_t kMaxLayers = 8;
struct MultiArgs {
  Args a[kMaxLayers];
  uint32_t blk_end[kMaxLayers];
  uint32_t n;
};

template <int G, int MODE, int XS, int NB, int FMT>
__global__ __launch_bounds__(kMaxBlock) void multi_decode_kernel(MultiArgs m) {
  extern __shared__ uint4 dyn[];
  __shared__ DecodeLds sm;
  uint32_t i = 0, b0 = 0;
  while (i + 1 < m.n && blockIdx.x >= m.blk_end[i]) b0 = m.blk_end[i++];
  decode_block<G, MODE, true, XS, NB, FMT>(m.a[i], blockIdx.x - b0, m.blk_end[i] - b0, sm, dyn);
}

// Fused GEMV for activations too large for LDS (whole-row steps, W >= 128).
// Chunks c and c + ncls start at the same column (ncls = N / gcd(C, N)), so a
// block of wavefronts holding chunks of one class walks the same columns in
// lockstep: the block stages tiles of tile_steps steps of column-paired
// activations (from a.xp) into LDS, double-buffered, with one barrier per
// tile.  Block b serves class b % ncls, chunks of index (b / ncls) * waves +
// wave within the class.
template <int G, int NB, int FMT>
__global__ __launch_bounds__(kMaxBlock) void gemv_tiled_kernel(Args a) {
  extern __shared__ uint4 dyn[];  // stream windows, then 2 x tile
  __shared__ DecodeLds sm;
  using Dec = Decoder<G, kGemv, true, kXTile, NB, FMT>;
  constexpr uint32_t W = Dec::W;
  stage_tables<kGemv>(a, sm);

  const uint32_t nthreads = blockDim.x;
  const uint32_t lane = threadIdx.x & (kWave - 1);
  const uint32_t wave = uniform(threadIdx.x / kWave);
  const uint32_t waves = uniform(nthreads / kWave);
  const uint32_t N = a.cols, B = a.batch, T = a.tile_steps;
  (void)B;
  const uint32_t cls = blockIdx.x % a.ncls;
  const uint32_t c = cls + a.ncls * ((blockIdx.x / a.ncls) * waves + wave);
  const bool has = c < a.n_chunks;
  const uint32_t col0 = uint32_t((uint64_t(cls) * a.chunk_syms) % N);
  const uint32_t nblk = N / 128;                      // 128-column blocks per row
  const uint32_t blk_u4 = pair_groups(B) * pair_width(B) * kWave / 4;  // 16-byte units per block
  const uint32_t step_u4 = (W / 128) * blk_u4;        // per step
  const uint32_t tile_u4 = T * step_u4;
  const uint32_t steps = a.chunk_syms / W;            // steps of a full chunk
  const uint32_t ntiles = (steps + T - 1) / T;
  const uint4 *src = reinterpret_cast<const uint4 *>(a.xp);
  uint4 *const tiles = dyn + waves * (kWinBytes / sizeof(uint4));

  // tile k covers steps [k T, k T + T): 128-column blocks from col0/128 + k T W/128;
  // each thread moves 16-byte units i = threadIdx.x + s * nthreads, s < kStageRegs,
  // unit i from block (tile's first block + i / blk_u4) mod nblk.  Both terms are
  // kept reduced mod nblk (the first advanced once per tile), so a unit's block
  // takes one compare and subtract instead of a division.
  static_assert(kStageRegs == 4, "staging uses four registers");
  const uint32_t adv = (T * (W / 128)) % nblk;
  uint32_t qoff[kStageRegs], roff[kStageRegs];
#pragma unroll
  for (uint32_t s = 0; s < kStageRegs; ++s) {
    const uint32_t i = threadIdx.x + s * nthreads;
    qoff[s] = (i / blk_u4) % nblk;
    roff[s] = i % blk_u4;
  }
  auto fetch = [&](uint32_t base, uint32_t s) -> uint4 {
    const uint32_t i = threadIdx.x + s * nthreads;
    if (i >= tile_u4) return uint4{0, 0, 0, 0};
    uint32_t blk = base + qoff[s];
    blk -= blk >= nblk ? nblk : 0;
    return src[blk * blk_u4 + roff[s]];
  };
  auto store = [&](uint32_t buf, uint32_t s, const uint4 v) {
    const uint32_t i = threadIdx.x + s * nthreads;
    if (i < tile_u4) tiles[buf * tile_u4 + i] = v;
  };

  uint32_t base = col0 / 128;  // first block of tile 0 (col0 < N)
  uint4 r0 = fetch(base, 0), r1 = fetch(base, 1), r2 = fetch(base, 2), r3 = fetch(base, 3);
  store(0, 0, r0);
  store(0, 1, r1);
  store(0, 2, r2);
  store(0, 3, r3);
  __syncthreads();  // tables and the first tile are in

  Dec d(a, has ? c : 0, lane, sm, dyn + wave * (kWinBytes / sizeof(uint4)), nullptr, nullptr);
  for (uint32_t k = 0; k < ntiles; ++k) {
    const bool more = k + 1 < ntiles;
    if (more) {
      base += adv;  // first block of tile k + 1
      base -= base >= nblk ? nblk : 0;
      r0 = fetch(base, 0);
      r1 = fetch(base, 1);
      r2 = fetch(base, 2);
      r3 = fetch(base, 3);
    }
    if (has) {
      const uint32_t *tile = reinterpret_cast<const uint32_t *>(tiles + (k & 1) * tile_u4);
      const uint32_t t0 = k * T, t1 = min(t0 + T, d.full);
      if (t0 < t1) d.run_steps(t0, t1, tile, step_u4 * 4);
      // the partial last step of the matrix's last chunk, while its tile is in LDS
      if (d.full >= t0 && d.full < t0 + T) d.tail(tile + (d.full - t0) * step_u4 * 4);
    }
    if (more) {
      const uint32_t buf = (k + 1) & 1;
      store(buf, 0, r0);
      store(buf, 1, r1);
      store(buf, 2, r2);
      store(buf, 3, r3);
    }
    __syncthreads();
  }
  if (has) d.finish();
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

// Rows whose steps are not whole (N not a multiple of W): the GEMV runs on
// the decoded codes, one block per row, each thread summing a fixed stride of
// columns and the block reducing in a fixed tree, so y does not depend on
// timing.  y = s * sum_j v(codes[r][j]) x[b][j] + bias.
constexpr int kRowThreads = 256;
__global__ __launch_bounds__(kRowThreads) void codes_gemv_kernel(Args a, const uint8_t *codes) {
  __shared__ float part[kRowThreads / kWave][kMaxBatch];
  const uint32_t r = blockIdx.x, t = threadIdx.x, N = a.cols;
  const uint8_t *q = codes + size_t(r) * N;
  const float *val = reinterpret_cast<const float *>(a.lut + 2 * kMaxSlots);
  float acc[kMaxBatch];
#pragma unroll
  for (int b = 0; b < kMaxBatch; ++b) acc[b] = 0.0f;
  for (uint32_t j = t; j < N; j += kRowThreads) {
    const float v = val[q[j]];
#pragma unroll
    for (int b = 0; b < kMaxBatch; ++b)
      if (b < int(a.batch)) acc[b] += v * bf16_to_f32(a.x[size_t(b) * N + j]);
  }
#pragma unroll
  for (int b = 0; b < kMaxBatch; ++b) {
    const float sum = wave_sum(acc[b]);
    if ((t & (kWave - 1)) == 0) part[t / kWave][b] = sum;
  }
  __syncthreads();
  if (t < a.batch) {
    float sum = 0.0f;
    for (int w = 0; w < kRowThreads / kWave; ++w) sum += part[w][t];
    const float bb = a.bias ? bf16_to_f32(a.bias[r]) : 0.0f;
    a.y[size_t(t) * a.rows + r] = bf16_to_f32(a.scale[r]) * sum + bb;
  }
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
  a.fmt = L->base_format;
  return a;
}

bool layer_ok(const eq_layer *L) {
  return L && L->version == 1 && L->lut && L->status && L->words && L->chunk_off && L->chunk_state && L->scale &&
         (L->lanes == 64 || L->lanes == 128 || L->lanes == 256) &&
         L->prob_bits >= kMinProbBits && L->prob_bits <= 12 && L->n_chunks > 0 && L->cols > 0 &&
         L->rows > 0 && (L->base_format == kFmtE4M3 || L->base_format == kFmtInt8);
}

constexpr size_t kStaticLds = sizeof(DecodeLds);

struct DeviceFacts {
  int lds_per_block = 64 * 1024;
  int cus = 256;
};

// Per-device limits, queried once per device.
DeviceFacts device_facts() {
  static std::atomic<int> lds[64], cus[64];
  int dev = 0;
  DeviceFacts f;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return f;
  int l = lds[dev].load(std::memory_order_relaxed), c = cus[dev].load(std::memory_order_relaxed);
  if (l == 0) {
    if (hipDeviceGetAttribute(&l, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) != hipSuccess ||
        l <= 0)
      l = f.lds_per_block;
    if (hipDeviceGetAttribute(&c, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        c <= 0)
      c = f.cus;
    lds[dev].store(l, std::memory_order_relaxed);
    cus[dev].store(c, std::memory_order_relaxed);
  }
  f.lds_per_block = l;
  f.cus = c;
  return f;
}

// Blocks of up to 16 wavefronts, one chunk per wavefront at a time.  With
// fewer chunks than wavefront slots, the chunks are spread evenly over the
// compute units (one block each); otherwise each wavefront loops over chunks.
uint32_t launch_waves(uint32_t n_chunks, int cus) {
  const uint32_t waves = (n_chunks + cus - 1) / cus;
  return waves < 1 ? 1 : (waves > kMaxWaves ? kMaxWaves : waves);
}

void launch_shape(uint32_t n_chunks, int cus, dim3 &grid, dim3 &block) {
  const uint32_t waves = launch_waves(n_chunks, cus);
  uint32_t blocks = (n_chunks + waves - 1) / waves;
  if (blocks > uint32_t(cus) * 4) blocks = uint32_t(cus) * 4;
  grid = dim3(blocks);
  block = dim3(waves * kWave);
}

uint32_t gcd_u32(uint32_t a, uint32_t b) {
  while (b) {
    const uint32_t t = a % b;
    a = b;
    b = t;
  }
  return a;
}

// LDS bytes of the activations staged whole (column pairs when usable).
size_t xlds_bytes(const Args &a) {
  const bool pairs = a.cols % a.lanes == 0 && a.lanes >= 128;
  return pairs ? pair_bytes(a.batch, a.cols) : size_t(a.batch) * a.cols * sizeof(uint16_t);
}

// Activation placement of a GEMV launch.
int gemv_xsrc(const Args &a, const DeviceFacts &f, uint32_t waves) {
  const bool uniform = a.cols % a.lanes == 0;
  const size_t xbytes = xlds_bytes(a);
  if (xbytes <= kMaxXLdsBytes &&
      kStaticLds + dyn_lds_bytes(waves, xbytes, false) <= size_t(f.lds_per_block))
    return kXLds;
  if (uniform && a.lanes >= 128 &&
      kStaticLds + dyn_lds_bytes(kMaxWaves, 2 * kMinTileBytes, false) <= size_t(f.lds_per_block))
    return kXTile;
  return kXGlobal;
}

// The base format a kernel is built for: only the in-register conversions
// (paired GEMV, pipelined BF16 steps) depend on it; every other path reads
// the layer's value table, so those share the E4M3 build.
template <int G, int MODE, bool UNIFORM, int XS, int NB, int FMT>
constexpr int kernel_fmt() {
  return Decoder<G, MODE, UNIFORM, XS, NB, kFmtE4M3>::PAIR ||
                 Decoder<G, MODE, UNIFORM, XS, NB, kFmtE4M3>::VBF16
             ? FMT
             : int(kFmtE4M3);
}

template <int MODE, bool UNIFORM, int XS, int NB, int FMT>
void launch_mode(const Args &a, hipStream_t s, const DeviceFacts &f) {
  dim3 grid, block;
  launch_shape(a.n_chunks, f.cus, grid, block);
  const size_t shm = dyn_lds_bytes(block.x / kWave, XS == kXLds ? xlds_bytes(a) : 0,
                                    MODE == kBf16 && UNIFORM);
  switch (a.lanes) {
    case 64:
      hipLaunchKernelGGL(
          (decode_kernel<1, MODE, UNIFORM, XS, NB, kernel_fmt<1, MODE, UNIFORM, XS, NB, FMT>()>),
          grid, block, shm, s, a);
      break;
    case 128:
      hipLaunchKernelGGL(
          (decode_kernel<2, MODE, UNIFORM, XS, NB, kernel_fmt<2, MODE, UNIFORM, XS, NB, FMT>()>),
          grid, block, shm, s, a);
      break;
    default:
      hipLaunchKernelGGL(
          (decode_kernel<4, MODE, UNIFORM, XS, NB, kernel_fmt<4, MODE, UNIFORM, XS, NB, FMT>()>),
          grid, block, shm, s, a);
      break;
  }
}

template <int MODE, bool UNIFORM, int XS, int FMT>
void launch_batch(const Args &a, hipStream_t s, const DeviceFacts &f) {
  if (MODE != kGemv || a.batch == 1) launch_mode<MODE, UNIFORM, XS, 1, FMT>(a, s, f);
  else if (a.batch == kMaxBatch) launch_mode<MODE, UNIFORM, XS, kMaxBatch, FMT>(a, s, f);
  else launch_mode<MODE, UNIFORM, XS, 0, FMT>(a, s, f);
}

template <int MODE, int FMT>
void launch_decode_fmt(const Args &a, hipStream_t s, const DeviceFacts &f) {
  const bool uniform = a.cols % a.lanes == 0;
  if (MODE != kGemv) {
    if (uniform) launch_batch<MODE, true, kXGlobal, FMT>(a, s, f);
    else launch_batch<MODE, false, kXGlobal, FMT>(a, s, f);
  } else if (gemv_xsrc(a, f, launch_waves(a.n_chunks, f.cus)) == kXLds) {
    launch_batch<MODE, true, kXLds, FMT>(a, s, f);  // GEMV: whole-row steps only
  } else {
    launch_batch<MODE, true, kXGlobal, FMT>(a, s, f);
  }
}

template <int MODE>
int launch_decode(const Args &a, hipStream_t s) {
  const DeviceFacts f = device_facts();
  if ((MODE == kGemv || MODE == kBf16) && a.fmt == kFmtInt8)
    launch_decode_fmt<MODE, kFmtInt8>(a, s, f);
  else launch_decode_fmt<MODE, kFmtE4M3>(a, s, f);
  return hipGetLastError() == hipSuccess ? EQ_OK : EQ_EHIP;
}

// Tiled GEMV launch: the number of wavefronts per block is the smallest that
// lets every block of every class run at once; tiles are as long as the
// LDS budget and the staging registers allow.
template <int NB>
int launch_tiled(Args a, hipStream_t s, const DeviceFacts &f) {
  const uint32_t W = a.lanes, C = a.chunk_syms, N = a.cols;
  a.ncls = N / gcd_u32(C % N, N);  // gcd(0, N) = N: one class
  const uint32_t per_cls = (a.n_chunks + a.ncls - 1) / a.ncls;
  uint32_t waves = kMaxWaves;
  for (uint32_t w = (a.n_chunks + f.cus - 1) / f.cus; w <= kMaxWaves; ++w) {
    if (w == 0) continue;
    if (a.ncls * ((per_cls + w - 1) / w) <= uint32_t(f.cus)) {
      waves = w;
      break;
    }
  }
  const uint32_t step_bytes =
      uint32_t(pair_bytes(a.batch, W));  // W columns of column-paired activations
  // Steps per tile: up to kTileBytes, as many as the block's threads stage
  // with their registers, and two tiles beside the tables and windows in LDS
  // (longer tiles mean fewer barriers, where the block's waves wait for the
  // slowest).
  uint32_t T = kTileBytes / step_bytes;
  const uint32_t max_by_regs = kStageRegs * waves * kWave * 16 / step_bytes;
  if (T > max_by_regs) T = max_by_regs;
  while (T > 1 && kStaticLds + dyn_lds_bytes(waves, 2 * size_t(T) * step_bytes, false) >
                      size_t(f.lds_per_block))
    --T;
  if (T < 1) T = 1;
  a.tile_steps = T;
  const dim3 grid(a.ncls * ((per_cls + waves - 1) / waves)), block(waves * kWave);
  const size_t shm = dyn_lds_bytes(waves, 2 * size_t(T) * step_bytes, false);
  const bool int8 = a.fmt == kFmtInt8;
  if (W == 128 && int8)
    hipLaunchKernelGGL((gemv_tiled_kernel<2, NB, kFmtInt8>), grid, block, shm, s, a);
  else if (W == 128)
    hipLaunchKernelGGL((gemv_tiled_kernel<2, NB, kFmtE4M3>), grid, block, shm, s, a);
  else if (int8)
    hipLaunchKernelGGL((gemv_tiled_kernel<4, NB, kFmtInt8>), grid, block, shm, s, a);
  else
    hipLaunchKernelGGL((gemv_tiled_kernel<4, NB, kFmtE4M3>), grid, block, shm, s, a);
  return hipGetLastError() == hipSuccess ? EQ_OK : EQ_EHIP;
}

size_t round256(size_t v) { return (v + 255) / 256 * 256; }

// Multi-layer launch shape: the fewest wavefronts per block (at most
// max_waves) for which two blocks per compute unit hold every chunk.  Each
// layer gets whole blocks, so the count is checked after rounding each
// layer's blocks up: blocks beyond two per compute unit would run as a
// second round and double the launch's time.  Launches that need several
// rounds anyway are balanced across compute units instead (below).
uint32_t multi_shape(const MultiArgs &m, int cus, uint32_t max_waves, MultiArgs &out) {
  uint64_t total = 0;
  for (uint32_t i = 0; i < m.n; ++i) total += m.a[i].n_chunks;
  const uint64_t slots = 2 * uint64_t(cus);
  uint32_t waves = uint32_t((total + slots - 1) / slots);
  waves = waves < 1 ? 1 : (waves > max_waves ? max_waves : waves);
  auto blocks_at = [&](uint32_t w) {
    uint64_t b = 0;
    for (uint32_t i = 0; i < m.n; ++i) b += (m.a[i].n_chunks + w - 1) / w;
    return b;
  };
  for (; waves < max_waves; ++waves)
    if (blocks_at(waves) <= slots) break;
  // More blocks than one round holds even at max_waves: blocks are handed to
  // compute units as others finish, so the busiest unit decodes about
  // ceil(blocks / cus) * waves chunks.  Take the wave count in
  // [max_waves / 2, max_waves] that makes this smallest (the larger on
  // ties): a partial last round otherwise leaves units idle while others
  // still decode two blocks.
  if (blocks_at(waves) > slots) {
    uint64_t best = ~uint64_t(0);
    for (uint32_t w = max_waves; w >= 1 && w >= (max_waves + 1) / 2; --w) {
      const uint64_t load = (blocks_at(w) + cus - 1) / cus * w;
      if (load < best) {
        best = load;
        waves = w;
      }
    }
  }
  out = m;
  uint32_t end = 0;
  for (uint32_t i = 0; i < m.n; ++i) {
    end += (m.a[i].n_chunks + waves - 1) / waves;
    out.blk_end[i] = end;
  }
  return waves;
}

template <int MODE, int XS, int NB, int FMT>
int launch_multi_fmt(const MultiArgs &m0, size_t xbytes, hipStream_t s, const DeviceFacts &f) {
  MultiArgs m;
  // BF16: no more wavefronts than let two blocks share a compute unit's LDS
  // (16 would leave room for one, with row tables and staging areas)
  uint32_t max_waves = kMaxWaves;
  if (MODE == kBf16)
    while (max_waves > 1 &&
           2 * (kStaticLds + dyn_lds_bytes(max_waves, xbytes, true)) > size_t(f.lds_per_block))
      --max_waves;
  const uint32_t waves = multi_shape(m0, f.cus, max_waves, m);
  const dim3 grid(m.blk_end[m.n - 1]), block(waves * kWave);
  const size_t shm = dyn_lds_bytes(waves, xbytes, MODE == kBf16);
  switch (m.a[0].lanes) {
    case 64:
      hipLaunchKernelGGL(
          (multi_decode_kernel<1, MODE, XS, NB, kernel_fmt<1, MODE, true, XS, NB, FMT>()>), grid,
          block, shm, s, m);
      break;
    case 128:
      hipLaunchKernelGGL(
          (multi_decode_kernel<2, MODE, XS, NB, kernel_fmt<2, MODE, true, XS, NB, FMT>()>), grid,
          block, shm, s, m);
      break;
    default:
      hipLaunchKernelGGL(
          (multi_decode_kernel<4, MODE, XS, NB, kernel_fmt<4, MODE, true, XS, NB, FMT>()>), grid,
          block, shm, s, m);
      break;
  }
  return hipGetLastError() == hipSuccess ? EQ_OK : EQ_EHIP;
}

// Layers of one launch share a base format (joint_ok).
template <int MODE, int XS, int NB>
int launch_multi(const MultiArgs &m, size_t xbytes, hipStream_t s, const DeviceFacts &f) {
  if ((MODE == kGemv || MODE == kBf16) && m.a[0].fmt == kFmtInt8)
    return launch_multi_fmt<MODE, XS, NB, kFmtInt8>(m, xbytes, s, f);
  return launch_multi_fmt<MODE, XS, NB, kFmtE4M3>(m, xbytes, s, f);
}

// Layers that can share one launch: whole-row steps, one lane count, one
// base format.
bool joint_ok(const eq_layer *const *L, uint32_t n) {
  for (uint32_t i = 0; i < n; ++i)
    if (L[i]->cols % L[i]->lanes != 0 || L[i]->lanes != L[0]->lanes ||
        L[i]->base_format != L[0]->base_format)
      return false;
  return true;
}

}  // namespace

extern "C" int eq_layer_prepare(const eq_layer *L, hipStream_t stream) {
  if (L && L->version == 2) return v2_prepare(L, stream);
  if (!layer_ok(L) || !L->sym || !L->freq || L->n_syms < 1 || L->n_syms > 256) return EQ_EINVAL;
  hipLaunchKernelGGL(prepare_kernel, dim3(1), dim3(1024), 0, stream, L->sym, L->freq, L->n_syms,
                     1u << L->prob_bits, L->base_format, L->lut, L->status);
  return hipGetLastError() == hipSuccess ? EQ_OK : EQ_EHIP;
}

extern "C" int eq_decode_codes(const eq_layer *L, uint8_t *codes, hipStream_t stream) {
  if (L && L->version == 2) return v2_decode_codes(L, codes, stream);
  if (!layer_ok(L) || !codes) return EQ_EINVAL;
  Args a = make_args(L);
  a.codes = codes;
  return launch_decode<kCodes>(a, stream);
}

extern "C" int eq_decode_bf16(const eq_layer *L, uint16_t *w, hipStream_t stream) {
  if (L && L->version == 2) return v2_decode_bf16(L, w, stream);
  if (!layer_ok(L) || !w) return EQ_EINVAL;
  Args a = make_args(L);
  a.wout = w;
  return launch_decode<kBf16>(a, stream);
}

// Workspace: row partials (2 per chunk and batch row), then room for the
// column-paired activations; for rows that are not whole steps, the decoded
// codes (one byte per weight).
extern "C" size_t eq_gemv_workspace_bytes(const eq_layer *L, uint32_t B) {
  if (L && L->version == 2) return v2_gemv_workspace_bytes(L, B);
  if (!layer_ok(L) || B < 1 || B > kMaxBatch) return 0;
  if (L->cols % L->lanes != 0) return round256(size_t(L->rows) * L->cols);
  return round256(size_t(2) * L->n_chunks * B * sizeof(float)) +
         round256(pair_bytes(B, L->cols));
}

extern "C" int eq_decode_gemv(const eq_layer *L, const uint16_t *x, uint32_t B,
                              const uint16_t *bias, float *y, void *ws, size_t ws_bytes,
                              hipStream_t stream) {
  if (L && L->version == 2) {
    if (uint64_t(B) * L->cols >= (uint64_t(1) << 32) ||
        uint64_t(B) * L->rows >= (uint64_t(1) << 32))
      return EQ_EINVAL;
    return v2_decode_gemv(L, x, B, bias, y, ws, ws_bytes, stream);
  }
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
  if (L->cols % L->lanes != 0) {
    // rows that are not whole steps: decode the codes, then a fixed-order GEMV
    uint8_t *codes = static_cast<uint8_t *>(ws);
    a.codes = codes;
    int rc = launch_decode<kCodes>(a, stream);
    if (rc != EQ_OK) return rc;
    hipLaunchKernelGGL(codes_gemv_kernel, dim3(L->rows), dim3(kRowThreads), 0, stream, a,
                       static_cast<const uint8_t *>(codes));
    return hipGetLastError() == hipSuccess ? EQ_OK : EQ_EHIP;
  }
  const size_t part_bytes = round256(size_t(2) * L->n_chunks * B * sizeof(float));
  a.xp = reinterpret_cast<const uint32_t *>(static_cast<char *>(ws) + part_bytes);
  const DeviceFacts f = device_facts();
  int rc;
  if (gemv_xsrc(a, f, launch_waves(L->n_chunks, f.cus)) == kXTile) {
    const uint32_t np = uint32_t(pair_bytes(B, L->cols) / sizeof(uint32_t));
    // the matrix-core GEMV (batch 8, 256 lanes) reads the quad layout
    const uint32_t quad = B == kMaxBatch && L->lanes == 256 ? 1u : 0u;
    hipLaunchKernelGGL(pair_layout_kernel, dim3((np + 255) / 256), dim3(256), 0, stream, x,
                       L->cols, B, quad, const_cast<uint32_t *>(a.xp));
    rc = (B == 1) ? launch_tiled<1>(a, stream, f)
                  : (B == kMaxBatch ? launch_tiled<kMaxBatch>(a, stream, f)
                                    : launch_tiled<0>(a, stream, f));
  } else {
    rc = launch_decode<kGemv>(a, stream);
  }
  if (rc != EQ_OK) return rc;
  // rows split between chunks exist only when chunks do not hold whole rows
  if (L->n_chunks > 1 && L->chunk_syms % L->cols != 0)
    hipLaunchKernelGGL(merge_rows_kernel, dim3((L->n_chunks + 254) / 256), dim3(256), 0, stream,
                       a);
  return hipGetLastError() == hipSuccess ? EQ_OK : EQ_EHIP;
}

// eq_decode_gemv_noalloc's workspace: one array per device, in the code
// object (no allocation call at any time).  Its device address comes from
// hipGetSymbolAddress on each device's first call, with that device current;
// the array's name is not a device address in host code.  Every call on a
// device shares it, so calls that overlap on one device race.  No kernel
// needs it cleared: each call writes every partial, activation pair or code
// before it reads it.
static __device__ __align__(256) unsigned char scratch[EQ_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;

static void *scratch_on_current_device() {
  static std::atomic<void *> ptr[kMaxDevices];
  static std::mutex mu;
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
  void *p = ptr[dev].load(std::memory_order_acquire);
  if (p) return p;
  std::lock_guard<std::mutex> lock(mu);
  p = ptr[dev].load(std::memory_order_relaxed);
  if (!p) {
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess) return nullptr;
    ptr[dev].store(p, std::memory_order_release);
  }
  return p;
}

extern "C" int eq_decode_gemv_noalloc(const eq_layer *L, const uint16_t *x, uint32_t B,
                                      const uint16_t *bias, float *y, hipStream_t stream) {
  const size_t need = eq_gemv_workspace_bytes(L, B);
  if (need == 0) return EQ_EINVAL;
  if (need > EQ_NOALLOC_SCRATCH_BYTES) return EQ_ESCRATCH;
  void *ws = scratch_on_current_device();
  if (!ws) return EQ_EHIP;
  return eq_decode_gemv(L, x, B, bias, y, ws, EQ_NOALLOC_SCRATCH_BYTES, stream);
}

extern "C" int eq_decode_bf16_multi(const eq_layer *const *L, uint16_t *const *w, uint32_t n,
                                    hipStream_t stream) {
  if (!L || !w || n < 1 || n > kMaxLayers) return EQ_EINVAL;
  bool v2 = false;
  for (uint32_t i = 0; i < n; ++i) {
    if (!L[i] || !w[i]) return EQ_EINVAL;
    v2 |= L[i]->version == 2;
    if (!(L[i]->version == 2 ? v2_layer_ok(L[i]) : layer_ok(L[i]))) return EQ_EINVAL;
  }
  if (v2 && v2_joint_out_ok(L, n)) return v2_decode_bf16_multi(L, w, n, stream);
  if (n == 1 || v2 || !joint_ok(L, n)) {
    for (uint32_t i = 0; i < n; ++i) {
      const int rc = eq_decode_bf16(L[i], w[i], stream);
      if (rc != EQ_OK) return rc;
    }
    return EQ_OK;
  }
  MultiArgs m{};
  m.n = n;
  for (uint32_t i = 0; i < n; ++i) {
    m.a[i] = make_args(L[i]);
    m.a[i].wout = w[i];
  }
  return launch_multi<kBf16, kXGlobal, 1>(m, 0, stream, device_facts());
}

extern "C" int eq_decode_codes_multi(const eq_layer *const *L, uint8_t *const *codes, uint32_t n,
                                     hipStream_t stream) {
  if (!L || !codes || n < 1 || n > kMaxLayers) return EQ_EINVAL;
  bool v2 = false;
  for (uint32_t i = 0; i < n; ++i) {
    if (!L[i] || !codes[i]) return EQ_EINVAL;
    v2 |= L[i]->version == 2;
    if (!(L[i]->version == 2 ? v2_layer_ok(L[i]) : layer_ok(L[i]))) return EQ_EINVAL;
  }
  if (v2 && v2_joint_out_ok(L, n)) return v2_decode_codes_multi(L, codes, n, stream);
  if (n == 1 || v2 || !joint_ok(L, n)) {
    for (uint32_t i = 0; i < n; ++i) {
      const int rc = eq_decode_codes(L[i], codes[i], stream);
      if (rc != EQ_OK) return rc;
    }
    return EQ_OK;
  }
  MultiArgs m{};
  m.n = n;
  for (uint32_t i = 0; i < n; ++i) {
    m.a[i] = make_args(L[i]);
    m.a[i].codes = codes[i];
  }
  return launch_multi<kCodes, kXGlobal, 1>(m, 0, stream, device_facts());
}

extern "C" size_t eq_gemv_multi_workspace_bytes(const eq_layer *const *L, uint32_t n, uint32_t B) {
  if (!L || n < 1 || n > kMaxLayers) return 0;
  size_t total = 0;
  for (uint32_t i = 0; i < n; ++i) {
    const size_t b = eq_gemv_workspace_bytes(L[i], B);
    if (b == 0) return 0;
    total += b;
  }
  return total;
}

extern "C" int eq_decode_gemv_multi(const eq_layer *const *L, uint32_t n, const uint16_t *x,
                                    uint32_t B, const uint16_t *const *bias, float *const *y,
                                    void *ws, size_t ws_bytes, hipStream_t stream) {
  if (!L || !y || !x || !ws || n < 1 || n > kMaxLayers || B < 1 || B > kMaxBatch)
    return EQ_EINVAL;
  bool v2 = false;
  for (uint32_t i = 0; i < n; ++i) {
    if (!L[i] || !y[i] || L[i]->cols != L[0]->cols) return EQ_EINVAL;
    v2 |= L[i]->version == 2;
    if (!(L[i]->version == 2 ? v2_layer_ok(L[i]) : layer_ok(L[i]))) return EQ_EINVAL;
  }
  if (ws_bytes < eq_gemv_multi_workspace_bytes(L, n, B)) return EQ_EINVAL;
  // layer i's workspace follows those of layers 0 .. i-1
  size_t off[kMaxLayers];
  for (uint32_t i = 0, o = 0; i < n; ++i) {
    off[i] = o;
    o += eq_gemv_workspace_bytes(L[i], B);
  }
  if (v2 && v2_joint_ok(L, n)) {
    void *wsi[kMaxLayers];
    for (uint32_t i = 0; i < n; ++i) wsi[i] = static_cast<char *>(ws) + off[i];
    return v2_decode_gemv_multi(L, n, x, B, bias, y, wsi, stream);
  }
  const DeviceFacts f = device_facts();
  MultiArgs m{};
  m.n = n;
  for (uint32_t i = 0; i < n; ++i) {
    m.a[i] = make_args(L[i]);
    m.a[i].x = x;
    m.a[i].batch = B;
    m.a[i].bias = bias ? bias[i] : nullptr;
    m.a[i].y = y[i];
    m.a[i].ws = reinterpret_cast<float *>(static_cast<char *>(ws) + off[i]);
  }
  MultiArgs shaped;
  const uint32_t waves = multi_shape(m, f.cus, kMaxWaves, shaped);
  const size_t xbytes = xlds_bytes(m.a[0]);
  const bool joint = n > 1 && !v2 && joint_ok(L, n) && xbytes <= kMaxXLdsBytes &&
                     kStaticLds + dyn_lds_bytes(waves, xbytes, false) <= size_t(f.lds_per_block);
  if (!joint) {
    for (uint32_t i = 0; i < n; ++i) {
      const int rc = eq_decode_gemv(L[i], x, B, bias ? bias[i] : nullptr, y[i],
                                    static_cast<char *>(ws) + off[i],
                                    eq_gemv_workspace_bytes(L[i], B), stream);
      if (rc != EQ_OK) return rc;
    }
    return EQ_OK;
  }
  const int rc = B == 1 ? launch_multi<kGemv, kXLds, 1>(m, xbytes, stream, f)
                        : (B == kMaxBatch ? launch_multi<kGemv, kXLds, kMaxBatch>(m, xbytes, stream, f)
                                          : launch_multi<kGemv, kXLds, 0>(m, xbytes, stream, f));
  if (rc != EQ_OK) return rc;
  for (uint32_t i = 0; i < n; ++i)
    if (L[i]->n_chunks > 1 && L[i]->chunk_syms % L[i]->cols != 0)
      hipLaunchKernelGGL(merge_rows_kernel, dim3((L[i]->n_chunks + 254) / 256), dim3(256), 0,
                         stream, m.a[i]);
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
