// gfx950 kernels for version-2 containers (eq.h): tile-ordered chunks and a
// phrase alphabet, rANS at 2^16.
//
// Alg. 2 of the paper with the coder of container version 2: one wavefront
// decodes one chunk (a tile of TR rows x TC columns); lane l holds the coder
// states of tile rows l, l + 64, ... (TR / 64 of them).  Every state walks its
// row's TC columns, one phrase of 4, 2 or 1 codes per step, so one state
// update yields 3-4 codes on the synthetic 2-bit layers.  The phrase table
// (kBuckets entries, indexed by the top 12 bits of the slot) sits in LDS.  A
// global entry holds what the state update needs and the phrase's values:
//   .x = (2^16 - F) | (2 * length) << 16      .y = 2^(16-R) * cum
//   .z, .w = the four codes' values as BF16 pairs (zero past the length)
// so that  x' = F (x >> 16) + (x mod 2^16) - cum  =  x - ((2^16 - F) (x >> 16) + cum)
// is one 16 x 16-bit multiply-add (high half of x selected by op_sel) and one
// subtraction.  The GEMV splits the entry in LDS into two 8-byte halves read
// by two 8-byte loads (a 16-byte LDS read at a random address costs about
// three times as much as an 8-byte one on gfx950): the state half (.x with
// the step of the state's position in the kernel's units, .y) at bucket * 8,
// and the value half (.z, .w) at kValHalf + bucket * 8, an offset that keeps
// the two loads from being merged.  Codes and BF16 output read one packed
// 8-byte entry {F | (cum + length) << 16, the four codes} per phrase.  Stream
// words are handed out with a wavefront ballot and a masked bit count in
// ascending state order, as the coder reads them.
//
// GEMV: all states of a chunk walk the same TC columns, so the chunk's
// activations sit in the wavefront's LDS: at batch 1 one aligned 8-byte
// record of four values per column, at batches 2-8 a table of value pairs;
// a phrase's four values meet them with two dot2 products per batch row.  A
// state's sum is its row's partial over the tile; partials of the NT column
// tiles are added in tile order by merge2_kernel (deterministic).  At batch 1
// the last states of a tile are compacted to one per lane.
//
// Codes and BF16 output: each phrase's codes go to an LDS ring of its row,
// and whole 32-code segments of rows leave the wavefront together, so that
// stores write contiguous lines.
//
// Row order: a container may cut its tiles over the rows in a stored order
// (row k of the tiling is matrix row order[k]; the encoder groups rows of
// like phrase counts, so a tile's states finish at nearly the same step).
// Only the outputs move: row sums (GEMV), scales and written rows go to the
// matrix row, the partial sums of the column tiles stay in stored order.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>

#include "eq.h"
#include "eq_device.h"
#include "eq_internal.h"
#include "eq_v2.h"

namespace {

using namespace eq_detail;
using namespace eq_dev;

constexpr int kMaxWaves2 = 16;
constexpr int kMaxBlock2 = kWave * kMaxWaves2;
// GEMV at 4 or 8 batch rows: at most 8 wavefronts per block (LDS allows about
// that many), so that a wavefront may hold up to 256 VGPRs (no spills).
constexpr int max_waves2(int mode, int nb) { return mode == 2 && nb >= 4 ? 8 : kMaxWaves2; }
constexpr int kMaxBatch2 = 8;
constexpr uint32_t kHalf2 = 512;           // stream words per window half
constexpr uint32_t kWin2 = 2 * kHalf2;     // per-wave LDS window (2 KiB)
// LDS table: state halves at [0, 32 KiB), value halves from kValHalf on.
constexpr uint32_t kValHalf = kBuckets * 8 + 8;
constexpr uint32_t kTableBytes2 = (kValHalf + kBuckets * 8 + 8 + 15) / 16 * 16;
// One more entry after the kBuckets: the identity (2^16 - F = 0, cum = 0,
// step 0, values 0), the step taken by states whose row segment is done.
constexpr uint32_t kIdentity2 = kBuckets * 8;
// Codes and BF16 output: the value half is the phrase's four codes, 4 bytes
// at kCodesHalf + bucket * 4 (the identity's after the kBuckets).
constexpr uint32_t kCodesHalf = kBuckets * 8 + 8;
constexpr uint32_t kTableCodes2 = (kCodesHalf + kBuckets * 4 + 4 + 15) / 16 * 16;
// Packed table (layers of more than one phrase; GEMV on E4M3 codes): one
// 8-byte entry per bucket, {F | (cum + length) << 16, the four codes}, and
// the identity {0, 0} after them.
constexpr uint32_t kTablePacked2 = kBuckets * 8 + 16;
// Codes and BF16 output leave the wavefront as whole 32-code segments of a
// row (64 bytes of BF16), four lanes per segment: each tile row has an LDS
// ring holding its current segment.  32-code rather than 64-code segments
// halve the rings, so more wavefronts fit a compute unit (8192 x 28672:
// codes 248 -> 232 us, BF16 298 -> 288 us).
constexpr uint32_t kSegShift = 5;
constexpr uint32_t kSeg = 1u << kSegShift;
constexpr uint32_t kRing = kSeg;
constexpr uint32_t kCPL = kSeg / 4;  // codes per lane when a segment is written out

enum Mode2 { kCodes2 = 0, kBf16_2 = 1, kGemv2 = 2 };

struct Args2 {
  const uint4 *lut;          // kBuckets phrase entries (see the file comment)
  const uint32_t *codes4;    // kBuckets phrase codes, little-endian
  const uint16_t *scale;
  const uint32_t *chunk_off;
  const uint32_t *chunk_state;
  const uint16_t *words;
  int32_t *status;
  uint32_t rows, cols, TR, TC, NT, n_chunks, padded_words;
  uint32_t wave_lds;         // bytes of dynamic LDS per wavefront after the table
  uint8_t *codes;
  uint16_t *wout;
  const uint16_t *x;
  uint32_t batch;
  uint32_t fmt;              // base format (codes to values at BF16 output)
  uint32_t n_syms;           // phrases in the alphabet
  const uint16_t *bias;
  float *y;
  float *ws;                 // partial row sums [batch][NT][rows] (NT > 1), stored order
  const uint32_t *order;     // matrix row of each stored row; null: the identity
};

// The matrix row of stored row k.  A damaged order section (a row out of
// range; the host checked its own copy) marks the layer corrupt and keeps
// the row in place, so no store leaves the output.
__device__ inline uint32_t out_row(const Args2 &a, uint32_t k) {
  if (!a.order) return k;
  const uint32_t r = as_const(a.order)[k];
  if (r < a.rows) return r;
  atomicOr(a.status, 1);
  return k;
}

// x' = x - ((2^16 - F) * (x >> 16) + cum): the 16-bit multiply takes the low
// half of e.x and the high half of x.
__device__ inline uint32_t state_update(uint32_t x, uint32_t ex, uint32_t ey) {
  uint32_t t;
  asm("v_mad_u32_u16 %0, %1, %2, %3 op_sel:[0,1,0,0]" : "=v"(t) : "v"(ex), "v"(x), "v"(ey));
  return x - t;
}

// Packed entry w = F | (cum + length) << 16 (cum has its low 16 - R >= 4
// bits zero, so the length 1, 2 or 4 sits there):
//   t = (x mod 2^16) - (cum + length)     one subtraction of selected halves
//   x' = F (x >> 16) + t + length         multiply-add, then the length back
__device__ inline uint32_t state_update_pk(uint32_t x, uint32_t w) {
  uint32_t t, y;
  asm("v_sub_u32_sdwa %0, %1, %2 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:WORD_0 "
      "src1_sel:WORD_1"
      : "=v"(t)
      : "v"(x), "v"(w));
  asm("v_mad_u32_u16 %0, %1, %2, %3 op_sel:[0,1,0,0]" : "=v"(y) : "v"(w), "v"(x), "v"(t));
  return y + ((w >> 16) & 7u);
}

typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
// the same at any byte address (outputs of an ordered layer: one store each)
typedef uint32_t u32x2u __attribute__((ext_vector_type(2), aligned(1)));
typedef uint32_t u32x4u __attribute__((ext_vector_type(4), aligned(1)));


// LDS byte offset of the state half of the bucket of state x (the table
// sits at LDS address 0): ((x mod 2^16) >> 4) * 8.
__device__ inline uint32_t bucket_addr(uint32_t x) { return (x >> 1) & 0x7FF8u; }
__device__ inline u32x2 state_half(uint32_t addr) { return *lds_ptr<const u32x2>(addr); }
__device__ inline u32x2 value_half(uint32_t addr) { return *lds_ptr<const u32x2>(addr + kValHalf); }

// Batch-1 GEMV: bytes of a wavefront's activation records (TC + 4 of 8
// bytes, rounded to 16).
__host__ __device__ constexpr uint32_t rec_bytes(uint32_t tc) { return ((tc + 4) * 8 + 15) / 16 * 16; }

// ORD (codes and BF16 only): outputs through the rows' offsets in LDS and
// 64-bit addresses, for launches with an ordered layer; without it, buffer
// stores from the tile's origin.
template <int G, int MODE, int NB, bool PK, bool ORD>
struct Tile {
  static constexpr uint32_t TR = G * kWave;
  // log2 of the position step per code (packed entries hold the length)
  static constexpr uint32_t kUnitShift =
      MODE != kGemv2 ? 0 : (NB == 1 ? 3 : (NB == 2 ? 3 : 4));
  // GEMV at batch 2-8: batch rows per pair-table entry (8 rows: two halves)
  static constexpr uint32_t NQ = NB < 4 ? NB : 4;
  const Args2 &a;
  uint32_t lane, c, r0, c0, rows, cols, tcol;
  int nb;
  uint32_t x[G];
  bool valid[G];
  uint32_t pos[G];   // GEMV: LDS byte address of the state's column (its
                     // activation record at batch 1, else in batch row 0);
                     // codes / BF16: its column in the tile
  uint32_t end;      // pos at the end of a row segment
  uint32_t qstride;  // GEMV at batch 8: bytes from one pair-table half to the other
  float srow[G];     // BF16: the state's row scale
  uint32_t rr[G];    // codes / BF16: LDS address of the state's ring
  uint32_t pend[G];  // codes / BF16: the codes of the state's current ring dword
                     // not yet written (pos mod 4 of them, low bytes first)
  bool cr[G];        // codes / BF16: the last phrase completed a segment
  uint32_t ring, list;  // codes / BF16: LDS addresses of the rings, the flush list
  uint32_t rmap;        // codes / BF16, ORD: LDS address of each tile row's matrix
                        // row times cols
  float acc[G][NB];
  // stream
  uint32_t p_end, wb, wa, ra, last8;
  uint4 next;
  uint4 *win4;
  __amdgpu_buffer_rsrc_t out_rsrc;

  __device__ __forceinline__ Tile(const Args2 &a_, uint32_t c_, uint32_t lane_, char *wave_lds)
      : a(a_), lane(lane_), c(c_) {
    const uint32_t b = c / a.NT;
    tcol = c - b * a.NT;
    r0 = b * TR;
    c0 = tcol * a.TC;
    rows = min(TR, a.rows - r0);
    cols = min(a.TC, a.cols - c0);
    nb = int(a.batch);  // <= NB; rows nb .. NB - 1 are zero activations
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const uint32_t s = g * kWave + lane;
      valid[g] = s < rows;
      x[g] = a.chunk_state[size_t(c) * TR + s];
    }
    const uint32_t p = as_const(a.chunk_off)[c];
    p_end = as_const(a.chunk_off)[c + 1];
    last8 = min(a.padded_words - 8, p_end & ~7u);
    win4 = reinterpret_cast<uint4 *>(wave_lds);
    wb = p & ~7u;
    wa = uniform(lds_addr(win4));
    ra = wa + 2 * (p - wb);
    win4[lane] = load_words(a.words, wb + 8 * lane, last8);
    win4[kHalf2 / 8 + lane] = load_words(a.words, wb + kHalf2 + 8 * lane, last8);
    if (MODE == kGemv2 && NB == 1) {
      // batch 1: record j holds the activations of columns j .. j + 3 (zero
      // past the tile row), so a phrase at column j reads 8 aligned bytes at
      // 8 j; records cols .. cols + 3 (all zero) are read by states whose
      // segment is done (or, on a damaged stream, overshot by up to 3)
      u32x2 *rec = reinterpret_cast<u32x2 *>(wave_lds + kWin2 * 2);
      const uint16_t *xr = a.x + c0;
      for (uint32_t j = lane; j < cols + 4; j += kWave) {
        uint32_t v[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = j + e < cols ? xr[j + e] : 0u;
        rec[j] = u32x2{v[0] | (v[1] << 16), v[2] | (v[3] << 16)};
      }
      const uint32_t x0 = uniform(lds_addr(rec));
#pragma unroll
      for (int g = 0; g < G; ++g) {
        pos[g] = x0;
        acc[g][0] = 0.0f;
      }
      end = x0 + 8 * cols;
      ring = x0 + rec_bytes(a.TC);  // the compaction scratch (kWave x 16 bytes)
    } else if (MODE == kGemv2) {
      // batch NB >= 2: pair table T[p] (4 NQ bytes at 4 NQ p), T[p][b] =
      // (x[b][p], x[b][p + 1]) as a BF16 pair, zero past the tile row and
      // for padded batch rows; a phrase at column p reads T[p] and T[p + 2]
      // (aligned 4 NQ-byte reads), and finished states read from T[cols]
      // on (up to T[cols + 6] on a damaged stream).  At batch 8 the table
      // has two halves, rows 0-3 and rows 4-7, each of 16-byte entries:
      // lanes read nearby columns, and 16-byte entries repeat the LDS banks
      // every 16 columns instead of 8, so fewer reads meet in a bank
      // (180 -> 170 us on the 8192 x 28672 matrix)
      uint32_t *tp = reinterpret_cast<uint32_t *>(wave_lds + kWin2 * 2);
      const uint32_t half = (a.TC + 8) * NQ;
      if (((reinterpret_cast<uintptr_t>(a.x) | (size_t(a.cols) * 2) | (size_t(c0) * 2)) & 15) ==
          0) {
        // 16-byte aligned rows: an item is 8 columns of one batch row, one
        // 16-byte load and the next column's value giving the 8 columns'
        // pairs (batch 8 on 8192 x 28672: 159 -> 157 us against one 2-byte
        // load per value)
        const uint32_t groups = (a.TC + 8 + 7) / 8;
        for (uint32_t it = lane; it < groups * NB; it += kWave) {
          const uint32_t bb = it / groups, p0 = 8 * (it % groups);
          uint32_t w[9];
#pragma unroll
          for (int k = 0; k < 9; ++k) w[k] = 0;
          if (bb < uint32_t(nb)) {
            const uint16_t *xr = a.x + size_t(bb) * a.cols + c0;
            if (p0 + 8 <= cols) {
              const uint4 v = *reinterpret_cast<const uint4 *>(xr + p0);
              w[0] = v.x & 0xFFFFu; w[1] = v.x >> 16; w[2] = v.y & 0xFFFFu; w[3] = v.y >> 16;
              w[4] = v.z & 0xFFFFu; w[5] = v.z >> 16; w[6] = v.w & 0xFFFFu; w[7] = v.w >> 16;
              w[8] = p0 + 8 < cols ? xr[p0 + 8] : 0u;
            } else {
#pragma unroll
              for (int k = 0; k < 9; ++k) w[k] = p0 + k < cols ? xr[p0 + k] : 0u;
            }
          }
          const uint32_t base = (bb / NQ) * half + bb % NQ;
#pragma unroll
          for (int k = 0; k < 8; ++k)
            if (p0 + k < a.TC + 8) tp[base + (p0 + k) * NQ] = w[k] | (w[k + 1] << 16);
        }
      } else {
        for (uint32_t e = lane; e < (a.TC + 8) * NB; e += kWave) {
          const uint32_t r = e % half, p = r / NQ, bb = (e / half) * NQ + r % NQ;
          uint32_t v = 0;
          if (bb < uint32_t(nb)) {
            const uint16_t *xr = a.x + size_t(bb) * a.cols + c0;
            v = (p < cols ? xr[p] : 0u) | ((p + 1 < cols ? uint32_t(xr[p + 1]) : 0u) << 16);
          }
          tp[e] = v;
        }
      }
      const uint32_t x0 = uniform(lds_addr(tp));
#pragma unroll
      for (int g = 0; g < G; ++g) {
        pos[g] = x0;
#pragma unroll
        for (int bb = 0; bb < NB; ++bb) acc[g][bb] = 0.0f;
      }
      end = x0 + 4 * NQ * cols;
      qstride = 4 * half;
    } else {
      ring = uniform(lds_addr(wave_lds + kWin2 * 2));
      list = ring + TR * kRing;
      rmap = list + TR * 8;
#pragma unroll
      for (int g = 0; g < G; ++g) {
        const uint32_t s = g * kWave + lane;
        const uint32_t orow = ORD && valid[g] ? out_row(a, r0 + s) : r0 + s;
        pos[g] = 0;
        rr[g] = ring + s * kRing;
        cr[g] = false;
        pend[g] = 0;
        srow[g] = MODE == kBf16_2 && valid[g] ? bf16_at(a.scale, orow) : 0.0f;
        if (ORD) *lds_ptr<uint32_t>(rmap + 4 * s) = valid[g] ? orow * a.cols : 0u;
      }
      end = cols;
      const uint32_t span = (rows - 1) * a.cols + cols;  // elements from the tile origin
      if (MODE == kCodes2)
        out_rsrc = __builtin_amdgcn_make_buffer_rsrc(a.codes + size_t(r0) * a.cols + c0, 0,
                                                     int(span), kBufferFlags);
      else
        out_rsrc = __builtin_amdgcn_make_buffer_rsrc(a.wout + size_t(r0) * a.cols + c0, 0,
                                                     int(2 * span), kBufferFlags);
    }
    __builtin_amdgcn_s_waitcnt(0);
    next = load_words(a.words, wb + kWin2 + 8 * lane, last8);
  }

  __device__ __forceinline__ void slide() {
    if (ra - wa >= 2 * kHalf2) {
      const uint4 keep = win4[kHalf2 / 8 + lane];
      win4[lane] = keep;
      win4[kHalf2 / 8 + lane] = next;
      wb += kHalf2;
      ra -= 2 * kHalf2;
      next = load_words(a.words, wb + kWin2 + 8 * lane, last8);
    }
  }

  // Activation operands per phrase: one per batch row (GEMV), else unused.
  static constexpr int NX = MODE == kGemv2 ? NB : 1;

  // The activations at state g's column, four per batch row (GEMV).
  __device__ __forceinline__ void read_x(int g, u32x2 (&xv)[NX]) {
    if (NB == 1) {
      xv[0] = *lds_ptr<const u32x2>(pos[g]);  // the column's record, 8-byte aligned
      return;
    }
    // T[p] and T[p + 2]: xv[b] = {pair (p, p + 1), pair (p + 2, p + 3)} of row b
    uint32_t lo[NB], hi[NB];
    if (NB == 2) {
      const u32x2 v0 = *lds_ptr<const u32x2>(pos[g]), v1 = *lds_ptr<const u32x2>(pos[g] + 16);
      lo[0] = v0.x; lo[1 % NB] = v0.y; hi[0] = v1.x; hi[1 % NB] = v1.y;
    } else {
#pragma unroll
      for (int q = 0; q < NB / 4; ++q) {
        const u32x4 v0 = *lds_ptr<const u32x4>(pos[g] + qstride * q);
        const u32x4 v1 = *lds_ptr<const u32x4>(pos[g] + 32 + qstride * q);
        lo[(4 * q) % NB] = v0.x; lo[(4 * q + 1) % NB] = v0.y;
        lo[(4 * q + 2) % NB] = v0.z; lo[(4 * q + 3) % NB] = v0.w;
        hi[(4 * q) % NB] = v1.x; hi[(4 * q + 1) % NB] = v1.y;
        hi[(4 * q + 2) % NB] = v1.z; hi[(4 * q + 3) % NB] = v1.w;
      }
    }
#pragma unroll
    for (int bb = 0; bb < NX; ++bb) xv[bb] = u32x2{lo[bb], hi[bb]};
  }

  // es: state half (.x high half = the position step in this kernel's units),
  // ev: value half (BF16 pairs, or the codes).
  // The entry of bucket address ba (state half; the value half unless PK).
  __device__ __forceinline__ void fetch(uint32_t ba, u32x2 &es, u32x2 &ev) {
    es = state_half(ba);
    if (!PK) ev = value_of(ba);
  }
  __device__ __forceinline__ uint32_t update(uint32_t xs, u32x2 es) {
    return PK ? state_update_pk(xs, es.x) : state_update(xs, es.x, es.y);
  }
  // The phrase's values from a packed entry: BF16 pairs (GEMV; E4M3 codes
  // converted in hardware, whose fp32 values are exact in BF16) or the codes.
  __device__ __forceinline__ u32x2 values(u32x2 es, u32x2 ev) {
    if (!PK) return ev;
    if (MODE != kGemv2) return u32x2{es.y, 0u};
    const float2v lo = __builtin_amdgcn_cvt_pk_f32_fp8(static_cast<int>(es.y), false);
    const float2v hi = __builtin_amdgcn_cvt_pk_f32_fp8(static_cast<int>(es.y), true);
    return u32x2{__builtin_amdgcn_perm(__float_as_uint(lo.y), __float_as_uint(lo.x), 0x07060302u),
                 __builtin_amdgcn_perm(__float_as_uint(hi.y), __float_as_uint(hi.x), 0x07060302u)};
  }

  // Use state g's phrase: its products with the activations (GEMV) or its
  // codes into the row's ring; then the state's position moves past it.
  __device__ __forceinline__ void use(int g, u32x2 es, u32x2 ev, const u32x2 (&xv)[NX]) {
    const uint32_t step = PK ? ((es.x >> 16) & 7u) << kUnitShift : es.x >> 16;
    if (MODE == kGemv2) {
#pragma unroll
      for (int bb = 0; bb < NX; ++bb)
        acc[g][bb] = dot2_bf16(ev.y, xv[bb].y, dot2_bf16(ev.x, xv[bb].x, acc[g][bb]));
    } else {
      // the phrase's codes (ev.x, zero past its length) after the state's
      // pending ones; a completed dword goes to the row's ring with an
      // aligned 4-byte write, the rest stays pending (unaligned LDS writes
      // were slower: codes 232 -> 203 us on 8192 x 28672).  Codes past the
      // segment's end start the next segment's first dword, which is written
      // only in a later step, after this step's flush has read the ring.
      const uint32_t q = pos[g] & (kSeg - 1), o = q & 3;
      const uint32_t lo = pend[g] | (ev.x << (8 * o));
      const uint32_t hi = o ? ev.x >> (32 - 8 * o) : 0u;
      if (o + step >= 4) {
        *lds_ptr<uint32_t>(rr[g] + (q & ~3u)) = lo;
        pend[g] = hi;
      } else {
        pend[g] = lo;
      }
      cr[g] = q + step >= kSeg;
    }
    pos[g] += step;
  }

  // One step (G = 1, no pipeline).  MASKED: only states whose segment is not
  // complete take part (else every state does).
  template <bool MASKED>
  __device__ __forceinline__ void step(const bool (&act)[G]) {
    slide();
    u32x2 es[G], ev[G];
    uint32_t ba[G];
    u32x2 xv[G][NX];
#pragma unroll
    for (int g = 0; g < G; ++g)
      if (!MASKED || act[g]) {
        ba[g] = bucket_addr(x[g]);
        es[g] = state_half(ba[g]);
      }
    if (MODE == kGemv2) {
#pragma unroll
      for (int g = 0; g < G; ++g)
        if (!MASKED || act[g]) read_x(g, xv[g]);
    }
    if (!PK) {
#pragma unroll
      for (int g = 0; g < G; ++g)
        if (!MASKED || act[g]) ev[g] = value_of(ba[g]);
    }
#pragma unroll
    for (int g = 0; g < G; ++g)
      if (!MASKED || act[g]) x[g] = update(x[g], es[g]);
    // renormalise in ascending state order (state g * 64 + lane)
    uint64_t need[G];
    uint32_t word[G];
    uint32_t r = ra;
#pragma unroll
    for (int g = 0; g < G; ++g) {
      need[g] = __builtin_amdgcn_ballot_w64((!MASKED || act[g]) && x[g] < 0x10000u);
      const uint32_t below = __builtin_amdgcn_mbcnt_hi(
          uint32_t(need[g] >> 32), __builtin_amdgcn_mbcnt_lo(uint32_t(need[g]), 0u));
      word[g] = lds_read_u16(r + 2 * below);
      r = add_twice(r, static_cast<uint32_t>(__popcll(need[g])));
    }
#pragma unroll
    for (int g = 0; g < G; ++g) {
      if (!MASKED || act[g]) use(g, es[g], values(es[g], ev[g]), xv[g]);
      else cr[g] = false;
    }
#pragma unroll
    for (int g = 0; g < G; ++g) x[g] = renorm_lanes(need[g], x[g], word[g]);
    ra = r;
    flush();
  }

  // The value half of a bucket: BF16 values (GEMV) or the four codes.
  __device__ __forceinline__ u32x2 value_of(uint32_t ba) {
    if (MODE == kGemv2) return value_half(ba);
    return u32x2{*lds_ptr<const uint32_t>((ba >> 1) + kCodesHalf),
                 0u};
  }

  // --- codes / BF16 output --------------------------------------------------
  // Store n (<= 8) codes of tile row `row` from column col0 on: `d` holds 8
  // codes (from the row's ring).  A whole 8-code piece goes out as one 8-byte
  // (codes) or 16-byte (BF16) store, so the four lanes of a segment write 32
  // or 64 contiguous bytes; a shorter piece, which only a row's last segment
  // has, element by element.
  __device__ __forceinline__ void store_piece(uint32_t row, uint32_t col0, u32x2 d, uint32_t n,
                                              float sc) {
    const uint32_t idx = row * a.cols + col0;  // < 2^31 (checked at launch)
    // ORD: the element offset of the piece in the whole matrix (< 2^32),
    // written through a global address
    const size_t at = ORD ? size_t(*lds_ptr<const uint32_t>(rmap + 4 * row)) + c0 + col0 : 0;
    if (MODE == kCodes2) {
      if (ORD) {
        uint8_t *dst = a.codes + at;
        if (n >= kCPL) {
          *reinterpret_cast<u32x2u *>(dst) = d;
        } else {
          for (uint32_t e = 0; e < n; ++e) dst[e] = static_cast<uint8_t>(d[e / 4] >> (8 * (e % 4)));
        }
      } else if (n >= kCPL) {
        __builtin_amdgcn_raw_buffer_store_b64(d, out_rsrc, idx, 0, 0);
      } else {
        for (uint32_t e = 0; e < n; ++e)
          __builtin_amdgcn_raw_buffer_store_b8(static_cast<uint8_t>(d[e / 4] >> (8 * (e % 4))),
                                               out_rsrc, idx + e, 0, 0);
      }
      return;
    }
    uint32_t o[4];
#pragma unroll
    for (int w = 0; w < 2; ++w) {
      float v0, v1, v2, v3;
      if (a.fmt == kFmtInt8) {
        v0 = static_cast<float>(static_cast<int8_t>(d[w]));
        v1 = static_cast<float>(static_cast<int8_t>(d[w] >> 8));
        v2 = static_cast<float>(static_cast<int8_t>(d[w] >> 16));
        v3 = static_cast<float>(static_cast<int8_t>(d[w] >> 24));
      } else {
        // E4M3FN to fp32 in hardware, two codes at a time
        const float2v lo = __builtin_amdgcn_cvt_pk_f32_fp8(static_cast<int>(d[w]), false);
        const float2v hi = __builtin_amdgcn_cvt_pk_f32_fp8(static_cast<int>(d[w]), true);
        v0 = lo.x; v1 = lo.y; v2 = hi.x; v3 = hi.y;
      }
      // s * v is exact in fp32; one rounding to BF16
      o[2 * w] = pack_bf16(sc * v0, sc * v1);
      o[2 * w + 1] = pack_bf16(sc * v2, sc * v3);
    }
    if (ORD) {
      uint16_t *dst = a.wout + at;
      if (n >= kCPL) {
        *reinterpret_cast<u32x4u *>(dst) = u32x4{o[0], o[1], o[2], o[3]};
      } else {
        for (uint32_t e = 0; e < n; ++e) dst[e] = static_cast<uint16_t>(o[e / 2] >> (16 * (e % 2)));
      }
    } else if (n >= kCPL) {
      __builtin_amdgcn_raw_buffer_store_b128(u32x4{o[0], o[1], o[2], o[3]}, out_rsrc, 2 * idx, 0,
                                             0);
    } else {
      for (uint32_t e = 0; e < n; ++e)
        __builtin_amdgcn_raw_buffer_store_b16(static_cast<uint16_t>(o[e / 2] >> (16 * (e % 2))),
                                              out_rsrc, 2 * (idx + e), 0, 0);
    }
  }

  // Write the list's n segments (entries: tile row | segment << 16, the row
  // scale), four lanes per segment.
  __device__ __forceinline__ void write_list(uint32_t n) {
    for (uint32_t k = 0; k < n; k += kWave / 4) {
      const uint32_t e = k + lane / 4, part = lane % 4;
      if (e < n) {
        const u32x2 ent = *lds_ptr<const u32x2>(list + 8 * e);
        const uint32_t row = ent.x & 0xFFFFu, col0 = (ent.x >> 16) * kSeg + kCPL * part;
        const uint32_t src = ring + row * kRing + kCPL * part;
        const uint32_t lim = end > col0 ? end - col0 : 0u;
        store_piece(row, col0, *lds_ptr<const u32x2>(src), min(lim, kCPL),
                    __uint_as_float(ent.y));
      }
    }
  }

  // After a step: the segments its phrases completed go out.
  __device__ __forceinline__ void flush() {
    if (MODE == kGemv2) return;
    uint32_t n = 0;
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const uint64_t m = __builtin_amdgcn_ballot_w64(cr[g]);
      if (m == 0) continue;
      if (cr[g]) {
        const uint32_t rank = __builtin_amdgcn_mbcnt_hi(
            uint32_t(m >> 32), __builtin_amdgcn_mbcnt_lo(uint32_t(m), 0u));
        // the segment just completed: the one before pos
        const uint32_t seg = (pos[g] >> kSegShift) - 1;
        *lds_ptr<u32x2>(list + 8 * (n + rank)) =
            u32x2{(g * kWave + lane) | (seg << 16), __float_as_uint(srow[g])};
      }
      n += static_cast<uint32_t>(__popcll(m));
    }
    if (n == 0) return;
    write_list(n);
#pragma unroll
    for (int g = 0; g < G; ++g) cr[g] = false;
  }

  // At the end of the tile: every row's last, partial segment.
  __device__ __forceinline__ void flush_tail() {
    if (MODE == kGemv2 || (end & (kSeg - 1)) == 0) return;
    // the codes still pending (end not a multiple of 4) into the ring
#pragma unroll
    for (int g = 0; g < G; ++g)
      if (valid[g] && (pos[g] & 3))
        *lds_ptr<uint32_t>(rr[g] + ((pos[g] & (kSeg - 1)) & ~3u)) = pend[g];
    uint32_t n = 0;
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const uint64_t m = __builtin_amdgcn_ballot_w64(valid[g]);
      if (valid[g]) {
        const uint32_t rank = __builtin_amdgcn_mbcnt_hi(
            uint32_t(m >> 32), __builtin_amdgcn_mbcnt_lo(uint32_t(m), 0u));
        *lds_ptr<u32x2>(list + 8 * (n + rank)) =
            u32x2{(g * kWave + lane) | ((end >> kSegShift) << 16), __float_as_uint(srow[g])};
      }
      n += static_cast<uint32_t>(__popcll(m));
    }
    write_list(n);
  }

  // --- pipelined full steps -------------------------------------------------
  // A state's step has three parts: I (read its table entry and, at batch 1,
  // its activations), U (update, ballot, read its stream word and, at batches
  // 2-8, its activations) and F (use the phrase, merge the word).  The lane's G states are offset by fractions of a step so that
  // every I -> U and U -> F latency is covered by other states' work, while
  // the words are still taken in the coder's order (step t: states 0..G-1,
  // then step t + 1).  With G = 4 a step is
  //   F0 I0' U2 | F1 I1' U3 | F2 I2' U0' | F3 I3' U1'      (' = step t + 1)
  // and with G = 2   F0 I0' U1 | F1 I1' U0'.
  u32x2 pes[G], pev[G];
  u32x2 pxv[G][NX];
  uint64_t pneed[G];
  uint32_t pword[G];
  bool pact[G];

  // MASK: a state whose segment is done (or whose row lies past the layer)
  // takes the identity entry: its state, position and sum stay as they are
  // and it reads no word (GEMV at batch 1 only: its activation read stays
  // inside the records).
  template <int g, bool MASK>
  __device__ __forceinline__ void p_issue() {
    uint32_t ba = bucket_addr(x[g]);
    if (MASK) {
      pact[g] = valid[g] && pos[g] < end;
      ba = pact[g] ? ba : kIdentity2;
    }
    pes[g] = state_half(ba);
    // batch 1 reads its activation record here; batches 2-8 at U (below)
    if (MODE == kGemv2 && NB == 1) read_x(g, pxv[g]);
    if (!PK) pev[g] = value_of(ba);
  }
  template <int g, bool MASK>
  __device__ __forceinline__ void p_update() {
    // a packed identity entry does not leave the state as it is: a finished
    // state keeps its value
    // batches 2-8: the activations are read one part later than the entry,
    // so at most two states' activations are held at once (190 instead of
    // 221 VGPRs; batch 8 on 8192 x 28672: 172.5 -> 166.7 us); the state's
    // position changes only in its F part, so the address is the same
    if (MODE == kGemv2 && NB > 1) read_x(g, pxv[g]);
    const uint32_t xn = update(x[g], pes[g]);
    x[g] = PK && MASK ? (pact[g] ? xn : x[g]) : xn;
    pneed[g] = __builtin_amdgcn_ballot_w64(x[g] < 0x10000u);
    const uint32_t below = __builtin_amdgcn_mbcnt_hi(
        uint32_t(pneed[g] >> 32), __builtin_amdgcn_mbcnt_lo(uint32_t(pneed[g]), 0u));
    pword[g] = lds_read_u16(ra + 2 * below);
    ra = add_twice(ra, static_cast<uint32_t>(__popcll(pneed[g])));
  }
  template <int g>
  __device__ __forceinline__ void p_finish() {
    use(g, pes[g], values(pes[g], pev[g]), pxv[g]);
    x[g] = renorm_lanes(pneed[g], x[g], pword[g]);
  }

  // One pipelined step: F(t) of every state, I(t + 1) after it, U of the
  // next in the coder's order.
  template <bool MASK>
  __device__ __forceinline__ void p_step() {
    constexpr int H = G / 2;
    // the window moves between steps (a step reads at most TR words, half a
    // window)
    slide();
    p_finish<0>();
    p_issue<0, MASK>();
    p_update<H, MASK>();
    p_finish<1 % G>();
    p_issue<1 % G, MASK>();
    if (G == 4) {
      p_update<3 % G, MASK>();
      p_finish<2 % G>();
      p_issue<2 % G, MASK>();
      p_update<0, MASK>();
      p_finish<3 % G>();
      p_issue<3 % G, MASK>();
      p_update<1 % G, MASK>();
    } else {
      p_update<0, MASK>();
    }
    flush();
  }

  // T steps, G = 2 or 4.  Without MASK every state takes part in all T (and
  // the wave lowers its issue priority through the steps so that waves that
  // are behind catch up); with MASK, T bounds the steps and the loop ends once
  // every segment is done.
  // COMPACT (batch-1 GEMV): leave the masked steps, at a step boundary,
  // once at most 64 states are still active (compact_finish takes over).
  template <bool MASK, bool COMPACT = false>
  __device__ __forceinline__ void run_pipelined(uint32_t T) {
    if (T == 0) return;
    constexpr int H = G / 2;
    slide();
    p_issue<0, MASK>();
    p_issue<1 % G, MASK>();
    if (G == 4) {
      p_issue<2 % G, MASK>();
      p_issue<3 % G, MASK>();
    }
    p_update<0, MASK>();
    if (G == 4) p_update<1 % G, MASK>();
    const uint32_t n = T - 1;
    if (MASK) {
      for (uint32_t t = 0; t < n; ++t) {
        p_step<true>();
        uint32_t n_act = 0;
#pragma unroll
        for (int g = 0; g < G; ++g)
          n_act += static_cast<uint32_t>(__popcll(__builtin_amdgcn_ballot_w64(pact[g])));
        // nothing of step t + 1 is pending but identity steps
        if (n_act == 0) return;
        // else complete step t + 1 (below) and hand over
        if (COMPACT && n_act <= kWave) break;
      }
    } else {
      uint32_t t = 0;
#pragma unroll 1
      for (uint32_t q = 0; q < 4; ++q) {
        set_prio_down(q);
        const uint32_t stop = q == 0 ? n / 2 : q == 1 ? n - n / 4 : q == 2 ? n - n / 16 : n;
        for (; t < stop; ++t) {
          asm("" : "+s"(t));
          p_step<false>();
        }
      }
    }
    slide();
    p_finish<0>();
    p_update<H, MASK>();
    p_finish<1 % G>();
    if (G == 4) {
      p_update<3 % G, MASK>();
      p_finish<2 % G>();
      p_finish<3 % G>();
    }
    flush();
  }

  __device__ __forceinline__ void run() {
    const bool all[G] = {};
    bool full = rows == TR;
    // Every state needs at least cols / 4 phrases, so in a full tile no state
    // finishes before step cols / 4: those steps need no masks.
    const uint32_t t1 = full ? cols / 4 : 0;
    if (G >= 2) {
      run_pipelined<false>(t1);
      // every phrase holds at least one code: at most cols steps in all (the
      // bound also ends the loop on a damaged stream)
      if (MODE == kGemv2 && NB == 1) {
        run_pipelined<true, true>(cols - t1);
        compact_finish();
        return;
      }
      run_pipelined<true>(cols - t1);
      flush_tail();
      finish();
      return;
    }
    // G = 1: one state per lane, steps one after the other
    for (uint32_t t = 0; t < t1; ++t) step<false>(all);
    for (uint32_t t = t1; t < cols; ++t) {
      bool act[G];
      bool any = false;
#pragma unroll
      for (int g = 0; g < G; ++g) {
        act[g] = valid[g] && pos[g] < end;
        any |= act[g];
      }
      if (__builtin_amdgcn_ballot_w64(any) == 0) break;
      step<true>(act);
    }
    flush_tail();
    finish();
  }

  // Batch-1 GEMV, after the masked steps: if states are still active, they
  // are at most 64.  Finished states write their sums and are checked; the
  // active ones move, in ascending state order (the order in which the coder
  // hands out words), to one state per lane through the wavefront's scratch,
  // and finish with single-state steps: a quarter of a four-state step.
  __device__ __forceinline__ void compact_finish() {
    bool act[G];
    uint32_t n_act = 0;
#pragma unroll
    for (int g = 0; g < G; ++g) {
      act[g] = valid[g] && pos[g] < end;
      n_act += static_cast<uint32_t>(__popcll(__builtin_amdgcn_ballot_w64(act[g])));
    }
    if (n_act == 0 || n_act > kWave) {  // done, or the step bound hit (damaged stream)
      finish();
      return;
    }
    bool bad = false;
    const uint32_t scr = ring;  // the scratch: kWave x 16 bytes after the records
    uint32_t base = 0;
#pragma unroll
    for (int g = 0; g < G; ++g) {
      if (valid[g] && !act[g]) {
        write_sum(g * kWave + lane, acc[g][0]);
        bad |= pos[g] != end;
      }
      bad |= !act[g] && x[g] != 0x10000u;
      const uint64_t m = __builtin_amdgcn_ballot_w64(act[g]);
      const uint32_t rank = base + __builtin_amdgcn_mbcnt_hi(
          uint32_t(m >> 32), __builtin_amdgcn_mbcnt_lo(uint32_t(m), 0u));
      // (four 4-byte writes: a vector built from the state arrays sent them
      // to private memory)
      const uint32_t xa = x[g], pa = pos[g], sa = __float_as_uint(acc[g][0]);
      if (act[g]) {
        const uint32_t d = scr + 16 * rank;
        *lds_ptr<uint32_t>(d) = xa;
        *lds_ptr<uint32_t>(d + 4) = pa;
        *lds_ptr<uint32_t>(d + 8) = sa;
        *lds_ptr<uint32_t>(d + 12) = g * kWave + lane;
      }
      base += static_cast<uint32_t>(__popcll(m));
    }
    const bool on = lane < n_act;
    u32x4 v = u32x4{0x10000u, end, 0u, 0u};
    if (on) v = *lds_ptr<const u32x4>(scr + 16 * lane);
    uint32_t x1 = v.x, p1 = v.y;
    float s1 = __uint_as_float(v.z);
    // every active state advances at least one column per step
    for (uint32_t t = 0; t < cols; ++t) {
      const bool a1 = on && p1 < end;
      if (__builtin_amdgcn_ballot_w64(a1) == 0) break;
      slide();
      const uint32_t ba = a1 ? bucket_addr(x1) : kIdentity2;
      const u32x2 es = state_half(ba);
      const u32x2 xv = *lds_ptr<const u32x2>(p1);  // records up to cols + 3 exist
      const u32x2 ev = value_half(ba);
      x1 = state_update(x1, es.x, es.y);
      const uint64_t need = __builtin_amdgcn_ballot_w64(x1 < 0x10000u);
      const uint32_t below = __builtin_amdgcn_mbcnt_hi(
          uint32_t(need >> 32), __builtin_amdgcn_mbcnt_lo(uint32_t(need), 0u));
      const uint32_t word = lds_read_u16(ra + 2 * below);
      ra = add_twice(ra, static_cast<uint32_t>(__popcll(need)));
      s1 = dot2_bf16(ev.y, xv.y, dot2_bf16(ev.x, xv.x, s1));
      p1 += es.x >> 16;
      x1 = renorm_lanes(need, x1, word);
    }
    if (on) {
      write_sum(v.w, s1);
      bad |= x1 != 0x10000u || p1 != end;
    }
    bad |= wb + (ra - wa) / 2 != p_end;
    if (__builtin_amdgcn_ballot_w64(bad) != 0 && lane == 0) atomicOr(a.status, 1);
  }

  // Batch-1 GEMV: the sum of tile row r (0 .. TR - 1) of this tile.
  __device__ __forceinline__ void write_sum(uint32_t r, float sum) {
    uint32_t row = r0 + r;
    if (a.NT == 1) {
      row = out_row(a, row);
      const float bias = a.bias ? bf16_to_f32(a.bias[row]) : 0.0f;
      a.y[row] = bf16_to_f32(a.scale[row]) * sum + bias;
    } else {
      a.ws[size_t(tcol) * a.rows + row] = sum;
    }
  }

  __device__ __forceinline__ void finish() {
    if (MODE == kGemv2) {
#pragma unroll
      for (int g = 0; g < G; ++g) {
        if (!valid[g]) continue;
        const uint32_t row = r0 + g * kWave + lane;
        const uint32_t orow = a.NT == 1 ? out_row(a, row) : row;
#pragma unroll
        for (int bb = 0; bb < NB; ++bb) {
          if (bb >= nb) continue;
          if (a.NT == 1) {
            const float bias = a.bias ? bf16_to_f32(a.bias[orow]) : 0.0f;
            a.y[size_t(bb) * a.rows + orow] = bf16_to_f32(a.scale[orow]) * acc[g][bb] + bias;
          } else {
            a.ws[(size_t(bb) * a.NT + tcol) * a.rows + row] = acc[g][bb];
          }
        }
      }
    }
    bool bad = wb + (ra - wa) / 2 != p_end;
#pragma unroll
    for (int g = 0; g < G; ++g) bad |= x[g] != 0x10000u || (valid[g] && pos[g] != end);
    if (__builtin_amdgcn_ballot_w64(bad) != 0 && lane == 0) atomicOr(a.status, 1);
  }
};

constexpr uint32_t table_bytes2(int mode, bool pk) {
  return pk ? kTablePacked2 : (mode == kGemv2 ? kTableBytes2 : kTableCodes2);
}

// Stage the layer's phrase table in LDS (address 0); returns its base.
template <int MODE, int NB, bool PK>
__device__ __forceinline__ char *stage_table2(const Args2 &a) {
  extern __shared__ uint4 dyn2[];
  // the phrase table at LDS address 0 (no static LDS in this kernel), the
  // position step in this kernel's units: record bytes (GEMV at batch 1),
  // activation bytes (GEMV), codes (codes and BF16 output)
  char *tab = reinterpret_cast<char *>(dyn2);
  // kStage of a thread's entries are loaded before any is written, so their
  // latencies overlap (one round for blocks of 512 threads or more)
  constexpr uint32_t kStage = 8;
  for (uint32_t i0 = threadIdx.x; i0 < kBuckets; i0 += kStage * blockDim.x) {
    uint4 e[kStage];
    uint32_t c4[kStage];
#pragma unroll
    for (uint32_t u = 0; u < kStage; ++u) {
      const uint32_t i = i0 + u * blockDim.x;
      if (i < kBuckets) {
        e[u] = a.lut[i];
        c4[u] = MODE != kGemv2 ? a.codes4[i] : 0u;
      }
    }
#pragma unroll
    for (uint32_t u = 0; u < kStage; ++u) {
      const uint32_t i = i0 + u * blockDim.x;
      if (i >= kBuckets) continue;
      const uint32_t len = e[u].x >> 17;
      if (PK) {
        const uint32_t F = 65536u - (e[u].x & 0xFFFFu);  // F < 2^16: K > 1
        *reinterpret_cast<u32x2 *>(tab + 8 * i) = u32x2{F | ((e[u].y | len) << 16), c4[u]};
      } else {
        const uint32_t step =
            MODE == kGemv2 ? (NB == 1 ? 8 * len : 4 * (NB < 4 ? NB : 4) * len) : len;
        *reinterpret_cast<u32x2 *>(tab + 8 * i) = u32x2{(e[u].x & 0xFFFFu) | (step << 16), e[u].y};
        if (MODE == kGemv2)
          *reinterpret_cast<u32x2 *>(tab + kValHalf + 8 * i) = u32x2{e[u].z, e[u].w};
        else
          *reinterpret_cast<uint32_t *>(tab + kCodesHalf + 4 * i) = c4[u];
      }
    }
  }
  if (threadIdx.x == 0) {
    *reinterpret_cast<u32x2 *>(tab + kIdentity2) = u32x2{0u, 0u};
    if (PK) {
    } else if (MODE == kGemv2)
      *reinterpret_cast<u32x2 *>(tab + kValHalf + kIdentity2) = u32x2{0u, 0u};
    else
      *reinterpret_cast<uint32_t *>(tab + kCodesHalf + kIdentity2 / 2) = 0u;
  }
  __syncthreads();
  return tab;
}

// Block bid of nblocks on layer a: its wavefronts decode their tiles.
template <int G, int MODE, int NB, bool PK, bool ORD>
__device__ __forceinline__ void run_tiles2(const Args2 &a, char *tab, uint32_t bid,
                                           uint32_t nblocks) {
  const uint32_t nw = blockDim.x / kWave, wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
  char *mine = tab + table_bytes2(MODE, PK) + size_t(wave) * a.wave_lds;
  // chunks strided over the layer (block bid, wave w: bid + w * nblocks, ...):
  // a tile's length is its longest row's, so tiles of one row band run long
  // or short together; spreading each block's tiles over all bands evens the
  // work of the compute units (batch-1 GEMV on 8192 x 28672: 67.0 -> 64.2 us)
  for (uint32_t c = uniform(wave * nblocks + bid); c < a.n_chunks; c += nblocks * nw) {
    Tile<G, MODE, NB, PK, ORD> t(a, c, lane, mine);
    t.run();
  }
}

// The work of block `bid` of `nblocks` on layer a: stage the phrase table,
// then each wavefront decodes its chunks.
template <int G, int MODE, int NB, bool PK, bool ORD>
__device__ __forceinline__ void decode2_block(const Args2 &a, uint32_t bid, uint32_t nblocks) {
  run_tiles2<G, MODE, NB, PK, ORD>(a, stage_table2<MODE, NB, PK>(a), bid, nblocks);
}

template <int G, int MODE, int NB, bool PK, bool ORD>
__global__ __launch_bounds__(kWave * max_waves2(MODE, NB)) void decode2_kernel(Args2 a) {
  decode2_block<G, MODE, NB, PK, ORD>(a, blockIdx.x, gridDim.x);
}

// Several layers in one launch (Sec. 2.2 block-wise decompression): blocks
// [blk_end[i - 1], blk_end[i]) work on layer i (a block stages one layer's
// table); the layers share the tile height and, for the GEMV, the input.
constexpr uint32_t kMaxLayers2 = 8;
struct MultiArgs2 {
  Args2 a[kMaxLayers2];
  uint32_t blk_end[kMaxLayers2];
  uint32_t n;
};

template <int G, int MODE, int NB, bool PK, bool ORD>
__global__ __launch_bounds__(kWave * max_waves2(MODE, NB)) void decode2_multi_kernel(MultiArgs2 m) {
  uint32_t i = 0, b0 = 0;
  while (i + 1 < m.n && blockIdx.x >= m.blk_end[i]) b0 = m.blk_end[i++];
  decode2_block<G, MODE, NB, PK, ORD>(m.a[i], blockIdx.x - b0, m.blk_end[i] - b0);
}

// Codes or BF16 of layers of several tile heights in one launch: a block
// runs its layer's tiles with the Tile of that height (the kernel holds all
// three, so registers and LDS per wavefront are those of the largest).
template <int MODE, bool PK, bool ORD>
__global__ __launch_bounds__(kWave * max_waves2(MODE, 1)) void decode2_mixed_kernel(MultiArgs2 m) {
  uint32_t i = 0, b0 = 0;
  while (i + 1 < m.n && blockIdx.x >= m.blk_end[i]) b0 = m.blk_end[i++];
  const Args2 &a = m.a[i];
  char *tab = stage_table2<MODE, 1, PK>(a);
  const uint32_t bid = blockIdx.x - b0, nb = m.blk_end[i] - b0;
  if (a.TR == 64) run_tiles2<1, MODE, 1, PK, ORD>(a, tab, bid, nb);
  else if (a.TR == 128) run_tiles2<2, MODE, 1, PK, ORD>(a, tab, bid, nb);
  else run_tiles2<4, MODE, 1, PK, ORD>(a, tab, bid, nb);
}

// Rows split over NT > 1 column tiles: y = s * (partials added in tile
// order) + bias, the partials of stored row k going to matrix row order[k].
// One block per 64 outputs (index i = batch row * rows + row, one per
// lane), kMergeParts wavefronts: wavefront p sums tiles
// [p NT / kMergeParts, (p + 1) NT / kMergeParts) in order (independent loads,
// so their latencies overlap, each a contiguous 256 bytes of the workspace),
// then the parts are added in order 0, 1, ... through LDS (deterministic).
// Each load reads 256 contiguous bytes; sixteen threads per output inside
// one wavefront read 16 bytes of each of 16 scattered segments per load and
// were slower (batch 8 on 8192 x 28672: 167.5 against 159 us).
constexpr uint32_t kMergeParts = 16;
constexpr uint32_t kMergeThreads = kWave * kMergeParts;
__device__ __forceinline__ void merge2(const Args2 &a, uint32_t blk) {
  __shared__ float part_sum[kMergeParts][kWave];
  const uint32_t lane = threadIdx.x % kWave, part = threadIdx.x / kWave;
  const uint32_t n = a.rows * a.batch;
  const uint32_t i = blk * kWave + lane;
  uint32_t row = 0;
  float sum = 0.0f;
  if (i < n) {
    const uint32_t bb = i / a.rows;
    row = i - bb * a.rows;
    const float *p = a.ws + size_t(bb) * a.NT * a.rows + row;
    const uint32_t t0 = part * a.NT / kMergeParts, t1 = (part + 1) * a.NT / kMergeParts;
    uint32_t t = t0;
    for (; t + 4 <= t1; t += 4) {
      const float v0 = p[size_t(t) * a.rows], v1 = p[size_t(t + 1) * a.rows];
      const float v2 = p[size_t(t + 2) * a.rows], v3 = p[size_t(t + 3) * a.rows];
      sum = (((sum + v0) + v1) + v2) + v3;
    }
    for (; t < t1; ++t) sum += p[size_t(t) * a.rows];
  }
  part_sum[part][lane] = sum;
  __syncthreads();
  if (part == 0 && i < n) {
    float total = part_sum[0][lane];
#pragma unroll
    for (uint32_t q = 1; q < kMergeParts; ++q) total += part_sum[q][lane];
    const uint32_t orow = out_row(a, row);
    const float bias = a.bias ? bf16_to_f32(a.bias[orow]) : 0.0f;
    a.y[i - row + orow] = bf16_to_f32(a.scale[orow]) * total + bias;
  }
}

__global__ __launch_bounds__(kMergeThreads) void merge2_kernel(Args2 a) { merge2(a, blockIdx.x); }


// Phrase table of a layer: bucket b (of kBuckets) belongs to symbol k when
// 2^(12-R) cum_k <= b < 2^(12-R) (cum_k + f_k).
__global__ __launch_bounds__(1024) void prepare2_kernel(const uint32_t *phr, const uint16_t *freq,
                                                        uint32_t K, uint32_t nq, uint32_t np,
                                                        uint32_t R, uint32_t fmt, uint4 *lut,
                                                        uint32_t *codes4, int32_t *status) {
  __shared__ uint32_t cum_s[kBuckets + 1];
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
  const uint32_t sh = 12 - R;
  for (uint32_t bkt = t; bkt < kBuckets; bkt += blockDim.x) {
    const uint32_t slot = bkt >> sh;  // in units of 2^-R
    uint32_t lo = 0, hi = K - 1;      // largest k with cum_k <= slot
    while (lo < hi) {
      const uint32_t mid = (lo + hi + 1) / 2;
      if (cum_s[mid] <= slot) lo = mid;
      else hi = mid - 1;
    }
    const uint32_t k = lo;
    const uint32_t F = uint32_t(freq[k]) << (16 - R);
    const uint32_t len = k < nq ? 4 : (k < nq + np ? 2 : 1);
    const uint32_t codes = phr[k];
    uint32_t v[4];
    for (uint32_t j = 0; j < 4; ++j) {
      const uint32_t code = (codes >> (8 * j)) & 0xFF;
      const float val = fmt == kFmtInt8 ? static_cast<float>(static_cast<int8_t>(code))
                                        : e4m3_value(code);
      v[j] = j < len ? (__float_as_uint(val) >> 16) : 0u;  // exact in BF16
    }
    lut[bkt] = make_uint4((65536u - F) | ((2 * len) << 16), cum_s[k] << (16 - R),
                          v[0] | (v[1] << 16), v[2] | (v[3] << 16));
    codes4[bkt] = codes;
  }
  if (t == 0) *status = 0;
}

Args2 make_args2(const eq_layer *L) {
  Args2 a{};
  a.lut = reinterpret_cast<const uint4 *>(L->lut);
  a.codes4 = L->lut + 4 * kBuckets;
  a.scale = L->scale;
  a.chunk_off = L->chunk_off;
  a.chunk_state = L->chunk_state;
  a.words = L->words;
  a.status = L->status;
  a.rows = L->rows;
  a.cols = L->cols;
  a.TR = L->lanes;
  a.TC = L->tile_cols;
  a.NT = (L->cols + L->tile_cols - 1) / L->tile_cols;
  a.n_chunks = L->n_chunks;
  a.padded_words = static_cast<uint32_t>(L->padded_words);
  a.fmt = L->base_format;
  a.n_syms = L->n_syms;
  a.order = L->row_order;
  return a;
}

struct Facts2 {
  int lds = 160 * 1024;
  int cus = 256;
};

Facts2 facts2() {
  static std::atomic<int> lds[64], cus[64];
  int dev = 0;
  Facts2 f;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return f;
  int l = lds[dev].load(std::memory_order_relaxed), c = cus[dev].load(std::memory_order_relaxed);
  if (l == 0) {
    if (hipDeviceGetAttribute(&l, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) != hipSuccess ||
        l <= 0)
      l = f.lds;
    if (hipDeviceGetAttribute(&c, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        c <= 0)
      c = f.cus;
    lds[dev].store(l, std::memory_order_relaxed);
    cus[dev].store(c, std::memory_order_relaxed);
  }
  f.lds = l;
  f.cus = c;
  return f;
}


// LDS per wavefront: the stream window, then (GEMV) the tile's activations:
// one 8-byte record per column at batch 1, else the rows; (codes, BF16) the
// rows' rings, the flush list and, in an ORD launch, the rows' offsets.
uint32_t wave_lds_bytes(int mode, const Args2 &a, bool ord) {
  uint32_t b = kWin2 * 2;
  if (mode != kGemv2) b += a.TR * (kRing + 8 + (ord ? 4 : 0));
  if (mode == kGemv2) {
    const uint32_t nbp = a.batch == 1 ? 1 : a.batch == 2 ? 2 : a.batch <= 4 ? 4 : 8;
    b += nbp == 1 ? rec_bytes(a.TC) + kWave * 16 : (a.TC + 8) * 4 * nbp;
  }
  return b;
}

// One block per compute unit (the table takes most of LDS), as many
// wavefronts as the chunks need for one round, at most what LDS holds.
// Wavefronts per block for layers of n[0..k-1] chunks (each layer's chunks in
// blocks of their own, a wavefront per chunk); 0 if not even one wavefront
// fits LDS.  Start from one block per compute unit (total chunks / CUs
// wavefronts) and add wavefronts until the blocks fit one round (the blocks
// that LDS lets each compute unit hold at once); when no count up to the
// limit does, take the count in [limit / 2, limit] that makes the busiest
// unit's share, ceil(blocks / CUs) x waves chunks, smallest (the larger on
// ties).
uint32_t choose_waves(const uint32_t *n, uint32_t k, uint32_t wmax, size_t tb, size_t wl,
                      const Facts2 &f) {
  while (wmax > 0 && tb + size_t(wmax) * wl > size_t(f.lds)) --wmax;
  if (wmax == 0) return 0;
  uint64_t total = 0;
  for (uint32_t i = 0; i < k; ++i) total += n[i];
  auto blocks = [&](uint32_t w) {
    uint64_t b = 0;
    for (uint32_t i = 0; i < k; ++i) b += (n[i] + w - 1) / w;
    return b;
  };
  auto slots = [&](uint32_t w) { return uint64_t(f.cus) * (size_t(f.lds) / (tb + size_t(w) * wl)); };
  uint32_t w = uint32_t(std::min<uint64_t>(std::max<uint64_t>((total + f.cus - 1) / f.cus, 1), wmax));
  while (w < wmax && blocks(w) > slots(w)) ++w;
  if (blocks(w) > slots(w)) {
    uint64_t best = ~uint64_t(0);
    for (uint32_t v = wmax; v >= 1 && v >= (wmax + 1) / 2; --v) {
      const uint64_t load = (blocks(v) + f.cus - 1) / f.cus * v;
      if (load < best) {
        best = load;
        w = v;
      }
    }
  }
  return w;
}

template <int MODE, int NB, bool PK, bool ORD>
int launch2_pk(Args2 a, hipStream_t s) {
  const Facts2 f = facts2();
  a.wave_lds = wave_lds_bytes(MODE, a, ORD);
  const size_t tb = table_bytes2(MODE, PK);
  const uint32_t waves = choose_waves(&a.n_chunks, 1, max_waves2(MODE, NB), tb, a.wave_lds, f);
  if (waves == 0) return EQ_EINVAL;
  const uint32_t blocks = (a.n_chunks + waves - 1) / waves;
  const size_t shm = tb + size_t(waves) * a.wave_lds;
  const dim3 grid(blocks), block(waves * kWave);
  switch (a.TR) {
    case 64: hipLaunchKernelGGL((decode2_kernel<1, MODE, NB, PK, ORD>), grid, block, shm, s, a); break;
    case 128: hipLaunchKernelGGL((decode2_kernel<2, MODE, NB, PK, ORD>), grid, block, shm, s, a); break;
    default: hipLaunchKernelGGL((decode2_kernel<4, MODE, NB, PK, ORD>), grid, block, shm, s, a); break;
  }
  return hipGetLastError() == hipSuccess ? EQ_OK : EQ_EHIP;
}

// The merges of a joint launch in one grid: blockIdx.y picks the layer.
// Layers of one column tile have no partials; blocks past a layer's outputs
// leave whole (before the block's barrier).
__global__ __launch_bounds__(kMergeThreads) void merge2_multi_kernel(MultiArgs2 m) {
  const Args2 &a = m.a[blockIdx.y];
  if (a.NT <= 1 || blockIdx.x * kWave >= a.rows * a.batch) return;
  merge2(a, blockIdx.x);
}

// Joint launch of m.n layers: one wavefront count for all (from the total
// chunks, LDS for the largest per-wavefront need), each layer's blocks in
// proportion to its chunks.
template <int MODE, int NB, bool PK, bool ORD, bool MIX = false>
int launch2_multi(MultiArgs2 m, hipStream_t s) {
  const Facts2 f = facts2();
  uint32_t wl = 0, n[kMaxLayers2];
  for (uint32_t i = 0; i < m.n; ++i) {
    wl = max(wl, wave_lds_bytes(MODE, m.a[i], ORD));
    n[i] = m.a[i].n_chunks;
  }
  const size_t tb = table_bytes2(MODE, PK);
  const uint32_t waves = choose_waves(n, m.n, max_waves2(MODE, NB), tb, wl, f);
  if (waves == 0) return EQ_EINVAL;
  uint32_t end = 0;
  for (uint32_t i = 0; i < m.n; ++i) {
    m.a[i].wave_lds = wl;
    end += (m.a[i].n_chunks + waves - 1) / waves;
    m.blk_end[i] = end;
  }
  const size_t shm = tb + size_t(waves) * wl;
  const dim3 grid(end), block(waves * kWave);
  if constexpr (MIX) {
    hipLaunchKernelGGL((decode2_mixed_kernel<MODE, PK, ORD>), grid, block, shm, s, m);
    return hipGetLastError() == hipSuccess ? EQ_OK : EQ_EHIP;
  }
  switch (m.a[0].TR) {
    case 64: hipLaunchKernelGGL((decode2_multi_kernel<1, MODE, NB, PK, ORD>), grid, block, shm, s, m); break;
    case 128: hipLaunchKernelGGL((decode2_multi_kernel<2, MODE, NB, PK, ORD>), grid, block, shm, s, m); break;
    default: hipLaunchKernelGGL((decode2_multi_kernel<4, MODE, NB, PK, ORD>), grid, block, shm, s, m); break;
  }
  return hipGetLastError() == hipSuccess ? EQ_OK : EQ_EHIP;
}

// Packed table entries for codes and BF16 output of layers of more than one
// phrase (one phrase has F = 2^16, which does not fit the entry's 16 bits).
// The GEMV keeps the split table: its phrase values as BF16 pairs cost no
// conversion, and its update two instructions less, which on gfx950
// outweighs the third LDS read per phrase (measured: 66 against 75 us on
// the 8192 x 28672 matrix at batch 1).
template <int MODE, int NB>
int launch2(Args2 a, hipStream_t s) {
  if constexpr (MODE != kGemv2) {
    // an ordered layer stores through 64-bit addresses; otherwise output
    // offsets from a tile's origin are 32-bit byte offsets
    if (a.order) {
      return a.n_syms > 1 ? launch2_pk<MODE, NB, true, true>(a, s)
                          : launch2_pk<MODE, NB, false, true>(a, s);
    }
    if (uint64_t(2) * a.TR * a.cols >= (uint64_t(1) << 31)) return EQ_EINVAL;
    if (a.n_syms > 1) return launch2_pk<MODE, NB, true, false>(a, s);
  }
  return launch2_pk<MODE, NB, false, false>(a, s);
}

size_t round256(size_t v) { return (v + 255) / 256 * 256; }

}  // namespace

namespace eq_detail {

bool v2_layer_ok(const eq_layer *L) {
  return L && L->version == 2 && L->lut && L->status && L->words && L->chunk_off &&
         L->chunk_state && L->scale && L->sym && L->freq &&
         (L->lanes == 64 || L->lanes == 128 || L->lanes == 256) && L->tile_cols > 0 &&
         L->tile_cols % 4 == 0 && L->prob_bits >= 10 && L->prob_bits <= 12 && L->n_syms >= 1 &&
         L->n_syms <= (1u << L->prob_bits) && L->rows > 0 && L->cols > 0 && L->n_chunks > 0 &&
         (L->base_format == kFmtE4M3 || L->base_format == kFmtInt8);
}

int v2_prepare(const eq_layer *L, hipStream_t s) {
  if (!v2_layer_ok(L)) return EQ_EINVAL;
  hipLaunchKernelGGL(prepare2_kernel, dim3(1), dim3(1024), 0, s,
                     reinterpret_cast<const uint32_t *>(L->sym), L->freq, L->n_syms, L->n_quads,
                     L->n_pairs, L->prob_bits, L->base_format, reinterpret_cast<uint4 *>(L->lut),
                     L->lut + 4 * kBuckets, L->status);
  return hipGetLastError() == hipSuccess ? EQ_OK : EQ_EHIP;
}

int v2_decode_codes(const eq_layer *L, uint8_t *codes, hipStream_t s) {
  if (!v2_layer_ok(L) || !codes) return EQ_EINVAL;
  Args2 a = make_args2(L);
  a.codes = codes;
  return launch2<kCodes2, 1>(a, s);
}

int v2_decode_bf16(const eq_layer *L, uint16_t *w, hipStream_t s) {
  if (!v2_layer_ok(L) || !w) return EQ_EINVAL;
  Args2 a = make_args2(L);
  a.wout = w;
  return launch2<kBf16_2, 1>(a, s);
}

// Workspace: the partial row sums of every column tile (none when a tile
// holds whole rows).
size_t v2_gemv_workspace_bytes(const eq_layer *L, uint32_t B) {
  if (!v2_layer_ok(L) || B < 1 || B > kMaxBatch2) return 0;
  const size_t NT = (L->cols + L->tile_cols - 1) / L->tile_cols;
  return NT > 1 ? round256(size_t(B) * NT * L->rows * sizeof(float)) : 256;
}

// Block-wise decode of version-2 layers to codes or BF16 (Sec. 2.2,
// block-wise decompression), each layer to its own output: one launch,
// blocks per layer in proportion to its tiles, so that small layers (the key
// and value projections of a block) run beside large ones instead of leaving
// most compute units idle in launches of their own.  Layers of several tile
// heights share the launch through decode2_mixed_kernel.  Packed table
// entries when every layer allows them.
bool v2_joint_out_ok(const eq_layer *const *L, uint32_t n) {
  for (uint32_t i = 0; i < n; ++i)
    if (!v2_layer_ok(L[i])) return false;
  return n >= 2 && n <= kMaxLayers2;
}

template <int MODE>
int v2_decode_out_multi(const eq_layer *const *L, uint32_t n, void *const *out, hipStream_t s) {
  if (!v2_joint_out_ok(L, n)) return EQ_EINVAL;
  MultiArgs2 m{};
  m.n = n;
  bool pk = true, ord = false, mix = false;
  for (uint32_t i = 0; i < n; ++i) {
    ord |= L[i]->row_order != nullptr;
    mix |= L[i]->lanes != L[0]->lanes;
  }
  for (uint32_t i = 0; i < n; ++i) {
    if (!out[i]) return EQ_EINVAL;
    // with an ordered layer every layer of the launch stores through 64-bit
    // addresses; otherwise output offsets from a tile's origin are 32-bit
    // byte offsets
    if (!ord && uint64_t(2) * L[i]->lanes * L[i]->cols >= (uint64_t(1) << 31)) return EQ_EINVAL;
    m.a[i] = make_args2(L[i]);
    if (MODE == kCodes2) m.a[i].codes = static_cast<uint8_t *>(out[i]);
    else m.a[i].wout = static_cast<uint16_t *>(out[i]);
    pk &= m.a[i].n_syms > 1;
  }
  if (mix) {
    if (ord)
      return pk ? launch2_multi<MODE, 1, true, true, true>(m, s)
                : launch2_multi<MODE, 1, false, true, true>(m, s);
    return pk ? launch2_multi<MODE, 1, true, false, true>(m, s)
              : launch2_multi<MODE, 1, false, false, true>(m, s);
  }
  if (ord)
    return pk ? launch2_multi<MODE, 1, true, true>(m, s) : launch2_multi<MODE, 1, false, true>(m, s);
  return pk ? launch2_multi<MODE, 1, true, false>(m, s) : launch2_multi<MODE, 1, false, false>(m, s);
}

int v2_decode_codes_multi(const eq_layer *const *L, uint8_t *const *codes, uint32_t n,
                          hipStream_t s) {
  void *out[kMaxLayers2] = {};
  for (uint32_t i = 0; i < n && i < kMaxLayers2; ++i) out[i] = codes[i];
  return v2_decode_out_multi<kCodes2>(L, n, out, s);
}

int v2_decode_bf16_multi(const eq_layer *const *L, uint16_t *const *w, uint32_t n,
                         hipStream_t s) {
  void *out[kMaxLayers2] = {};
  for (uint32_t i = 0; i < n && i < kMaxLayers2; ++i) out[i] = w[i];
  return v2_decode_out_multi<kBf16_2>(L, n, out, s);
}

bool v2_joint_ok(const eq_layer *const *L, uint32_t n) {
  for (uint32_t i = 0; i < n; ++i)
    if (!v2_layer_ok(L[i]) || L[i]->lanes != L[0]->lanes || L[i]->cols != L[0]->cols)
      return false;
  return n >= 2 && n <= kMaxLayers2;
}

int v2_decode_gemv_multi(const eq_layer *const *L, uint32_t n, const uint16_t *x, uint32_t B,
                         const uint16_t *const *bias, float *const *y, void *const *ws,
                         hipStream_t s) {
  if (!v2_joint_ok(L, n) || !x || !y || B < 1 || B > kMaxBatch2) return EQ_EINVAL;
  MultiArgs2 m{};
  m.n = n;
  for (uint32_t i = 0; i < n; ++i) {
    if (!y[i] || !ws[i]) return EQ_EINVAL;
    m.a[i] = make_args2(L[i]);
    m.a[i].x = x;
    m.a[i].batch = B;
    m.a[i].bias = bias ? bias[i] : nullptr;
    m.a[i].y = y[i];
    m.a[i].ws = static_cast<float *>(ws[i]);
  }
  const int rc = B == 1   ? launch2_multi<kGemv2, 1, false, false>(m, s)
                 : B == 2 ? launch2_multi<kGemv2, 2, false, false>(m, s)
                 : B <= 4 ? launch2_multi<kGemv2, 4, false, false>(m, s)
                          : launch2_multi<kGemv2, 8, false, false>(m, s);
  if (rc != EQ_OK) return rc;
  uint32_t omax = 0;
  bool any = false;
  for (uint32_t i = 0; i < n; ++i) {
    omax = max(omax, L[i]->rows * B);
    any |= m.a[i].NT > 1;
  }
  if (any)
    hipLaunchKernelGGL(merge2_multi_kernel, dim3((omax + kWave - 1) / kWave, n),
                       dim3(kMergeThreads), 0, s, m);
  return hipGetLastError() == hipSuccess ? EQ_OK : EQ_EHIP;
}

int v2_decode_gemv(const eq_layer *L, const uint16_t *x, uint32_t B, const uint16_t *bias,
                   float *y, void *ws, size_t ws_bytes, hipStream_t s) {
  if (!v2_layer_ok(L) || !x || !y || B < 1 || B > kMaxBatch2) return EQ_EINVAL;
  if (!ws || ws_bytes < v2_gemv_workspace_bytes(L, B)) return EQ_EINVAL;
  Args2 a = make_args2(L);
  a.x = x;
  a.batch = B;
  a.bias = bias;
  a.y = y;
  a.ws = static_cast<float *>(ws);
  // batch padded to 1, 2, 4 or 8 rows
  const int rc = B == 1   ? launch2<kGemv2, 1>(a, s)
                 : B == 2 ? launch2<kGemv2, 2>(a, s)
                 : B <= 4 ? launch2<kGemv2, 4>(a, s)
                          : launch2<kGemv2, 8>(a, s);
  if (rc != EQ_OK) return rc;
  if (a.NT > 1) {
    const uint32_t n = L->rows * B;
    hipLaunchKernelGGL(merge2_kernel, dim3((n + kWave - 1) / kWave), dim3(kMergeThreads), 0, s,
                       a);
  }
  return hipGetLastError() == hipSuccess ? EQ_OK : EQ_EHIP;
}

}  // namespace eq_detail
