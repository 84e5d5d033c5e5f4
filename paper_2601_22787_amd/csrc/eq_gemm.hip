// Prefill path of libeq (declared in include/eq.h): the linear layer
// y = x W_hat^T + b (Sec. 2.1) for a batch of B tokens, with W_hat = s_i *
// v(q_ij) taken from the decoded codes.  The paper decompresses a block's
// weights to a Float8 buffer and multiplies with an FP8-weight / 16-bit
// activation GEMM (Sec. 2.2 block-wise pipeline, App. A.1); here the codes
// (one byte per weight, from eq_decode_codes) feed a W8A16 GEMM on the gfx950
// matrix cores: the codes are converted to BF16 in registers, the products are
// accumulated in fp32 by v_mfma_f32_32x32x16_bf16, and s_i (and the bias)
// are applied once per output in the epilogue, as QMatMul(W_q, S, x) does.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>

#include "eq.h"
#include "eq_internal.h"

namespace {

using namespace eq_detail;

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float float2v __attribute__((ext_vector_type(2)));
typedef float floatx16 __attribute__((ext_vector_type(16)));

// Block tile: BT tokens x BO output rows, kBK input columns per stage, with
// the block's wavefronts each owning a WT x WO sub-tile as MFMA tiles of
// 32 x 32.  LDS rows are padded (X: 144 B per token row, codes: 72 B per
// output row) so that the 16-byte and 8-byte fragment reads of a quarter
// wavefront fall into distinct banks.  Two LDS stages (dynamic LDS).
constexpr int kBK = 64;
constexpr int kXStride = kBK * 2 + 16;  // bytes per token row of the X tile
constexpr int kCStride = kBK + 8;       // bytes per output row of the code tile

template <int BT, int BO>
constexpr int stage_bytes() {
  return BT * kXStride + BO * kCStride;
}

struct GemmArgs {
  const uint8_t *codes;   // [M][N]
  const uint16_t *x;      // [B][N] BF16
  const uint16_t *scale;  // [M] BF16
  const uint16_t *bias;   // [M] BF16 or null
  float *y;               // [B][M]
  uint32_t B, M, N;
  uint32_t gx, gy;        // output-row blocks, token blocks
  uint32_t group;         // token blocks per group of the launch order
  uint32_t splits;        // slices of the input columns (split-K), >= 1
  uint32_t split_stages;  // 64-column stages per slice
  float *part;            // [splits][B][M] partial sums when splits > 1
};

__device__ inline float bf16_to_f32(uint16_t b) { return __uint_as_float(uint32_t(b) << 16); }

__device__ inline uint32_t pack_bf16(float a, float b) {
  const float2v v = {a, b};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2));
}

// Eight codes (bytes of c, in order) to eight BF16 values, exactly (every
// E4M3 value and every integer in [-127, 127] is a BF16 value).
template <int FMT>
__device__ inline bf16x8 codes_to_bf16x8(uint2 c) {
  uint4 r;
  if (FMT == kFmtInt8) {
    r.x = pack_bf16(float(int8_t(c.x)), float(int8_t(c.x >> 8)));
    r.y = pack_bf16(float(int8_t(c.x >> 16)), float(int8_t(c.x >> 24)));
    r.z = pack_bf16(float(int8_t(c.y)), float(int8_t(c.y >> 8)));
    r.w = pack_bf16(float(int8_t(c.y >> 16)), float(int8_t(c.y >> 24)));
  } else {
    r.x = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(c.x, 1.0f, false));
    r.y = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(c.x, 1.0f, true));
    r.z = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(c.y, 1.0f, false));
    r.w = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(c.y, 1.0f, true));
  }
  return __builtin_bit_cast(bf16x8, r);
}

// Launch order.  Workgroups are dealt to the 8 XCDs round robin (each XCD
// has its own L2), so block i is renumbered so that every XCD receives a
// contiguous range of the logical order.  The logical order is slice by
// slice of the input columns, and within a slice walks groups of `group`
// token blocks, output-row block by output-row block, so that the blocks
// resident on one XCD share few X and code tiles.  The grid is padded to a
// multiple of 8; padding blocks exit at once.
__device__ inline bool block_tile(const GemmArgs &a, uint32_t &ob, uint32_t &tb,
                                  uint32_t &split) {
  const uint32_t nb = a.gx * a.gy;
  const uint32_t per = gridDim.x / 8;
  uint32_t logical = (blockIdx.x % 8) * per + blockIdx.x / 8;
  if (logical >= nb * a.splits) return false;
  split = logical / nb;
  logical %= nb;
  const uint32_t span = a.group * a.gx;          // blocks per group of token blocks
  const uint32_t first = (logical / span) * a.group;
  const uint32_t rows = min(a.group, a.gy - first);
  const uint32_t in = logical % span;
  tb = first + in % rows;
  ob = in / rows;
  return true;
}

// One block: tokens [tb BT, +BT) x output rows [ob BO, +BO).  Stage k holds
// input columns [64 k, 64 k + 64); the next stage's global loads are in
// flight in registers while the current one is multiplied, and are written
// to the other LDS buffer afterwards (one barrier per stage).  Out-of-range
// tokens, rows and columns read as zeros (N is a multiple of 16, so a
// 16-byte chunk is either wholly inside a row or wholly past its end): every
// lane loads from an address clamped into the matrix and selects zero at
// the LDS store, so the loads are unconditional and the wait before the
// stores covers only the stage being stored, not the one issued after it.
template <int FMT, int BT, int BO, int WT, int WO>
__global__ __launch_bounds__((BT / WT) * (BO / WO) * 64) void gemm_codes_kernel(GemmArgs a) {
  constexpr int kWaves = (BT / WT) * (BO / WO);
  constexpr int kThreads = kWaves * 64;
  constexpr int kXChunks = BT * (kBK * 2 / 16) / kThreads;  // 16-byte chunks per thread
  constexpr int kCChunks = BO * (kBK / 16) / kThreads;
  constexpr int TI = WT / 32, TJ = WO / 32;                   // MFMA tiles per wave
  static_assert(kXChunks * kThreads == BT * 8 && kCChunks * kThreads == BO * 4, "staging");
  extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
  uint32_t ob, tb, split;
  if (!block_tile(a, ob, tb, split)) return;
  const uint32_t N = a.N;
  const uint32_t o0 = ob * BO, t0 = tb * BT;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wt = wave / (BO / WO), wo = wave % (BO / WO);
  const int r32 = lane & 31, g = lane >> 5;
  uint8_t *const xs0 = smem;
  uint8_t *const cs0 = smem + BT * kXStride;
  constexpr int kStage = stage_bytes<BT, BO>();

  // two register sets of staged loads: the loads of stage k + 2 are issued
  // while stage k is multiplied, and written to LDS at the end of stage
  // k + 1, so each load has two stages of compute to arrive
  struct Staged {
    uint4 x[kXChunks], c[kCChunks];
    uint32_t ok;  // bit r: x chunk r in range; bit 16 + r: code chunk r
  };
  auto gload = [&](Staged &st, uint32_t k0) {
    st.ok = 0;
#pragma unroll
    for (int r = 0; r < kXChunks; ++r) {
      const int c = tid + kThreads * r, row = c >> 3, col = c & 7;
      const uint32_t t = t0 + row, k = k0 + col * 8;
      const uint4 v = *reinterpret_cast<const uint4 *>(a.x + size_t(min(t, a.B - 1)) * N +
                                                       min(k, N - 8));
      st.x[r] = v;
      st.ok |= uint32_t(t < a.B && k < N) << r;
    }
#pragma unroll
    for (int r = 0; r < kCChunks; ++r) {
      const int c = tid + kThreads * r, row = c >> 2, col = c & 3;
      const uint32_t o = o0 + row, k = k0 + col * 16;
      const uint4 v = *reinterpret_cast<const uint4 *>(a.codes + size_t(min(o, a.M - 1)) * N +
                                                       min(k, N - 16));
      st.c[r] = v;
      st.ok |= uint32_t(o < a.M && k < N) << (16 + r);
    }
  };
  auto lstore = [&](const Staged &st, int buf) {
    uint8_t *const xs = xs0 + buf * kStage, *const cs = cs0 + buf * kStage;
#pragma unroll
    for (int r = 0; r < kXChunks; ++r) {
      const int c = tid + kThreads * r, row = c >> 3, col = c & 7;
      *reinterpret_cast<uint4 *>(xs + row * kXStride + col * 16) =
          (st.ok >> r & 1) ? st.x[r] : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int r = 0; r < kCChunks; ++r) {
      const int c = tid + kThreads * r, row = c >> 2, col = c & 3;
      const uint4 v = (st.ok >> (16 + r) & 1) ? st.c[r] : make_uint4(0, 0, 0, 0);
      uint2 *d = reinterpret_cast<uint2 *>(cs + row * kCStride + col * 16);
      d[0] = make_uint2(v.x, v.y);
      d[1] = make_uint2(v.z, v.w);
    }
  };

  floatx16 acc[TI][TJ];
#pragma unroll
  for (int i = 0; i < TI; ++i)
#pragma unroll
    for (int j = 0; j < TJ; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.0f;

  // fragments of 16 columns ks*16 ..: lane (r32, g) holds the 8 consecutive
  // columns ks*16 + 8g .. of token row r32 (A) and of output row r32 (B)
  auto frags = [&](const uint8_t *xs, const uint8_t *cs, int ks, bf16x8 *af, bf16x8 *bf) {
#pragma unroll
    for (int i = 0; i < TI; ++i) {
      const int row = wt * WT + i * 32 + r32;
      af[i] = *reinterpret_cast<const bf16x8 *>(xs + row * kXStride + (ks * 16 + g * 8) * 2);
    }
#pragma unroll
    for (int j = 0; j < TJ; ++j) {
      const int row = wo * WO + j * 32 + r32;
      bf[j] = codes_to_bf16x8<FMT>(
          *reinterpret_cast<const uint2 *>(cs + row * kCStride + ks * 16 + g * 8));
    }
  };
  auto compute = [&](int buf) {
    const uint8_t *const xs = xs0 + buf * kStage, *const cs = cs0 + buf * kStage;
#pragma unroll
    for (int ks = 0; ks < kBK / 16; ++ks) {
      bf16x8 af[TI], bf[TJ];
      frags(xs, cs, ks, af, bf);
#pragma unroll
      for (int i = 0; i < TI; ++i)
#pragma unroll
        for (int j = 0; j < TJ; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bf[j], acc[i][j], 0, 0, 0);
    }
    // issue order: the first 16 columns' fragment reads, then one matrix
    // instruction and one of the later fragment reads in turn (left to the
    // compiler, the reads of a step come in one burst before its products)
    __builtin_amdgcn_sched_group_barrier(0x100, TI + TJ, 0);  // LDS reads
#pragma unroll
    for (int r = 0; r < 3 * (TI + TJ); ++r) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // matrix instruction
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // LDS read
    }
    __builtin_amdgcn_sched_group_barrier(0x008, 4 * TI * TJ, 0);
  };

  // stage kt: LDS buffer kt & 1; register set p holds stage kt + 1 on entry
  // and receives stage kt + 2 (sets alternate, so the loop is unrolled by 2)
  // this block's slice: stages [split * split_stages, +split_stages) of all
  // (N + 63) / 64 (the launcher makes every slice non-empty)
  const uint32_t k_first = split * a.split_stages;
  const uint32_t nk = min(a.split_stages, (N + kBK - 1) / kBK - k_first);
  const uint32_t kbase = k_first * kBK;
  Staged s0, s1;
  gload(s0, kbase);
  lstore(s0, 0);
  if (nk > 1) gload(s1, kbase + kBK);
  __syncthreads();
  auto stage = [&](uint32_t kt, Staged &next, Staged &after) {
    // near the end the last stage is loaded again (and not stored): the
    // loads stay unconditional, so the waits can count them exactly
    gload(after, kbase + min(kt + 2, nk - 1) * kBK);
    compute(kt & 1);
    if (kt + 1 < nk) lstore(next, (kt + 1) & 1);
    __syncthreads();
  };
  uint32_t kt = 0;
  for (; kt + 1 < nk; kt += 2) {
    stage(kt, s1, s0);
    stage(kt + 1, s0, s1);
  }
  if (kt < nk) stage(kt, s1, s0);

  // epilogue: element v of lane (r32, g) in tile (i, j) is token row
  // 8 (v / 4) + 4 g + v % 4 and output row r32 of that tile.  One slice:
  // y = s * sum + bias; several: the slice's raw sums, reduced afterwards.
  float *const part = a.part + size_t(split) * a.B * a.M;
#pragma unroll
  for (int j = 0; j < TJ; ++j) {
    const uint32_t o = o0 + wo * WO + j * 32 + r32;
    if (o >= a.M) continue;
    const float s = bf16_to_f32(a.scale[o]);
    const float b = a.bias ? bf16_to_f32(a.bias[o]) : 0.0f;
#pragma unroll
    for (int i = 0; i < TI; ++i)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const uint32_t t = t0 + wt * WT + i * 32 + 8 * (v / 4) + 4 * g + (v % 4);
        if (t >= a.B) continue;
        if (a.splits > 1) part[size_t(t) * a.M + o] = acc[i][j][v];
        else a.y[size_t(t) * a.M + o] = s * acc[i][j][v] + b;
      }
  }
}

// y[t][o] = s_o * (partial sums of the slices, in slice order) + bias_o:
// the same result whatever the timing of the slices.
__global__ void reduce_splits_kernel(GemmArgs a) {
  const size_t i = size_t(blockIdx.x) * blockDim.x + threadIdx.x;
  const size_t n = size_t(a.B) * a.M;
  if (i >= n) return;
  const uint32_t o = uint32_t(i % a.M);
  float sum = 0.0f;
  for (uint32_t k = 0; k < a.splits; ++k) sum += a.part[k * n + i];
  a.y[i] = bf16_to_f32(a.scale[o]) * sum + (a.bias ? bf16_to_f32(a.bias[o]) : 0.0f);
}

template <int FMT, int BT, int BO, int WT, int WO>
void launch_gemm(GemmArgs a, hipStream_t stream) {
  constexpr int kThreads = (BT / WT) * (BO / WO) * 64;
  a.gx = (a.M + BO - 1) / BO;
  a.gy = (a.B + BT - 1) / BT;
  a.group = 4;
  const uint32_t nb = a.gx * a.gy * a.splits;
  const dim3 grid((nb + 7) / 8 * 8), block(kThreads);
  constexpr size_t shm = 2 * stage_bytes<BT, BO>();
  hipLaunchKernelGGL((gemm_codes_kernel<FMT, BT, BO, WT, WO>), grid, block, shm, stream, a);
}

// Tile and split-K choice.  A 256 x 256 block (8 wavefronts of 128 x 64)
// does a stage's work at about 1.4x the rate of 128 x 128 blocks (4
// wavefronts of 64 x 64; measured per stage on the config-4 matrices), so it
// is used unless its padding (tokens and rows rounded up to 256) costs more
// than that.  Up to 64 tokens the GEMM is bound by the stream of codes, read
// once in all: blocks of 32 or 64 tokens x 256 rows (4 wavefronts of 32 or
// 64 x 64) load a quarter or half of the activation rows a 128 x 128 block
// loads per code (8192 x 28672 at 16 tokens: 70 -> 46 us).  When the tiles
// leave compute units idle, the input columns are cut into slices (at most
// 16, each at least 4 stages of 64 columns) whose partial sums are reduced in
// slice order: 256 x 256 blocks one per compute unit; blocks of up to 128
// tokens, of which two fit a compute unit, one round of two per unit (the
// codes are then read once in all; 8192 x 28672 at 65-128 tokens: 92-100 ->
// 77-85 us); with several 128-token blocks one per unit measured faster.
enum GemmTile { kTile256, kTile128, kTile64x256, kTile32x256 };

struct GemmPlan {
  GemmTile tile;
  uint32_t splits, split_stages;
};

GemmPlan plan_gemm(uint32_t B, uint32_t M, uint32_t N, int cus) {
  const uint32_t stages = (N + kBK - 1) / kBK;
  const uint64_t t256 = uint64_t((M + 255) / 256) * ((B + 255) / 256);
  const uint64_t t128 = uint64_t((M + 127) / 128) * ((B + 127) / 128);
  GemmPlan p{kTile128, 1, stages};
  uint64_t tiles = t128;
  if (B <= 64) {
    p.tile = B <= 32 ? kTile32x256 : kTile64x256;
    tiles = (M + 255) / 256;
  } else if (10 * 4 * t256 <= 14 * t128) {  // padded areas, in 128 x 128 units
    p.tile = kTile256;
    tiles = t256;
  }
  if (tiles >= uint64_t(cus)) return p;
  uint64_t want = p.tile == kTile256 ? uint64_t(cus) / tiles
                  : B <= 128 ? std::max<uint64_t>(1, 2 * uint64_t(cus) / tiles)
                             : (uint64_t(cus) + tiles - 1) / tiles;
  want = want < 16 ? want : 16;
  const uint64_t cap = stages / 4;
  const uint64_t sp = want < cap ? want : cap;
  if (sp <= 1) return p;
  p.split_stages = uint32_t((stages + sp - 1) / sp);
  p.splits = (stages + p.split_stages - 1) / p.split_stages;  // every slice non-empty
  return p;
}

template <int FMT>
void launch_gemm_fmt(GemmArgs a, const GemmPlan &p, hipStream_t stream) {
  a.splits = p.splits;
  a.split_stages = p.split_stages;
  switch (p.tile) {
    case kTile256: launch_gemm<FMT, 256, 256, 128, 64>(a, stream); break;
    case kTile64x256: launch_gemm<FMT, 64, 256, 64, 64>(a, stream); break;
    case kTile32x256: launch_gemm<FMT, 32, 256, 32, 64>(a, stream); break;
    default: launch_gemm<FMT, 128, 128, 64, 64>(a, stream); break;
  }
  if (p.splits > 1) {
    const size_t n = size_t(a.B) * a.M;
    hipLaunchKernelGGL(reduce_splits_kernel, dim3(uint32_t((n + 255) / 256)), dim3(256), 0, stream,
                       a);
  }
}

// Compute units of the current device, queried once per device.
int compute_units() {
  static std::atomic<int> cached[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  int c = cached[dev].load(std::memory_order_relaxed);
  if (c == 0) {
    if (hipDeviceGetAttribute(&c, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        c <= 0)
      c = 256;
    cached[dev].store(c, std::memory_order_relaxed);
  }
  return c;
}

bool gemm_shape_ok(const eq_layer *L, uint32_t B) {
  // the grid (blocks of 128 x 128 at least) stays below 2^31 workgroups
  return L && L->scale && L->rows > 0 && L->cols > 0 && L->cols % 16 == 0 && B >= 1 &&
         (L->base_format == kFmtE4M3 || L->base_format == kFmtInt8) &&
         uint64_t(B) * L->cols < (uint64_t(1) << 40) &&
         ((uint64_t(B) + 127) / 128) * ((uint64_t(L->rows) + 127) / 128) < (uint64_t(1) << 30);
}

size_t round256(size_t v) { return (v + 255) / 256 * 256; }

size_t partial_bytes(const eq_layer *L, uint32_t B) {
  const GemmPlan p = plan_gemm(B, L->rows, L->cols, compute_units());
  return p.splits > 1 ? round256(size_t(p.splits) * B * L->rows * sizeof(float)) : 0;
}

}  // namespace

extern "C" size_t eq_gemm_codes_workspace_bytes(const eq_layer *L, uint32_t B) {
  if (!gemm_shape_ok(L, B)) return 0;
  return partial_bytes(L, B);
}

// Batches up to this size go to the fused decode-GEMV (see eq_decode_gemm).
constexpr uint32_t kFusedMaxBatch = 8;

extern "C" size_t eq_gemm_workspace_bytes(const eq_layer *L, uint32_t B) {
  if (!gemm_shape_ok(L, B)) return 0;
  const size_t gemm = round256(size_t(L->rows) * L->cols) + partial_bytes(L, B);
  return B <= kFusedMaxBatch ? std::max(gemm, eq_gemv_workspace_bytes(L, B)) : gemm;
}

extern "C" int eq_gemm_codes(const eq_layer *L, const uint8_t *codes, const uint16_t *x,
                             uint32_t B, const uint16_t *bias, float *y, void *ws,
                             size_t ws_bytes, hipStream_t stream) {
  if (!gemm_shape_ok(L, B) || !codes || !x || !y) return EQ_EINVAL;
  if ((reinterpret_cast<uintptr_t>(codes) | reinterpret_cast<uintptr_t>(x)) & 15) return EQ_EINVAL;
  const GemmPlan p = plan_gemm(B, L->rows, L->cols, compute_units());
  if (p.splits > 1 && (!ws || ws_bytes < partial_bytes(L, B) ||
                       (reinterpret_cast<uintptr_t>(ws) & 3)))
    return EQ_EINVAL;
  GemmArgs a{codes, x, L->scale, bias, y, B, L->rows, L->cols, 0, 0, 0, 1, 0,
             static_cast<float *>(ws)};
  if (L->base_format == kFmtInt8) launch_gemm_fmt<kFmtInt8>(a, p, stream);
  else launch_gemm_fmt<kFmtE4M3>(a, p, stream);
  return hipGetLastError() == hipSuccess ? EQ_OK : EQ_EHIP;
}

extern "C" int eq_decode_gemm(const eq_layer *L, const uint16_t *x, uint32_t B,
                              const uint16_t *bias, float *y, void *ws, size_t ws_bytes,
                              hipStream_t stream) {
  if (!gemm_shape_ok(L, B) || !x || !y || !ws) return EQ_EINVAL;
  if (ws_bytes < eq_gemm_workspace_bytes(L, B)) return EQ_EINVAL;
  // Up to 8 tokens the fused decode-GEMV is faster than decoding the codes
  // and multiplying on the matrix cores: it never writes the codes, and at
  // such batches the GEMM cannot use the matrix cores' width (8192 x 28672,
  // 8 tokens: 142-146 us against 107 + 94 us).
  if (B <= kFusedMaxBatch) return eq_decode_gemv(L, x, B, bias, y, ws, ws_bytes, stream);
  uint8_t *codes = static_cast<uint8_t *>(ws);
  const size_t code_bytes = round256(size_t(L->rows) * L->cols);
  const int rc = eq_decode_codes(L, codes, stream);
  if (rc != EQ_OK) return rc;
  return eq_gemm_codes(L, codes, x, B, bias, y, codes + code_bytes, ws_bytes - code_bytes,
                       stream);
}
