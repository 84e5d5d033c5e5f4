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

#include "eq.h"
#include "eq_internal.h"

namespace {

using namespace eq_detail;

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float float2v __attribute__((ext_vector_type(2)));
typedef float floatx16 __attribute__((ext_vector_type(16)));

// Block tile: kBT tokens x kBO output rows, kBK input columns per stage.
// Four wavefronts, each owning a 64 x 64 quarter as 2 x 2 MFMA tiles of
// 32 x 32.  LDS rows are padded (X: 144 B per token row, codes: 72 B per
// output row) so that the 16-byte and 8-byte fragment reads of a quarter
// wavefront fall into distinct banks.
constexpr int kBT = 128, kBO = 128, kBK = 64;
constexpr int kThreads = 256;
constexpr int kXStride = kBK * 2 + 16;  // bytes per token row of the X tile
constexpr int kCStride = kBK + 8;       // bytes per output row of the code tile
constexpr int kXTileBytes = kBT * kXStride;
constexpr int kCTileBytes = kBO * kCStride;

struct GemmArgs {
  const uint8_t *codes;   // [M][N]
  const uint16_t *x;      // [B][N] BF16
  const uint16_t *scale;  // [M] BF16
  const uint16_t *bias;   // [M] BF16 or null
  float *y;               // [B][M]
  uint32_t B, M, N;
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

// One block: tokens [t0, t0 + 128) x output rows [o0, o0 + 128).  Stage k
// holds input columns [64 k, 64 k + 64); the next stage's global loads are in
// flight in registers while the current one is multiplied, and are written to
// the other LDS buffer afterwards (one barrier per stage).  Out-of-range
// tokens, rows and columns are loaded as zeros (N is a multiple of 16, so a
// 16-byte chunk is either wholly inside a row or wholly past its end).
template <int FMT>
__global__ __launch_bounds__(kThreads) void gemm_codes_kernel(GemmArgs a) {
  __shared__ __attribute__((aligned(16))) uint8_t xs[2][kXTileBytes];
  __shared__ __attribute__((aligned(16))) uint8_t cs[2][kCTileBytes];
  const uint32_t N = a.N;
  const uint32_t o0 = blockIdx.x * kBO, t0 = blockIdx.y * kBT;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wt = wave >> 1, wo = wave & 1;
  const int r32 = lane & 31, g = lane >> 5;

  // global -> register staging: X 1024 chunks of 16 B (4 per thread), codes
  // 512 chunks (2 per thread)
  uint4 xr[4], cr[2];
  auto gload = [&](uint32_t k0) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int c = tid + kThreads * r, row = c >> 3, col = c & 7;
      const uint32_t t = t0 + row, k = k0 + col * 8;
      xr[r] = (t < a.B && k < N) ? *reinterpret_cast<const uint4 *>(a.x + size_t(t) * N + k)
                                 : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int r = 0; r < 2; ++r) {
      const int c = tid + kThreads * r, row = c >> 2, col = c & 3;
      const uint32_t o = o0 + row, k = k0 + col * 16;
      cr[r] = (o < a.M && k < N) ? *reinterpret_cast<const uint4 *>(a.codes + size_t(o) * N + k)
                                 : make_uint4(0, 0, 0, 0);
    }
  };
  auto lstore = [&](int buf) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int c = tid + kThreads * r, row = c >> 3, col = c & 7;
      *reinterpret_cast<uint4 *>(&xs[buf][row * kXStride + col * 16]) = xr[r];
    }
#pragma unroll
    for (int r = 0; r < 2; ++r) {
      const int c = tid + kThreads * r, row = c >> 2, col = c & 3;
      uint2 *d = reinterpret_cast<uint2 *>(&cs[buf][row * kCStride + col * 16]);
      d[0] = make_uint2(cr[r].x, cr[r].y);
      d[1] = make_uint2(cr[r].z, cr[r].w);
    }
  };

  floatx16 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.0f;

  const uint32_t nk = (N + kBK - 1) / kBK;
  gload(0);
  lstore(0);
  __syncthreads();
  for (uint32_t kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < nk) gload((kt + 1) * kBK);
#pragma unroll
    for (int ks = 0; ks < kBK / 16; ++ks) {
      // fragments: lane (r32, g) holds 8 consecutive columns ks*16 + 8g ..
      // of token row r32 (A) and of output row r32 (B)
      bf16x8 af[2], bf[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        const int row = wt * 64 + i * 32 + r32;
        af[i] = *reinterpret_cast<const bf16x8 *>(&xs[cur][row * kXStride + (ks * 16 + g * 8) * 2]);
      }
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const int row = wo * 64 + j * 32 + r32;
        const uint2 c = *reinterpret_cast<const uint2 *>(&cs[cur][row * kCStride + ks * 16 + g * 8]);
        bf[j] = codes_to_bf16x8<FMT>(c);
      }
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bf[j], acc[i][j], 0, 0, 0);
    }
    if (kt + 1 < nk) lstore(cur ^ 1);
    __syncthreads();
  }

  // epilogue: element v of lane (r32, g) in tile (i, j) is token row
  // 8 (v / 4) + 4 g + v % 4 and output row r32 of that tile
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const uint32_t o = o0 + wo * 64 + j * 32 + r32;
    if (o >= a.M) continue;
    const float s = bf16_to_f32(a.scale[o]);
    const float b = a.bias ? bf16_to_f32(a.bias[o]) : 0.0f;
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const uint32_t t = t0 + wt * 64 + i * 32 + 8 * (v / 4) + 4 * g + (v % 4);
        if (t < a.B) a.y[size_t(t) * a.M + o] = s * acc[i][j][v] + b;
      }
  }
}

bool gemm_shape_ok(const eq_layer *L, uint32_t B) {
  return L && L->scale && L->rows > 0 && L->cols > 0 && L->cols % 16 == 0 && B >= 1 &&
         (L->base_format == kFmtE4M3 || L->base_format == kFmtInt8) &&
         uint64_t(B) * L->cols < (uint64_t(1) << 40);
}

}  // namespace

extern "C" size_t eq_gemm_workspace_bytes(const eq_layer *L) {
  if (!L || L->rows == 0 || L->cols == 0) return 0;
  return (size_t(L->rows) * L->cols + 255) / 256 * 256;
}

extern "C" int eq_gemm_codes(const eq_layer *L, const uint8_t *codes, const uint16_t *x,
                             uint32_t B, const uint16_t *bias, float *y, hipStream_t stream) {
  if (!gemm_shape_ok(L, B) || !codes || !x || !y) return EQ_EINVAL;
  if ((reinterpret_cast<uintptr_t>(codes) | reinterpret_cast<uintptr_t>(x)) & 15) return EQ_EINVAL;
  GemmArgs a{codes, x, L->scale, bias, y, B, L->rows, L->cols};
  const dim3 grid((L->rows + kBO - 1) / kBO, (B + kBT - 1) / kBT), block(kThreads);
  if (L->base_format == kFmtInt8)
    hipLaunchKernelGGL(gemm_codes_kernel<kFmtInt8>, grid, block, 0, stream, a);
  else
    hipLaunchKernelGGL(gemm_codes_kernel<kFmtE4M3>, grid, block, 0, stream, a);
  return hipGetLastError() == hipSuccess ? EQ_OK : EQ_EHIP;
}

extern "C" int eq_decode_gemm(const eq_layer *L, const uint16_t *x, uint32_t B,
                              const uint16_t *bias, float *y, void *ws, size_t ws_bytes,
                              hipStream_t stream) {
  if (!gemm_shape_ok(L, B) || !x || !y || !ws) return EQ_EINVAL;
  if (ws_bytes < eq_gemm_workspace_bytes(L)) return EQ_EINVAL;
  uint8_t *codes = static_cast<uint8_t *>(ws);
  const int rc = eq_decode_codes(L, codes, stream);
  if (rc != EQ_OK) return rc;
  return eq_gemm_codes(L, codes, x, B, bias, y, stream);
}
