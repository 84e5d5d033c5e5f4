// Device helpers shared by the decode kernels of both container versions
// (eq_decode.hip, eq_decode2.hip).
#pragma once
#include <hip/hip_runtime.h>

#include <cstdint>

namespace eq_dev {

constexpr int kWave = 64;
constexpr int32_t kBufferFlags = 0x00020000;  // buffer resource word 3 (gfx9 family)

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float float2v __attribute__((ext_vector_type(2)));
typedef short short4v __attribute__((ext_vector_type(4)));
typedef float float4v __attribute__((ext_vector_type(4)));

__device__ inline float bf16_to_f32(uint16_t b) { return __uint_as_float(uint32_t(b) << 16); }

// Two fp32 values to two nearest-even BF16 (low half: a).
__device__ inline uint32_t pack_bf16(float a, float b) {
  const float2v v = {a, b};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2));
}

// acc + lo16(a) * lo16(b) + hi16(a) * hi16(b), operands as BF16 pairs.
__device__ inline float dot2_bf16(uint32_t a, uint32_t b, float acc) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, a),
                                        __builtin_bit_cast(bf16x2, b), acc, false);
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

// Wave issue priority 3 - q (q = 0..3, wave-uniform).
__device__ inline void set_prio_down(uint32_t q) {
  switch (q) {
    case 0: __builtin_amdgcn_s_setprio(3); break;
    case 1: __builtin_amdgcn_s_setprio(2); break;
    case 2: __builtin_amdgcn_s_setprio(1); break;
    default: __builtin_amdgcn_s_setprio(0); break;
  }
}

// LDS pointers as 32-bit byte addresses, so that wave-uniform positions can
// live in scalar registers and be advanced by scalar arithmetic.
typedef __attribute__((address_space(3))) const uint16_t lds_u16;
__device__ inline uint32_t lds_addr(const void *p) {
  return static_cast<uint32_t>(
      reinterpret_cast<uintptr_t>((__attribute__((address_space(3))) const void *)p));
}
// An LDS pointer from its 32-bit byte address (through uintptr_t: LDS
// pointers are 32-bit on the device, 64-bit in the host pass).
template <typename T>
__device__ inline __attribute__((address_space(3))) T *lds_ptr(uint32_t addr) {
  return (__attribute__((address_space(3))) T *)(uintptr_t)addr;
}
__device__ inline uint32_t lds_read_u16(uint32_t addr) { return *lds_ptr<const uint16_t>(addr); }
__device__ inline void lds_write_u16(uint32_t addr, uint32_t v) {
  *lds_ptr<uint16_t>(addr) = static_cast<uint16_t>(v);
}

// a + 2 * b on the scalar unit in one instruction (both wave-uniform).  The
// instruction writes SCC, which the compiler must not keep live across it.
__device__ inline uint32_t add_twice(uint32_t a, uint32_t b) {
  uint32_t r;
  asm("s_lshl1_add_u32 %0, %1, %2" : "=s"(r) : "s"(b), "s"(a) : "scc");
  return r;
}

// Per-lane select by a wave mask (bit l of m picks b for lane l), as one
// v_cndmask.  Written out so that the compiler keeps it branch-free and does
// not sink the loads feeding b into a branch.
__device__ inline uint32_t select_by_mask(uint64_t m, uint32_t a, uint32_t b) {
  uint32_t r;
  asm("v_cndmask_b32_e64 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(b), "s"(m));
  return r;
}

// Renormalisation of the lanes whose bit is set in m: x = (x << 16) | w on
// those lanes (x < 2^16 there; only the low 16 bits of w are used), x
// unchanged on the others.  One v_perm_b32 under exec = exec & m instead of a
// shift-or and a select: the two scalar instructions that narrow and restore
// exec issue beside other waves' vector work.  They write SCC.
__device__ inline uint32_t renorm_lanes(uint64_t m, uint32_t x, uint32_t w) {
  uint64_t saved;
  // result bytes 3..0 = x byte 1, x byte 0, w byte 1, w byte 0
  asm("s_and_saveexec_b64 %1, %2\n\t"
      "v_perm_b32 %0, %0, %3, %4\n\t"
      "s_mov_b64 exec, %1"
      : "+v"(x), "=&s"(saved)
      : "s"(m), "v"(w), "s"(0x05040100u)
      : "scc");
  return x;
}

// Read-only inputs seen through the constant address space, so that loads
// at wave-uniform addresses become scalar (SMEM) loads and never wait on the
// vector memory counter.
typedef const __attribute__((address_space(4))) uint32_t const_u32;

__device__ inline const_u32 *as_const(const void *p) { return (const_u32 *)(p); }

// BF16 element i of a read-only array (i wave-uniform), via the aligned dword
// that holds it.  The array needs only 2-byte alignment (a bias may be a view
// at an odd element): scalar loads ignore the low two address bits, so the
// dword is addressed explicitly and the half picked by bit 1 of the address.
__device__ inline float bf16_at(const uint16_t *base, uint32_t i) {
  const uintptr_t at = reinterpret_cast<uintptr_t>(base) + 2 * uintptr_t(i);
  const uint32_t w = *as_const(reinterpret_cast<const void *>(at & ~uintptr_t(3)));
  return __uint_as_float((at & 2) ? (w & 0xFFFF0000u) : (w << 16));
}

// 16 stream words starting at word index i (a multiple of 8), clamped to the
// padded section so that a read ahead never leaves the container.
__device__ inline uint4 load_words(const uint16_t *words, uint32_t i, uint32_t last8) {
  return *reinterpret_cast<const uint4 *>(words + min(i, last8));
}


}  // namespace eq_dev
