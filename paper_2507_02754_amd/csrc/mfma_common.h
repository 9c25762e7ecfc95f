// Device helpers shared by the gfx950 MFMA kernels (bf16 operands, fp32
// accumulation with v_mfma_f32_32x32x16_bf16).
//
// Register layouts used throughout (one 64-lane wavefront, lane = 32*h + c):
//   A operand (32 x 16, row-major M x K): lane supplies row c, K-slots 8h..8h+7
//   B operand (16 x 32, K x N):           lane supplies column c, K-slots 8h..8h+7
//   C/D accumulator (32 x 32):            lane holds column c, register v holds
//                                          row 8*(v/4) + 4*h + (v%4)
// Only the C/D layout matters for correctness: the A and B operands of one
// instruction use the same (h, slot) -> K mapping, so any consistent K
// ordering chosen by the caller contracts correctly.
#pragma once

#include "sa_internal.h"

namespace sa {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef unsigned u32x4_t __attribute__((ext_vector_type(4)));
typedef unsigned u32x2_t __attribute__((ext_vector_type(2)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

__device__ __forceinline__ f32x16_t mfma32(u32x4_t a, u32x4_t b, f32x16_t c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                 __builtin_bit_cast(bf16x8_t, b), c, 0, 0, 0);
}

// Two floats -> packed bf16 pair (round to nearest even, v_cvt_pk_bf16_f32).
__device__ __forceinline__ unsigned pack_bf16x2(float lo, float hi) {
  f32x2_t v = {lo, hi};
  return __builtin_bit_cast(unsigned, __builtin_convertvector(v, bf16x2_t));
}

__device__ __forceinline__ float bf16_lo(unsigned x) { return __uint_as_float(x << 16); }
__device__ __forceinline__ float bf16_hi(unsigned x) { return __uint_as_float(x & 0xffff0000u); }

// Value of `x` held by lane (lane ^ 32): v_permlane32_swap exchanges the upper
// half of its first operand with the lower half of its second.
__device__ __forceinline__ float swap_halves(float x) {
  const unsigned u = __float_as_uint(x);
  auto p = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  const bool upper = (threadIdx.x & 32) != 0;
  return __uint_as_float(upper ? p[0] : p[1]);
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }
__device__ __forceinline__ float fast_log2(float x) { return __builtin_amdgcn_logf(x); }

// Butterfly over the 32 lanes sharing lane>>5 (xor 1..16).
__device__ __forceinline__ float max32(float x) {
#pragma unroll
  for (int off = 16; off > 0; off >>= 1) x = fmaxf(x, __shfl_xor(x, off));
  return x;
}
__device__ __forceinline__ float sum32(float x) {
#pragma unroll
  for (int off = 16; off > 0; off >>= 1) x += __shfl_xor(x, off);
  return x;
}

__device__ __forceinline__ u32x4_t ldg128(const uint16_t* p) {
  return *reinterpret_cast<const u32x4_t*>(p);
}

}  // namespace sa
