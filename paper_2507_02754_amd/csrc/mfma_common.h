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

// Accumulator register v of a 32x32 tile holds row 8*(v/4) + 4*h + (v%4).
__device__ __forceinline__ int acc_row(int v, int h) { return 8 * (v >> 2) + 4 * h + (v & 3); }

// A/B-operand fragment (32 rows x 16 K-slots) from a row-major bf16 LDS tile:
// lane (h, c) takes row c, columns 16t + 8h .. 16t + 8h + 7.
template <int STRIDE>
__device__ __forceinline__ u32x4_t frag_rows(const uint16_t* tile, int c, int h, int t) {
  return *reinterpret_cast<const u32x4_t*>(tile + c * STRIDE + 16 * t + 8 * h);
}

// Fragment whose K-slots run over 16 of the 32 rows of a transposed LDS tile
// (tile[col][row]), in the order a 32x32 accumulator produces them: slot e of
// half h is row 16u + 8(e/4) + 4h + e%4, so accumulator registers 8u..8u+7 of
// one product can feed the next product directly.
template <int STRIDE>
__device__ __forceinline__ u32x4_t frag_cols(const uint16_t* ttile, int row, int h, int u) {
  const uint16_t* p = ttile + row * STRIDE + 16 * u + 4 * h;
  const u32x2_t a0 = *reinterpret_cast<const u32x2_t*>(p);
  const u32x2_t a1 = *reinterpret_cast<const u32x2_t*>(p + 8);
  return u32x4_t{a0[0], a0[1], a1[0], a1[1]};
}

// Packs accumulator registers 8u..8u+7 (fp32) into a bf16 operand fragment.
__device__ __forceinline__ u32x4_t pack_frag(const float* x, int u) {
  u32x4_t r;
#pragma unroll
  for (int e = 0; e < 4; ++e) r[e] = pack_bf16x2(x[8 * u + 2 * e], x[8 * u + 2 * e + 1]);
  return r;
}

// Staging of one 32-row block of a [.., N, H, D] bf16 tensor into LDS, as a
// row-major tile ([32][D + 8], ROW) and/or a transposed tile ([D][32 + 4], TR);
// rows outside [0, N) read as zero. One work item = (row pair p, 8-column
// chunk dc); the paddings keep the fragment reads above conflict-free.
template <int D, int NTHREADS, bool ROW, bool TR>
struct BlockStage {
  static constexpr int rStride = D + 8;
  static constexpr int tStride = 32 + 4;
  static constexpr int rowBytes = ROW ? 32 * rStride * 2 : 0;
  static constexpr int tBytes = TR ? D * tStride * 2 : 0;
  static constexpr int bytes = rowBytes + tBytes;
  static constexpr int items = 16 * (D / 8);
  static constexpr int perThread = (items + NTHREADS - 1) / NTHREADS;
  u32x4_t reg[perThread][2];

  // `slot` is the caller's thread index, possibly rotated so that two stagings
  // issued together use disjoint threads.
  __device__ __forceinline__ void load(const uint16_t* src, size_t base, size_t rs, int jb, int N,
                                       int slot) {
#pragma unroll
    for (int x = 0; x < perThread; ++x) {
      const int it = slot + x * NTHREADS;
      const int p = it & 15, dc = it >> 4;
#pragma unroll
      for (int y = 0; y < 2; ++y) {
        const int j = jb + 2 * p + y;
        u32x4_t z = {0u, 0u, 0u, 0u};
        if (it < items && j >= 0 && j < N) z = ldg128(src + base + static_cast<size_t>(j) * rs + 8 * dc);
        reg[x][y] = z;
      }
    }
  }
  __device__ __forceinline__ void store(char* dst, int slot) const {
    uint16_t* rm = reinterpret_cast<uint16_t*>(dst);
    uint16_t* tr = reinterpret_cast<uint16_t*>(dst + rowBytes);
#pragma unroll
    for (int x = 0; x < perThread; ++x) {
      const int it = slot + x * NTHREADS;
      if (it >= items) continue;
      const int p = it & 15, dc = it >> 4;
      if (ROW) {
        *reinterpret_cast<u32x4_t*>(rm + (2 * p) * rStride + 8 * dc) = reg[x][0];
        *reinterpret_cast<u32x4_t*>(rm + (2 * p + 1) * rStride + 8 * dc) = reg[x][1];
      }
      if (TR) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const unsigned a = reg[x][0][e], b = reg[x][1][e];
          *reinterpret_cast<unsigned*>(tr + (8 * dc + 2 * e) * tStride + 2 * p) = (a & 0xffffu) | (b << 16);
          *reinterpret_cast<unsigned*>(tr + (8 * dc + 2 * e + 1) * tStride + 2 * p) =
              (a >> 16) | (b & 0xffff0000u);
        }
      }
    }
  }
};

}  // namespace sa
