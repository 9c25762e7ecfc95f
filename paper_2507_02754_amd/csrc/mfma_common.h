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

#include <type_traits>

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

// x + b for kernels instantiated with operand bias constants, x otherwise (so
// the plain instantiation carries no extra instruction).
template <bool BIAS>
__device__ __forceinline__ float plus_bias(float x, float b) {
  if constexpr (BIAS)
    return x + b;
  else
    return x;
}

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

// Raw buffer resource over `bytes` bytes at `p` (gfx9 descriptor word 3). Loads
// through it return 0 for any offset at or past `bytes`, including offsets that
// are negative as 32-bit integers: the hardware range check zero-fills the rows
// outside [0, N) of a staged block without per-lane bounds arithmetic.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* p, unsigned bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), 0, static_cast<int>(bytes), 0x00020000);
}
__device__ __forceinline__ u32x4_t ldbuf128(__amdgpu_buffer_rsrc_t r, int off) {
  return __builtin_bit_cast(u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0));
}
__device__ __forceinline__ u32x2_t ldbuf64(__amdgpu_buffer_rsrc_t r, int off) {
  return __builtin_bit_cast(u32x2_t, __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, 0));
}
__device__ __forceinline__ unsigned ldbuf32(__amdgpu_buffer_rsrc_t r, int off) {
  return __builtin_bit_cast(unsigned, __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0));
}

// Chunkwise cross product for the determinant logits of Section 5: per
// 3-component chunk, det[a; b; c] = a . (b x c). x[0 .. 11] and y[0 .. 11]
// hold components 8 ch - 2 .. 8 ch + 9 of two vectors (a 3-chunk reaches at
// most 2 components past a 16-byte slot of 8); out[e] = (x cross y) at
// component 8 ch + e, and 0 for the D mod 3 trailing components (>= DC). The
// chunk position m = (8 ch + e) mod 3 is taken at run time (ch may differ
// between lanes): all three forms are evaluated and the right one selected.
template <int DC>
__device__ __forceinline__ void cross8_rt(const float* x, const float* y, int ch, float* out) {
  const int m0 = (2 * ch) % 3;  // position of component 8 ch in its chunk
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const int m = (m0 + e) % 3;
    // chunk starting at window index e + 2 - m
    const float c0 = x[e + 3] * y[e + 4] - x[e + 4] * y[e + 3];  // m = 0: b = e + 2
    const float c1 = x[e + 3] * y[e + 1] - x[e + 1] * y[e + 3];  // m = 1: b = e + 1
    const float c2 = x[e] * y[e + 1] - x[e + 1] * y[e];          // m = 2: b = e
    const float v = m == 0 ? c0 : m == 1 ? c1 : c2;
    out[e] = 8 * ch + e < DC ? v : 0.f;
  }
}
// Byte-range of one head's rows of a [.., N, H, D] bf16 tensor, from row 0 to
// the end of row N-1 (rows are rs_bytes apart).
__device__ __forceinline__ unsigned head_bytes(int N, int rs_bytes, int D) {
  return static_cast<unsigned>(N - 1) * static_cast<unsigned>(rs_bytes) + 2u * static_cast<unsigned>(D);
}

// ---- swizzled row-major tiles in LDS ----
//
// A tile holds 32 rows of D bf16 with no padding; row r's 16-byte chunk ch is
// stored at chunk slot ch ^ swz(r), swz(r) = 4*(r%4) + (r/4)%4 (mod D/8). This
// keeps both reads below free of bank conflicts at D = 128: 16 lanes reading
// one chunk of 16 different rows (row fragments), and the transposing read of
// 4 consecutive rows x 16 consecutive columns per 16 lanes.
template <int D>
struct SwzTile {
  static constexpr int CH = D / 8;  // 16-byte chunks per row
  static constexpr int bytes = 32 * D * 2;
  static constexpr int instrs = 32 * CH / 64;  // 64-lane x 16-byte transfers per tile
  __device__ static __forceinline__ int swz(int r) { return (4 * (r & 3) + ((r >> 2) & 3)) & (CH - 1); }
  __device__ static __forceinline__ int off(int r, int ch) { return (r * CH + (ch ^ swz(r))) * 16; }
};

// Row fragment (lane (h, c): row c, K-slots = columns 16t + 8h .. +7).
template <int D>
__device__ __forceinline__ u32x4_t frag_row_swz(const char* tile, int c, int h, int t) {
  return *reinterpret_cast<const u32x4_t*>(tile + SwzTile<D>::off(c, 2 * t + h));
}

typedef short s16x4_t __attribute__((ext_vector_type(4)));
__device__ __forceinline__ u32x2_t ds_read_tr16(const char* p) {
  const s16x4_t v = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      reinterpret_cast<__attribute__((address_space(3))) s16x4_t*>(reinterpret_cast<uintptr_t>(p)));
  return __builtin_bit_cast(u32x2_t, v);
}

// Typed access through LDS-address-space pointers: offsets added to such a
// pointer fold into the DS instructions' immediate offset field.
typedef __attribute__((address_space(3))) char lds_char;
__device__ __forceinline__ lds_char* to_lds(char* p) { return (lds_char*)(p); }
template <typename V>
__device__ __forceinline__ V lds_ld(const lds_char* p) {
  return *reinterpret_cast<const __attribute__((address_space(3))) V*>(p);
}
template <typename V>
__device__ __forceinline__ void lds_st(lds_char* p, V v) {
  *reinterpret_cast<__attribute__((address_space(3))) V*>(p) = v;
}
// Buffer load of 16 bytes per lane straight into LDS: lane l's bytes go to
// dst + 16 l (dst wave-uniform). Out-of-range offsets load zeros, as for
// register loads. (The builtin exists only in the device pass.)
__device__ __forceinline__ void load_lds16(__amdgpu_buffer_rsrc_t r, lds_char* dst, int voff, int soff = 0) {
#if defined(__HIP_DEVICE_COMPILE__)
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (__attribute__((address_space(3))) void*)(dst), 16, voff, soff, 0, 0);
#endif
}
__device__ __forceinline__ u32x2_t lds_tr16(const lds_char* p) {
  const s16x4_t v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4_t*)(p));
  return __builtin_bit_cast(u32x2_t, v);
}

// Transposed fragment from a row-major swizzled tile: lane (h, c) gets column
// 32 dt + c, K-slot e of half h = row 16u + 8(e/4) + 4h + e%4 (the order the
// 32x32 accumulator produces). Two ds_read_b64_tr_b16: within each group of 16
// lanes, output lane i receives element i%4 of the 8 bytes addressed by lane
// 4e + i/4, so lane s of a group addresses row (base + s/4), columns 4(s%4)..+3.
template <int D>
__device__ __forceinline__ u32x4_t frag_tr_swz(const char* tile, int lane, int dt, int u) {
  const int grp = lane >> 4, s = lane & 15, h = grp >> 1;
  const int col = 32 * dt + 16 * (grp & 1) + 4 * (s & 3);
  const int ch = col >> 3, within = (col & 7) * 2;
  const int r0 = 16 * u + 4 * h + (s >> 2);
  const u32x2_t a = ds_read_tr16(tile + SwzTile<D>::off(r0, ch) + within);
  const u32x2_t b = ds_read_tr16(tile + SwzTile<D>::off(r0 + 8, ch) + within);
  return u32x4_t{a[0], a[1], b[0], b[1]};
}

// ---- fragment-major tiles in LDS ----
//
// A tile holds 32 rows of D bf16. The 16-byte chunk ch = 2t + hc of row r
// (columns 8ch .. 8ch + 7) is stored in 1 KB block t at lane slot
// 32 hc + (r ^ (4 hc + 8 (t & 1))). This layout gives:
//   * row fragments (lane (h, c): row c, columns 16t + 8h .. + 7) as one
//     ds_read_b128 per lane at a per-lane base (two bases, by t parity) plus
//     the immediate 1024 t, the 64 lanes hitting 64 distinct 16-byte slots;
//   * transposed fragments through ds_read_b64_tr_b16 at two per-lane bases
//     plus immediates (2048 dt + 256 u), each half-wavefront covering all 64
//     banks once;
//   * staging stores of 4 (D = 128) or 8 (D = 64) full rows per wavefront
//     instruction that touch every bank equally (the minimum LDS cycles).
template <int D>
struct FragTile {
  static constexpr int CH = D / 8;  // 16-byte chunks per row
  static constexpr int bytes = 32 * D * 2;
  static constexpr int instrs = 32 * CH / 64;  // 64-lane x 16-byte transfers per tile
  __device__ static __forceinline__ int slot(int r, int ch) {
    const int t = ch >> 1, hc = ch & 1;
    return t * 1024 + (32 * hc + (r ^ (4 * hc + 8 * (t & 1)))) * 16;
  }
  // Row fragment t of lane (h, c) is at row_base(p = t & 1) + 1024 t.
  __device__ static __forceinline__ int row_base(int lane, int p) {
    const int c = lane & 31, h = lane >> 5;
    return (32 * h + (c ^ (4 * h + 8 * p))) * 16;
  }
  // Transposed fragment (dt, u): two ds_read_b64_tr_b16 at tr_base(lane, 0)
  // and tr_base(lane, 1), each plus 2048 dt + 256 u. Lane (h, c) receives
  // column 32 dt + c, K-slot e of half h = row 16u + 8(e/4) + 4h + e%4 (the
  // accumulator's row order): within a 16-lane group (grp = lane / 16), lane s
  // addresses row 16u + 4(grp/2) + s/4 (+ 8 for the second read), columns
  // 32 dt + 16(grp%2) + 4(s%4) .. + 3.
  __device__ static __forceinline__ int tr_base(int lane, int second) {
    const int grp = lane >> 4, sl = lane & 15;
    const int p = grp & 1, hg = grp >> 1, hd = (sl >> 1) & 1, x = sl >> 2;
    return 1024 * p + 512 * hd + (4 * (hg ^ hd) + x) * 16 + 8 * (sl & 1) + 128 * (second ^ p);
  }
};

// Waits for this wavefront's LDS operations, then synchronises the
// workgroup. Volatile asm with a memory clobber so the compiler keeps LDS
// accesses on their side of it, and without the vmcnt(0) wait that
// __syncthreads adds, so global loads in flight stay in flight.
__device__ __forceinline__ void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// The same through builtins, so that the compiler's wait-count tracking knows
// every LDS read issued before it has completed (it does not look inside the
// inline assembly above and would otherwise wait again for them later).
__device__ __forceinline__ void lds_barrier_tracked() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0); vmcnt and expcnt at their maxima
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

template <int CTRL>
__device__ __forceinline__ float dpp_f(float x) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xF, 0xF, false));
}

// Reduction over the 32 lanes of each half-wavefront (lanes with the same
// lane >> 5) without LDS: DPP lane ^ 1 and lane ^ 2 (quad permutations), the
// mirror within 8 and within 16 lanes, then v_permlane16_swap for lane ^ 16.
// Every lane of the half ends with the result.
template <typename Op>
__device__ __forceinline__ float reduce32(float x, Op op) {
  x = op(x, dpp_f<0xB1>(x));   // quad_perm [1,0,3,2]
  x = op(x, dpp_f<0x4E>(x));   // quad_perm [2,3,0,1]
  x = op(x, dpp_f<0x141>(x));  // row_half_mirror
  x = op(x, dpp_f<0x140>(x));  // row_mirror
  auto p = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return op(__uint_as_float(p[0]), __uint_as_float(p[1]));
}

// Sums v[j] over the 32 lanes of each half-wavefront (lanes with the same
// lane >> 5), for NV values per lane, without LDS: each step pairs every lane
// with one partner, and the lane keeps the sum of one half of its values
// while the partner keeps the other half (v_permlane16_swap for the lane ^ 16
// pairs, then DPP row_mirror, row_half_mirror and quad permutations). On
// return v[0 .. NV/32 - 1] hold the sums of values j0 .. j0 + NV/32 - 1, with
// j0 = sum over the bits b of c = lane & 31, from bit 4 down, of
// bit * NV / 2^(step+1).
// Level S (0..4) of the reduction below, so that callers can spread the
// levels over other work; levels must run in order.
template <int NV, int S>
__device__ __forceinline__ void reduce_lanes32_level(float* v, int lane) {
  static_assert(NV >= 32 && NV % 32 == 0, "one value per lane at least");
  constexpr int N1 = NV / 2;
  if constexpr (S == 0) {
#pragma unroll
    for (int j = 0; j < N1; ++j) {
      auto p = __builtin_amdgcn_permlane16_swap(__float_as_uint(v[j]), __float_as_uint(v[j + N1]), false, false);
      v[j] = __uint_as_float(p[0]) + __uint_as_float(p[1]);
    }
  } else {
    // 0x140 row_mirror (lane ^ 15 within 16), 0x141 row_half_mirror (lane ^ 7
    // within 8), 0x4E quad_perm [2,3,0,1], 0xB1 quad_perm [1,0,3,2]
    constexpr int C = S == 1 ? 0x140 : S == 2 ? 0x141 : S == 3 ? 0x4E : 0xB1;
    constexpr int bit = 16 >> S;
    constexpr int n = N1 >> S;
#pragma unroll
    for (int j = 0; j < n; ++j) {
      const float a = v[j] + dpp_f<C>(v[j]), b = v[j + n] + dpp_f<C>(v[j + n]);
      v[j] = (lane & bit) ? b : a;
    }
  }
}
template <int NV>
__device__ __forceinline__ void reduce_lanes32(float* v, int lane) {
  reduce_lanes32_level<NV, 0>(v, lane);
  reduce_lanes32_level<NV, 1>(v, lane);
  reduce_lanes32_level<NV, 2>(v, lane);
  reduce_lanes32_level<NV, 3>(v, lane);
  reduce_lanes32_level<NV, 4>(v, lane);
}

// Accumulator register v of a 32x32 tile holds row 8*(v/4) + 4*h + (v%4).
__device__ __forceinline__ int acc_row(int v, int h) { return 8 * (v >> 2) + 4 * h + (v & 3); }

// Packs accumulator registers 8u..8u+7 (fp32) into a bf16 operand fragment.
__device__ __forceinline__ u32x4_t pack_frag(const float* x, int u) {
  u32x4_t r;
#pragma unroll
  for (int e = 0; e < 4; ++e) r[e] = pack_bf16x2(x[8 * u + 2 * e], x[8 * u + 2 * e + 1]);
  return r;
}

}  // namespace sa
