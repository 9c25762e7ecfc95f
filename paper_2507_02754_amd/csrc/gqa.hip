// Grouped-query attention support for the backward (Section 6's production
// layout: H query heads share Hkv heads of K, K', V, V'; query head h reads
// K-side head h / G with G = H / Hkv).
//
// The backward for Hkv < H is the per-query-head backward followed by a sum of
// the K-side gradients over each group's G query heads (each K-side element
// enters every logit of those heads). Two HBM-bound kernels wrap the
// per-head backward kernels:
//   expand_heads_kernel  copies K, K', V, V' from [B, N, Hkv, D] to
//                        [B, N, H, D] (head h gets K-side head h / G);
//   group_sum_kernel     sums dK, dK', dV, dV' from [B, N, H, D] over each
//                        group into [B, N, Hkv, D], in fp32, heads in
//                        ascending order, rounded once to the data type.
// Both treat the four tensors in one launch (blockIdx.y) and stream 16-byte
// (expand) or 4-element (sum) vectors with consecutive lanes on consecutive
// addresses. The fixed summation order keeps the backward deterministic.
#include "sa_internal.h"
#include "simplicial_attn.h"

namespace sa {
namespace {

struct Quad {
  const void* src[4];
  void* dst[4];
};

constexpr int kThreads = 256;
constexpr long long kMaxBlocks = 8192;

// One thread per 16-byte vector of the [B*N*H, D] destination.
__global__ __launch_bounds__(kThreads) void expand_heads_kernel(Quad p, long long rows, int H,
                                                                int G, int vpr) {
  const uint4* __restrict__ src = static_cast<const uint4*>(p.src[blockIdx.y]);
  uint4* __restrict__ dst = static_cast<uint4*>(p.dst[blockIdx.y]);
  const long long total = rows * vpr;
  const int Hkv = H / G;
  for (long long idx = static_cast<long long>(blockIdx.x) * kThreads + threadIdx.x; idx < total;
       idx += static_cast<long long>(gridDim.x) * kThreads) {
    const long long row = idx / vpr;  // (b, n, h) row of the destination
    const int c = static_cast<int>(idx - row * vpr);
    const long long bn = row / H;
    const int h = static_cast<int>(row - bn * H);
    dst[idx] = src[(bn * Hkv + h / G) * vpr + c];
  }
}

// One thread per 4 consecutive elements of the [B*N*Hkv, D] destination. Row
// r = (b, n, hk) of the destination sums source rows r*G + t, t = 0..G-1
// (query heads hk*G + t of position (b, n)).
template <bool BF16>
__global__ __launch_bounds__(kThreads) void group_sum_kernel(Quad p, long long rows, int G,
                                                             int qpr) {
  const long long total = rows * qpr;
  for (long long idx = static_cast<long long>(blockIdx.x) * kThreads + threadIdx.x; idx < total;
       idx += static_cast<long long>(gridDim.x) * kThreads) {
    const long long row = idx / qpr;
    const int c = static_cast<int>(idx - row * qpr);
    const long long in0 = row * G * qpr + c;
    float a[4];
    if constexpr (BF16) {
      const uint2* __restrict__ src = static_cast<const uint2*>(p.src[blockIdx.y]);
      for (int t = 0; t < G; ++t) {
        const uint2 x = src[in0 + static_cast<long long>(t) * qpr];
        const float f[4] = {bf16_to_f32(static_cast<uint16_t>(x.x)),
                            bf16_to_f32(static_cast<uint16_t>(x.x >> 16)),
                            bf16_to_f32(static_cast<uint16_t>(x.y)),
                            bf16_to_f32(static_cast<uint16_t>(x.y >> 16))};
#pragma unroll
        for (int e = 0; e < 4; ++e) a[e] = t == 0 ? f[e] : a[e] + f[e];
      }
      uint2 o;
      o.x = static_cast<uint32_t>(f32_to_bf16(a[0])) | (static_cast<uint32_t>(f32_to_bf16(a[1])) << 16);
      o.y = static_cast<uint32_t>(f32_to_bf16(a[2])) | (static_cast<uint32_t>(f32_to_bf16(a[3])) << 16);
      static_cast<uint2*>(p.dst[blockIdx.y])[idx] = o;
    } else {
      const float4* __restrict__ src = static_cast<const float4*>(p.src[blockIdx.y]);
      for (int t = 0; t < G; ++t) {
        const float4 x = src[in0 + static_cast<long long>(t) * qpr];
        const float f[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) a[e] = t == 0 ? f[e] : a[e] + f[e];
      }
      static_cast<float4*>(p.dst[blockIdx.y])[idx] = make_float4(a[0], a[1], a[2], a[3]);
    }
  }
}

unsigned grid_for(long long items) {
  const long long blocks = (items + kThreads - 1) / kThreads;
  return static_cast<unsigned>(blocks < kMaxBlocks ? blocks : kMaxBlocks);
}

}  // namespace

hipError_t gqa_expand(const Shape& s, const void* const src[4], void* const dst[4],
                      hipStream_t st) {
  Quad p;
  for (int t = 0; t < 4; ++t) {
    p.src[t] = src[t];
    p.dst[t] = dst[t];
  }
  const int esize = s.dtype == SA_DTYPE_BF16 ? 2 : 4;
  const int vpr = s.D * esize / 16;       // D >= 16, so a row is a whole number of vectors
  const long long rows = static_cast<long long>(s.B) * s.N * s.H;
  hipLaunchKernelGGL(expand_heads_kernel, dim3(grid_for(rows * vpr), 4), dim3(kThreads), 0, st, p,
                     rows, s.H, s.H / s.Hkv, vpr);
  return hipGetLastError();
}

hipError_t gqa_group_sum(const Shape& s, const void* const src[4], void* const dst[4],
                         hipStream_t st, int ntens) {
  Quad p;
  for (int t = 0; t < 4; ++t) {
    p.src[t] = src[t];
    p.dst[t] = dst[t];
  }
  const int qpr = s.D / 4;
  const long long rows = static_cast<long long>(s.B) * s.N * s.Hkv;
  const dim3 grid(grid_for(rows * qpr), ntens);
  if (s.dtype == SA_DTYPE_BF16)
    hipLaunchKernelGGL(group_sum_kernel<true>, grid, dim3(kThreads), 0, st, p, rows, s.H / s.Hkv,
                       qpr);
  else
    hipLaunchKernelGGL(group_sum_kernel<false>, grid, dim3(kThreads), 0, st, p, rows, s.H / s.Hkv,
                       qpr);
  return hipGetLastError();
}

}  // namespace sa
