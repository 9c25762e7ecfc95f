// Generic HIP path: correct for every supported dtype, head_dim and window
// pair, written for clarity rather than speed. It serves shapes the MFMA
// kernels do not specialise (fp32 data, w2 not a multiple of 32, small
// head_dim) and is the fallback the fast paths are tested against.
//
// One workgroup of 256 threads owns one output row. Threads stride over the
// (j, k) pairs of that row, each keeping a private D-vector accumulator in
// registers; a wavefront shuffle reduction plus a small LDS pass combines
// them. All arithmetic is fp32; exponentials use expf.
//
// Forward (Section 4, Eqs. (3d-attention), (softmax), (attenval)): two passes
// over the pairs -- the first finds the row maximum of the logits, the second
// sums exp(logit - max) and the exp-weighted v_j o v'_k.
// Backward (Section 7): dQ per query row; dK/dV per K-row j and dK'/dV' per
// K'-row k, each gathering its own pairs, so no atomics are needed and the
// result is deterministic.
#include "sa_internal.h"

#include <math.h>

namespace sa {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;

template <typename T>
__device__ __forceinline__ float ld(const T* p);
template <>
__device__ __forceinline__ float ld<float>(const float* p) {
  return *p;
}
template <>
__device__ __forceinline__ float ld<uint16_t>(const uint16_t* p) {
  return bf16_to_f32(*p);
}

template <typename T>
__device__ __forceinline__ void st(T* p, float x);
template <>
__device__ __forceinline__ void st<float>(float* p, float x) {
  *p = x;
}
template <>
__device__ __forceinline__ void st<uint16_t>(uint16_t* p, float x) {
  *p = f32_to_bf16(x);
}

__device__ __forceinline__ float wave_max(float x) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) x = fmaxf(x, __shfl_xor(x, off));
  return x;
}

__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) x += __shfl_xor(x, off);
  return x;
}

// Block-wide max/sum of one scalar; every thread gets the result.
__device__ float block_max(float x, float* red) {
  x = wave_max(x);
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) red[w] = x;
  __syncthreads();
  float r = red[0];
  for (int i = 1; i < kWaves; ++i) r = fmaxf(r, red[i]);
  __syncthreads();
  return r;
}

__device__ float block_sum(float x, float* red) {
  x = wave_sum(x);
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) red[w] = x;
  __syncthreads();
  float r = 0.f;
  for (int i = 0; i < kWaves; ++i) r += red[i];
  __syncthreads();
  return r;
}

// Sums acc[D] over the block; thread t < D receives component t (others 0).
template <int D>
__device__ float block_sum_vec(float (&acc)[D], float* red /* [kWaves * D] */) {
#pragma unroll
  for (int d = 0; d < D; ++d) acc[d] = wave_sum(acc[d]);
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) {
#pragma unroll
    for (int d = 0; d < D; ++d) red[w * D + d] = acc[d];
  }
  __syncthreads();
  float r = 0.f;
  if (threadIdx.x < D) {
    for (int i = 0; i < kWaves; ++i) r += red[i * D + threadIdx.x];
  }
  __syncthreads();
  return r;
}

// Row pointer helper for [B, N, heads, D] tensors: base of (b, 0, h, 0),
// stride heads*D (heads = H for Q-side tensors, Hkv for K/V-side ones).
struct Rows {
  size_t base, stride;
  __device__ Rows(int b, int h, const Shape& s) : Rows(b, h, s.H, s) {}
  __device__ Rows(int b, int h, int heads, const Shape& s)
      : base((static_cast<size_t>(b) * s.N * heads + h) * s.D),
        stride(static_cast<size_t>(heads) * s.D) {}
  __device__ size_t at(int n) const { return base + static_cast<size_t>(n) * stride; }
};

// Operands x and y are read with the constant bx / by added to every element
// (the K' / V' bias constants; 0 for the other tensors).
template <typename T, int D>
__device__ __forceinline__ float tri(const float* a, const T* x, float bx, const T* y, float by) {
  float s = 0.f;
#pragma unroll 8
  for (int d = 0; d < D; ++d) s += a[d] * (ld(x + d) + bx) * (ld(y + d) + by);
  return s;
}

// Determinant logits (Section 5, Eq. (logits)): sum over the 3-component
// chunks c of det([a_c; x_c; y_c]) = a_c . (x_c cross y_c); the D mod 3
// trailing components take no part.
template <typename T, int D>
__device__ __forceinline__ float tri_det(const float* a, const T* x, float bx, const T* y, float by) {
  float s = 0.f;
  for (int c = 0; c + 2 < D; c += 3) {
    const float x0 = ld(x + c) + bx, x1 = ld(x + c + 1) + bx, x2 = ld(x + c + 2) + bx;
    const float y0 = ld(y + c) + by, y1 = ld(y + c + 1) + by, y2 = ld(y + c + 2) + by;
    s += a[c] * (x1 * y2 - x2 * y1) + a[c + 1] * (x2 * y0 - x0 * y2) + a[c + 2] * (x0 * y1 - x1 * y0);
  }
  return s;
}

// Logit of form FORM (0: trilinear, Eq. (3d-attention); 1: determinant) with
// operands in the order (a, x, y) of the form.
template <typename T, int D, int FORM>
__device__ __forceinline__ float logit3(const float* a, const T* x, float bx, const T* y, float by) {
  if constexpr (FORM == 0)
    return tri<T, D>(a, x, bx, y, by);
  else
    return tri_det<T, D>(a, x, bx, y, by);
}

// acc += w * dA/da for A = form(a, x, y): x o y (trilinear) or, per chunk,
// x cross y (determinant; trailing components get nothing).
template <typename T, int D, int FORM>
__device__ __forceinline__ void add_partial(float (&acc)[D], float w, const T* x, float bx, const T* y,
                                            float by) {
  if constexpr (FORM == 0) {
#pragma unroll
    for (int d = 0; d < D; ++d) acc[d] += w * (ld(x + d) + bx) * (ld(y + d) + by);
  } else {
#pragma unroll
    for (int c = 0; c + 2 < D; c += 3) {
      const float x0 = ld(x + c) + bx, x1 = ld(x + c + 1) + bx, x2 = ld(x + c + 2) + bx;
      const float y0 = ld(y + c) + by, y1 = ld(y + c + 1) + by, y2 = ld(y + c + 2) + by;
      acc[c] += w * (x1 * y2 - x2 * y1);
      acc[c + 1] += w * (x2 * y0 - x0 * y2);
      acc[c + 2] += w * (x0 * y1 - x1 * y0);
    }
  }
}

// ---------------------------------------------------------------- forward ---
template <typename T, int D, int FORM>
__global__ __launch_bounds__(kThreads) void fwd_kernel(Shape s, const T* __restrict__ q,
                                                       const T* __restrict__ k,
                                                       const T* __restrict__ kp,
                                                       const T* __restrict__ v,
                                                       const T* __restrict__ vp, T* __restrict__ out,
                                                       float* __restrict__ lse) {
  const int i = blockIdx.x % s.N;
  const int bh = blockIdx.x / s.N;
  const int b = bh / s.H, h = bh % s.H;
  const Rows rows(b, h, s);                          // q, out
  const Rows kvr(b, h / (s.H / s.Hkv), s.Hkv, s);    // k, k', v, v'
  __shared__ float qs[D];
  __shared__ float red[kWaves * D];
  __shared__ float sred[kWaves];
  if (threadIdx.x < D) qs[threadIdx.x] = ld(q + rows.at(i) + threadIdx.x) * s.scale;
  __syncthreads();

  const int j0 = max(0, i - s.w1 + 1), nj = i - j0 + 1;
  const int k0 = max(0, i - s.w2 + 1), nk = i - k0 + 1;
  const int np = nj * nk;

  float m = -INFINITY;
  for (int p = threadIdx.x; p < np; p += kThreads) {
    const int j = j0 + p / nk, kk = k0 + p % nk;
    m = fmaxf(m, logit3<T, D, FORM>(qs, k + kvr.at(j), 0.f, kp + kvr.at(kk), s.kp_bias));
  }
  m = block_max(m, sred);

  float l = 0.f;
  float acc[D];
#pragma unroll
  for (int d = 0; d < D; ++d) acc[d] = 0.f;
  for (int p = threadIdx.x; p < np; p += kThreads) {
    const int j = j0 + p / nk, kk = k0 + p % nk;
    const float e = expf(logit3<T, D, FORM>(qs, k + kvr.at(j), 0.f, kp + kvr.at(kk), s.kp_bias) - m);
    l += e;
    const T* vj = v + kvr.at(j);
    const T* vk = vp + kvr.at(kk);
#pragma unroll
    for (int d = 0; d < D; ++d) acc[d] += e * ld(vj + d) * (ld(vk + d) + s.vp_bias);
  }
  l = block_sum(l, sred);
  const float o = block_sum_vec<D>(acc, red);
  if (threadIdx.x < D) st(out + rows.at(i) + threadIdx.x, o / l);
  if (threadIdx.x == 0) lse[static_cast<size_t>(bh) * s.N + i] = m + logf(l);
}

// ------------------------------------------------------------------ delta ---
template <typename T>
__global__ void delta_kernel(Shape s, const T* __restrict__ out, const T* __restrict__ dout,
                             float* __restrict__ delta) {
  const int64_t idx = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  const int64_t total = static_cast<int64_t>(s.B) * s.H * s.N;
  if (idx >= total) return;
  const int i = static_cast<int>(idx % s.N);
  const int bh = static_cast<int>(idx / s.N);
  const size_t off = ((static_cast<size_t>(bh / s.H) * s.N + i) * s.H + bh % s.H) * s.D;
  float acc = 0.f;
  for (int d = 0; d < s.D; ++d) acc += ld(out + off + d) * ld(dout + off + d);
  delta[idx] = acc;
}

// --------------------------------------------------------------------- dQ ---
template <typename T, int D, int FORM>
__global__ __launch_bounds__(kThreads) void dq_kernel(Shape s, const T* __restrict__ q,
                                                      const T* __restrict__ k,
                                                      const T* __restrict__ kp,
                                                      const T* __restrict__ v,
                                                      const T* __restrict__ vp,
                                                      const T* __restrict__ dout,
                                                      const float* __restrict__ lse,
                                                      const float* __restrict__ delta,
                                                      T* __restrict__ dq) {
  const int i = blockIdx.x % s.N;
  const int bh = blockIdx.x / s.N;
  const int b = bh / s.H, h = bh % s.H;
  const Rows rows(b, h, s);
  __shared__ float qs[D];
  __shared__ float ds_[D];
  __shared__ float red[kWaves * D];
  if (threadIdx.x < D) {
    qs[threadIdx.x] = ld(q + rows.at(i) + threadIdx.x) * s.scale;
    ds_[threadIdx.x] = ld(dout + rows.at(i) + threadIdx.x);
  }
  __syncthreads();
  const float lse_i = lse[static_cast<size_t>(bh) * s.N + i];
  const float delta_i = delta[static_cast<size_t>(bh) * s.N + i];
  const int j0 = max(0, i - s.w1 + 1), nj = i - j0 + 1;
  const int k0 = max(0, i - s.w2 + 1), nk = i - k0 + 1;
  const int np = nj * nk;

  float acc[D];
#pragma unroll
  for (int d = 0; d < D; ++d) acc[d] = 0.f;
  for (int p = threadIdx.x; p < np; p += kThreads) {
    const int j = j0 + p / nk, kk = k0 + p % nk;
    const T* kj = k + rows.at(j);
    const T* kk_ = kp + rows.at(kk);
    const float pr = expf(logit3<T, D, FORM>(qs, kj, 0.f, kk_, s.kp_bias) - lse_i);
    const float dp = tri<T, D>(ds_, v + rows.at(j), 0.f, vp + rows.at(kk), s.vp_bias);
    const float dsv = pr * (dp - delta_i);
    add_partial<T, D, FORM>(acc, dsv, kj, 0.f, kk_, s.kp_bias);
  }
  const float g = block_sum_vec<D>(acc, red);
  if (threadIdx.x < D) st(dq + rows.at(i) + threadIdx.x, g * s.scale);
}

// ------------------------------------------------------- dK / dV / dK' / dV' ---
// One workgroup per key row r of the K/V side (SIDE 0: window w1, partner
// window w2) or of the K'/V' side (SIDE 1: window w2, partner window w1). The
// pairs touching r are (i, o) with i in [r, r + w_self) and o in (i - w_other, i].
// MODE 0 produces the key gradient, MODE 1 the value gradient. For the
// determinant form (FORM 1) the operand order follows the cyclic identities
// q . (k x k') = k . (k' x q) = k' . (q x k).
template <typename T, int D, int SIDE, int MODE, int FORM>
__global__ __launch_bounds__(kThreads) void keyside_kernel(
    Shape s, const T* __restrict__ q, const T* __restrict__ kself, const T* __restrict__ kother,
    const T* __restrict__ vself, const T* __restrict__ vother, const T* __restrict__ dout,
    const float* __restrict__ lse, const float* __restrict__ delta, T* __restrict__ grad) {
  const int r = blockIdx.x % s.N;
  const int bh = blockIdx.x / s.N;
  const int b = bh / s.H, h = bh % s.H;
  const Rows rows(b, h, s);
  const int wself = SIDE == 0 ? s.w1 : s.w2;
  const int wother = SIDE == 0 ? s.w2 : s.w1;
  __shared__ float kr[D];
  __shared__ float vr[D];
  __shared__ float red[kWaves * D];
  // Bias constants: K' / V' are the self operands of SIDE 1, the other
  // operands of SIDE 0.
  const float bks = SIDE == 1 ? s.kp_bias : 0.f, bvs = SIDE == 1 ? s.vp_bias : 0.f;
  const float bko = SIDE == 0 ? s.kp_bias : 0.f, bvo = SIDE == 0 ? s.vp_bias : 0.f;
  if (threadIdx.x < D) {
    kr[threadIdx.x] = (ld(kself + rows.at(r) + threadIdx.x) + bks) * s.scale;
    vr[threadIdx.x] = ld(vself + rows.at(r) + threadIdx.x) + bvs;
  }
  __syncthreads();
  const int na = min(wself, s.N - r);
  const int np = na * wother;
  const size_t stat = static_cast<size_t>(bh) * s.N;

  float acc[D];
#pragma unroll
  for (int d = 0; d < D; ++d) acc[d] = 0.f;
  for (int p = threadIdx.x; p < np; p += kThreads) {
    const int i = r + p / wother;
    const int o = i - p % wother;
    if (o < 0) continue;
    const T* qi = q + rows.at(i);
    const T* ko = kother + rows.at(o);
    const T* doi = dout + rows.at(i);
    const T* vo = vother + rows.at(o);
    const float a = FORM == 0 || SIDE == 1 ? logit3<T, D, FORM>(kr, qi, 0.f, ko, bko)
                                           : logit3<T, D, FORM>(kr, ko, bko, qi, 0.f);
    const float pr = expf(a - lse[stat + i]);
    if (MODE == 0) {
      const float dp = tri<T, D>(vr, doi, 0.f, vo, bvo);
      const float dsv = pr * (dp - delta[stat + i]);
      if (FORM == 0 || SIDE == 1)
        add_partial<T, D, FORM>(acc, dsv, qi, 0.f, ko, bko);
      else
        add_partial<T, D, FORM>(acc, dsv, ko, bko, qi, 0.f);
    } else {
#pragma unroll
      for (int d = 0; d < D; ++d) acc[d] += pr * ld(doi + d) * (ld(vo + d) + bvo);
    }
  }
  const float g = block_sum_vec<D>(acc, red);
  if (threadIdx.x < D) st(grad + rows.at(r) + threadIdx.x, MODE == 0 ? g * s.scale : g);
}

template <typename T, int D, int FORM>
hipError_t fwd_f(const Shape& s, const void* q, const void* k, const void* kp, const void* v,
                 const void* vp, void* out, float* lse, hipStream_t st) {
  const unsigned grid = static_cast<unsigned>(s.N) * s.B * s.H;
  hipLaunchKernelGGL((fwd_kernel<T, D, FORM>), dim3(grid), dim3(kThreads), 0, st, s,
                     static_cast<const T*>(q), static_cast<const T*>(k), static_cast<const T*>(kp),
                     static_cast<const T*>(v), static_cast<const T*>(vp), static_cast<T*>(out),
                     lse);
  return hipGetLastError();
}

template <typename T, int D>
hipError_t fwd_t(const Shape& s, const void* q, const void* k, const void* kp, const void* v,
                 const void* vp, void* out, float* lse, hipStream_t st) {
  return s.form == 0 ? fwd_f<T, D, 0>(s, q, k, kp, v, vp, out, lse, st)
                     : fwd_f<T, D, 1>(s, q, k, kp, v, vp, out, lse, st);
}

template <typename T, int D, int FORM>
hipError_t bwd_stage_f(const Shape& s, BwdStage stage, const T* q, const T* k, const T* kp,
                       const T* v, const T* vp, const T* dout, const float* lse,
                       const float* delta, void* g0, void* g1, void* g2, hipStream_t st) {
  const unsigned grid = static_cast<unsigned>(s.N) * s.B * s.H;
  if (stage == BwdStage::Query) {
    hipLaunchKernelGGL((dq_kernel<T, D, FORM>), dim3(grid), dim3(kThreads), 0, st, s, q, k, kp, v,
                       vp, dout, lse, delta, static_cast<T*>(g0));
    hipLaunchKernelGGL((keyside_kernel<T, D, 1, 0, FORM>), dim3(grid), dim3(kThreads), 0, st, s, q,
                       kp, k, vp, v, dout, lse, delta, static_cast<T*>(g1));
    hipLaunchKernelGGL((keyside_kernel<T, D, 1, 1, FORM>), dim3(grid), dim3(kThreads), 0, st, s, q,
                       kp, k, vp, v, dout, lse, delta, static_cast<T*>(g2));
  } else {
    hipLaunchKernelGGL((keyside_kernel<T, D, 0, 0, FORM>), dim3(grid), dim3(kThreads), 0, st, s, q,
                       k, kp, v, vp, dout, lse, delta, static_cast<T*>(g0));
    hipLaunchKernelGGL((keyside_kernel<T, D, 0, 1, FORM>), dim3(grid), dim3(kThreads), 0, st, s, q,
                       k, kp, v, vp, dout, lse, delta, static_cast<T*>(g1));
  }
  return hipGetLastError();
}

template <typename T, int D>
hipError_t bwd_stage_t(const Shape& s, BwdStage stage, const void* q_, const void* k_, const void* kp_,
                       const void* v_, const void* vp_, const void* dout_, const float* lse,
                       const float* delta, void* g0, void* g1, void* g2, hipStream_t st) {
  const T* q = static_cast<const T*>(q_);
  const T* k = static_cast<const T*>(k_);
  const T* kp = static_cast<const T*>(kp_);
  const T* v = static_cast<const T*>(v_);
  const T* vp = static_cast<const T*>(vp_);
  const T* dout = static_cast<const T*>(dout_);
  return s.form == 0
             ? bwd_stage_f<T, D, 0>(s, stage, q, k, kp, v, vp, dout, lse, delta, g0, g1, g2, st)
             : bwd_stage_f<T, D, 1>(s, stage, q, k, kp, v, vp, dout, lse, delta, g0, g1, g2, st);
}

}  // namespace

#define SA_DISPATCH_D(T, FN, ...)              \
  switch (s.D) {                              \
    case 16: return FN<T, 16>(__VA_ARGS__);   \
    case 32: return FN<T, 32>(__VA_ARGS__);   \
    case 64: return FN<T, 64>(__VA_ARGS__);   \
    case 128: return FN<T, 128>(__VA_ARGS__); \
    default: return hipErrorInvalidValue;     \
  }

hipError_t generic_fwd(const Shape& s, const void* q, const void* k, const void* kp, const void* v,
                       const void* vp, void* out, float* lse, hipStream_t st) {
  if (s.dtype == 0) {
    SA_DISPATCH_D(float, fwd_t, s, q, k, kp, v, vp, out, lse, st);
  }
  SA_DISPATCH_D(uint16_t, fwd_t, s, q, k, kp, v, vp, out, lse, st);
}

hipError_t launch_delta(const Shape& s, const void* out, const void* dout, float* delta,
                        hipStream_t st) {
  const int64_t total = static_cast<int64_t>(s.B) * s.H * s.N;
  const unsigned grid = static_cast<unsigned>((total + 255) / 256);
  if (s.dtype == 0) {
    hipLaunchKernelGGL(delta_kernel<float>, dim3(grid), dim3(256), 0, st, s,
                       static_cast<const float*>(out), static_cast<const float*>(dout), delta);
  } else {
    hipLaunchKernelGGL(delta_kernel<uint16_t>, dim3(grid), dim3(256), 0, st, s,
                       static_cast<const uint16_t*>(out), static_cast<const uint16_t*>(dout),
                       delta);
  }
  return hipGetLastError();
}

hipError_t generic_bwd_stage(const Shape& s, BwdStage stage, const void* q, const void* k,
                             const void* kp, const void* v, const void* vp, const void* dout,
                             const float* lse, const float* delta, void* g0, void* g1, void* g2,
                             hipStream_t st) {
  if (s.dtype == 0) {
    SA_DISPATCH_D(float, bwd_stage_t, s, stage, q, k, kp, v, vp, dout, lse, delta, g0, g1, g2, st);
  }
  SA_DISPATCH_D(uint16_t, bwd_stage_t, s, stage, q, k, kp, v, vp, dout, lse, delta, g0, g1, g2, st);
}

}  // namespace sa
