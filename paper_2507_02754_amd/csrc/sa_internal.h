// Internal declarations shared by the library's translation units (not part of
// the public ABI). Host launchers return hipError_t; the C-ABI layer in api.hip
// maps errors to SA_* status codes.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace sa {

// Problem description after host validation. Tensors are [B, N, H, D]
// contiguous; per-query statistics are [B, H, N].
struct Shape {
  int B, N, H, D;
  int w1, w2;
  float scale;
  int dtype;  // SA_DTYPE_*
  // Heads of K, K', V, V' (grouped-query attention: query head h reads K/V
  // head h / (H / Hkv)). The forward and the MFMA backward kernels read the
  // K side with this head count (the key side walks a group's query heads;
  // the query side writes per-query-head dK', dV' for gqa_group_sum); the
  // generic backward runs with Hkv == H.
  int Hkv;
  // Logit form: 0 trilinear (Section 4), 1 sum of 3 x 3 determinants over
  // 3-component chunks (Section 5).
  int form;
  // Largest backward workspace the caller can provide, in bytes (0: no
  // limit). The MFMA backward plan lengthens its query chunks until its
  // workspace fits (fewer chunk-boundary partial sums).
  size_t ws_cap;
  // Constants added to every element of K' and V' after loading (the
  // K2_BIAS / V2_BIAS constants of the paper's Appendix B kernel); 0 for the
  // plain operation. Masked pairs stay excluded whatever the bias.
  float kp_bias, vp_bias;
};

// bf16 is carried as raw 16-bit patterns (uint16_t) in every kernel.
__device__ __forceinline__ float bf16_to_f32(uint16_t x) {
  return __uint_as_float(static_cast<uint32_t>(x) << 16);
}

// float -> bf16, round to nearest even; NaN stays NaN (quiet bit forced).
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return static_cast<uint16_t>((u >> 16) | 0x40u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return static_cast<uint16_t>(u >> 16);
}

// ---- generic path (any supported dtype / head_dim / windows) --------------
hipError_t generic_fwd(const Shape& s, const void* q, const void* k, const void* kp, const void* v,
                       const void* vp, void* out, float* lse, hipStream_t st);
// The backward is split into a query-side stage (dQ, dK', dV') and a key-side
// stage (dK, dV); both read Delta, which the preprocessing stage writes.
enum class BwdStage { Query, Key };
hipError_t generic_bwd_stage(const Shape& s, BwdStage stage, const void* q, const void* k,
                             const void* kp, const void* v, const void* vp, const void* dout,
                             const float* lse, const float* delta, void* g0, void* g1, void* g2,
                             hipStream_t st);

// ---- gfx950 MFMA path (bf16, head_dim 64/128, w2 <= 64) --------------------
bool mfma_fwd_supported(const Shape& s);
hipError_t mfma_fwd(const Shape& s, const void* q, const void* k, const void* kp, const void* v,
                    const void* vp, void* out, float* lse, hipStream_t st);

// Backward work split and workspace layout of the MFMA path. The workspace
// holds Delta ([B, H, N] floats) followed by four arrays of chunk-boundary
// partial sums (head/tail x dk'/dv', each [B*H, nchunks, W2P - 1, D] floats);
// with determinant logits then the query side's dQ~ rows ([B*H, N, 32, D]
// floats at dqt_off).
struct BwdPlan {
  int G, W2P, CQ, nchunks;
  size_t halo_floats, delta_off, halo_off, dqt_off, bytes;
};
BwdPlan mfma_bwd_plan(const Shape& s);
bool mfma_bwd_supported(const Shape& s);
hipError_t mfma_bwd_delta(const Shape& s, const void* out, const void* dout, void* workspace,
                          hipStream_t st);
// Query side: g0 = dq, g1 = dk', g2 = dv'. Key side: g0 = dk, g1 = dv.
hipError_t mfma_bwd_stage(const Shape& s, BwdStage stage, const void* q, const void* k,
                          const void* kp, const void* v, const void* vp, const void* dout,
                          const float* lse, void* g0, void* g1, void* g2, void* workspace,
                          hipStream_t st);

// Key-side backward stage of the MFMA path (dK, dV) given Delta.
hipError_t mfma_bwd_key(const Shape& s, const void* q, const void* k, const void* kp, const void* v,
                        const void* vp, const void* dout, const float* lse, const float* delta,
                        void* dk, void* dv, hipStream_t st);

// Fused backward (w2 <= 32, trilinear logits, bf16, head_dim 128, one K-side
// head per query head): one kernel computes S and dP once per (row block, key
// group) and produces dK, dV directly and per-workgroup partial sums of dq,
// dk', dv'; a second kernel adds the partials. A workgroup owns kw keys.
// Workspace: Delta ([B, H, N] floats, as in BwdPlan) then the partials,
// offsets in floats: dq at pq_off ([B*H, njb, RQ, D]; row i - kw jb), dk' at
// pk_off and dv' at pv_off ([B*H, njb, RK, D]; row k - kw jb + 31),
// njb = ceil(N / kw), RQ = kw - 1 + w1, RK = kw + 30 + w1.
struct FusedPlan {
  int kw, njb, RQ, RK;
  size_t delta_floats, pq_off, pk_off, pv_off, bytes;
};
FusedPlan mfma_fused_plan(const Shape& s);
bool mfma_fused_supported(const Shape& s);
hipError_t mfma_bwd_fused(const Shape& s, const void* q, const void* k, const void* kp, const void* v,
                          const void* vp, const void* dout, const float* lse, void* dk, void* dv,
                          void* workspace, hipStream_t st);
hipError_t mfma_bwd_fused_reduce(const Shape& s, void* dq, void* dkp, void* dvp, const void* workspace,
                                 hipStream_t st);

// Query-side backward stage for w2 <= 32 (dq, dk', dv' and the chunk-boundary
// partial sums in `halo`; the fix-up kernel runs afterwards).
bool mfma_bwd_query_supported(const Shape& s);
hipError_t mfma_bwd_query(const Shape& s, const BwdPlan& plan, const void* q, const void* k,
                          const void* kp, const void* v, const void* vp, const void* dout,
                          const float* lse, const float* delta, void* dq, void* dkp, void* dvp,
                          float* halo, float* dqt, hipStream_t st);

// Grouped-query backward helpers (s.H query heads, s.Hkv K-side heads; the
// four src/dst pointers are K, K', V, V' or their gradients).
// gqa_expand: dst[t] [B, N, H, D] = src[t] [B, N, Hkv, D] with head h taken
// from K-side head h / (H / Hkv).
hipError_t gqa_expand(const Shape& s, const void* const src[4], void* const dst[4],
                      hipStream_t st);
// gqa_group_sum: dst[t] [B, N, Hkv, D] = fp32 sum over each group's query
// heads (ascending) of src[t] [B, N, H, D], rounded once to the data type,
// for t < ntens.
hipError_t gqa_group_sum(const Shape& s, const void* const src[4], void* const dst[4],
                         hipStream_t st, int ntens = 4);

// Delta_i = <dO_i, O_i> for every query, [B, H, N] float32.
hipError_t launch_delta(const Shape& s, const void* out, const void* dout, float* delta,
                        hipStream_t st);

}  // namespace sa
