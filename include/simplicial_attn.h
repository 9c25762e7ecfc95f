/*
 * simplicial_attn.h -- C ABI of the MI355X (gfx950) causal sliding-window
 * 2-simplicial (trilinear) attention library, libsimplicial_attn.so.
 *
 * The operation (arXiv 2507.02754, Section 4 Eqs. (3d-attention), (softmax),
 * (attenval), over the sliding windows of Section 6): for every batch b, head h
 * and query i,
 *
 *     A[i,j,k] = scale * sum_d Q[i,d] K[j,d] K'[k,d]      j in (i-w1, i], k in (i-w2, i]
 *     P[i,j,k] = exp(A[i,j,k] - LSE[i]),  LSE[i] = log sum_{j,k} exp(A[i,j,k])
 *     O[i,d]   = sum_{j,k} P[i,j,k] V[j,d] V'[k,d]
 *
 * Windows are clipped at 0 and include the diagonal, so every query has at
 * least the pair (i, i). The backward computes the gradients of Section 7's
 * equations (dQ, dK, dK' carry one factor of `scale`; dV, dV' none).
 *
 * Conventions shared by every entry point
 *   Layout   Q, K, K', V, V', O, dO and all gradients are contiguous row-major
 *            [B, N, H, D] (batch, sequence, head, head_dim). LSE is contiguous
 *            [B, H, N] float32, natural logarithm.
 *   dtype    SA_DTYPE_F32 or SA_DTYPE_BF16, applied to every tensor except LSE
 *            (always float32). bf16 data is accumulated in float32.
 *   Pointers device pointers (hipMalloc'd or torch CUDA tensors), 16-byte
 *            aligned. The caller owns every buffer; the library allocates no
 *            device memory and keeps no state between calls (re-entrant).
 *   Stream   a hipStream_t passed as void* (NULL = the default stream). Calls
 *            only enqueue work on it and return without synchronising.
 *   Errors   each call returns SA_OK (0) or an SA_ERR_* code. All argument
 *            validation happens on the host before any HIP call, so invalid
 *            calls are rejected even where no GPU is present. No C++ exception
 *            crosses the ABI and the library never aborts. A kernel launch
 *            failure is reported as SA_ERR_HIP; an asynchronous device fault
 *            surfaces on the caller's next synchronisation.
 */
#ifndef SIMPLICIAL_ATTN_H
#define SIMPLICIAL_ATTN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SIMPLICIAL_ATTN_ABI_VERSION 6

#define SA_DTYPE_F32 0
#define SA_DTYPE_BF16 1

#define SA_OK 0
#define SA_ERR_INVALID 1     /* null pointer, non-positive size, w < 1, misaligned pointer, overflow */
#define SA_ERR_UNSUPPORTED 2 /* head_dim or dtype this build does not implement */
#define SA_ERR_WORKSPACE 3   /* workspace smaller than simplicial_attn_bwd_workspace_size() */
#define SA_ERR_HIP 4         /* HIP runtime reported an error when launching */
#define SA_ERR_SCRATCH 5     /* simplicial_attn_bwd_noalloc: sizes need more than its fixed scratch */

/* Bytes of the fixed device scratch array of simplicial_attn_bwd_noalloc (64 MiB per GPU). */
#define SA_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)

/*
 * Forward pass (Section 4 equations over Section 6's windows).
 *   q, k, kp, v, vp  inputs Q, K, K', V, V'   [B, N, H, D], dtype
 *   out              output O                 [B, N, H, D], dtype, fully overwritten
 *   lse              log-sum-exp per query    [B, H, N], float32, fully overwritten
 *   B, N, H, D       sizes; D in {16, 32, 64, 128}
 *   w1, w2           window lengths of K/V and K'/V' (>= 1; larger than N is legal)
 *   scale            logit scale (the paper's 1/sqrt(D)); any finite value
 *   dtype            SA_DTYPE_F32 or SA_DTYPE_BF16
 *   stream           hipStream_t or NULL
 */
int simplicial_attn_fwd(const void* q, const void* k, const void* kp, const void* v, const void* vp,
                        void* out, float* lse, int64_t B, int64_t N, int64_t H, int64_t D, int32_t w1,
                        int32_t w2, float scale, int32_t dtype, void* stream);

/*
 * Forward pass with grouped-query attention (the layout of Section 6's
 * production setting, where many query heads share one K/K'/V/V' head):
 * query head h reads K-side head h / (H / Hkv). Same operation and conventions
 * as simplicial_attn_fwd, except
 *   q, out           [B, N, H, D]
 *   k, kp, v, vp     [B, N, Hkv, D]
 *   lse              [B, H, N]
 *   Hkv              K-side heads, 1 <= Hkv <= H, H % Hkv == 0 (else SA_ERR_INVALID)
 * Hkv == H is exactly simplicial_attn_fwd. The matching backward is
 * simplicial_attn_bwd_gqa.
 */
int simplicial_attn_fwd_gqa(const void* q, const void* k, const void* kp, const void* v,
                            const void* vp, void* out, float* lse, int64_t B, int64_t N, int64_t H,
                            int64_t Hkv, int64_t D, int32_t w1, int32_t w2, float scale,
                            int32_t dtype, void* stream);

/*
 * Bytes of device workspace simplicial_attn_bwd needs for these sizes (the
 * per-query Delta = <dO_i, O_i> and the partial sums the backward reduces
 * deterministically). Returns 0 for arguments simplicial_attn_bwd would reject.
 */
size_t simplicial_attn_bwd_workspace_size(int64_t B, int64_t N, int64_t H, int64_t D, int32_t w1,
                                          int32_t w2, int32_t dtype);

/*
 * Backward pass (Section 7's gradient equations; dsoftmax read as
 * dS = P * (dP - Delta_i), Delta_i = <dO_i, O_i>).
 *   q, k, kp, v, vp    forward inputs                    [B, N, H, D], dtype
 *   out, lse           forward outputs of the same call  [B, N, H, D] dtype / [B, H, N] f32
 *   dout               upstream gradient dO               [B, N, H, D], dtype
 *   dq, dk, dkp, dv, dvp  gradients, fully overwritten   [B, N, H, D], dtype
 *   workspace          device scratch of at least simplicial_attn_bwd_workspace_size()
 *                      bytes, 16-byte aligned; contents on entry are ignored
 *   other arguments    as simplicial_attn_fwd
 * The result is bitwise deterministic: no floating-point atomics are used.
 * It runs Section 7's two kernels (query side and key side; see the stage
 * entry points below). The fused backward below is the alternative with one
 * computation of S and dP.
 */
int simplicial_attn_bwd(const void* q, const void* k, const void* kp, const void* v, const void* vp,
                        const void* out, const void* dout, const float* lse, void* dq, void* dk,
                        void* dkp, void* dv, void* dvp, void* workspace, size_t workspace_bytes,
                        int64_t B, int64_t N, int64_t H, int64_t D, int32_t w1, int32_t w2,
                        float scale, int32_t dtype, void* stream);

/*
 * Forward and backward with the K' and V' bias constants of the paper's
 * Appendix B kernels (the K2_BIAS / V2_BIAS constants, there a "KV2 norm"
 * applied to every loaded K' / V' element): the operation of simplicial_attn_fwd
 * / simplicial_attn_bwd with K' + kp_bias and V' + vp_bias (every element
 * shifted by the constant) in place of K' and V'. Masked pairs stay excluded
 * whatever the constants. dK' and dV' are the gradients with respect to the
 * given K' and V' (a constant shift does not change them). Arguments, layouts,
 * workspace (simplicial_attn_bwd_workspace_size) and errors as the plain pair;
 * non-finite constants are SA_ERR_INVALID. Constants 0 give exactly the plain
 * pair's results.
 */
int simplicial_attn_fwd_biased(const void* q, const void* k, const void* kp, const void* v,
                               const void* vp, void* out, float* lse, int64_t B, int64_t N,
                               int64_t H, int64_t D, int32_t w1, int32_t w2, float scale,
                               float kp_bias, float vp_bias, int32_t dtype, void* stream);
int simplicial_attn_bwd_biased(const void* q, const void* k, const void* kp, const void* v,
                               const void* vp, const void* out, const void* dout, const float* lse,
                               void* dq, void* dk, void* dkp, void* dv, void* dvp, void* workspace,
                               size_t workspace_bytes, int64_t B, int64_t N, int64_t H, int64_t D,
                               int32_t w1, int32_t w2, float scale, float kp_bias, float vp_bias,
                               int32_t dtype, void* stream);

/*
 * The backward without any allocation, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc). Same operation, arguments, results and errors as
 * simplicial_attn_bwd, except that there is no workspace argument: the
 * workspace is a file-scope device array of SA_NOALLOC_SCRATCH_BYTES that each
 * GPU holds from the first call on that device (or the library's first use of
 * it) until the process ends. The call makes no hipMalloc/hipFree and calls no
 * allocating library routine; its first call on a device looks up that
 * device's copy of the array (hipGetSymbolAddress, with the device current).
 *   Limit  the per-query Delta (4 bytes per query and head) plus the partial
 *          sums of the backward's deterministic reduction must fit the array.
 *          When the workspace simplicial_attn_bwd_workspace_size() reports
 *          fits, the kernels, their work split and the result are exactly
 *          those of simplicial_attn_bwd (bitwise). Otherwise the query-side
 *          kernel walks longer query chunks so that fewer partial sums are
 *          kept (same gradients up to the order of fp32 additions at chunk
 *          boundaries, still deterministic); sizes for which even that does
 *          not fit return SA_ERR_SCRATCH, before any HIP call.
 *   Races  every call on one GPU uses that GPU's one array, and every call
 *          overwrites what it reads from it (contents on entry are ignored),
 *          so calls that overlap in time on one GPU (other streams, other
 *          host threads) race; calls ordered on one stream do not.
 */
int simplicial_attn_bwd_noalloc(const void* q, const void* k, const void* kp, const void* v,
                                const void* vp, const void* out, const void* dout, const float* lse,
                                void* dq, void* dk, void* dkp, void* dv, void* dvp, int64_t B,
                                int64_t N, int64_t H, int64_t D, int32_t w1, int32_t w2, float scale,
                                int32_t dtype, void* stream);

/*
 * Forward and backward with the determinant logits of Section 5, Eq. (logits)
 * (rotation-invariant, so usable with position rotations applied to Q, K, K'):
 *   A_ijk = scale * sum_l det([q_i^(l); k_j^(l); k'_k^(l)])
 * over the 3-component chunks l = 0 .. floor(D/3) - 1 (components 3l .. 3l+2);
 * for D not a multiple of 3 the D mod 3 trailing components enter no logit and
 * get zero dQ, dK, dK'. Softmax, output, windows, arguments, layouts and
 * errors are those of simplicial_attn_fwd / simplicial_attn_bwd; the backward
 * workspace is at least simplicial_attn_det_bwd_workspace_size() bytes. Eq.
 * (logits) carries no scale factor: scale = 1 is the paper's form.
 * Kernels: for bf16 data with D in {64, 128} and w2 <= 32 both run on the MFMA
 * kernels (the modulated query of the trilinear kernels is formed as the
 * chunkwise cross product k'_k x q_i; the backward's workspace then also
 * holds the query side's fp32 dQ~ rows, 4 * 32 * D bytes per query and head,
 * from which a separate kernel forms dQ and dK'); every other shape runs on
 * the plain fp32 kernels.
 */
int simplicial_attn_det_fwd(const void* q, const void* k, const void* kp, const void* v,
                            const void* vp, void* out, float* lse, int64_t B, int64_t N, int64_t H,
                            int64_t D, int32_t w1, int32_t w2, float scale, int32_t dtype,
                            void* stream);
size_t simplicial_attn_det_bwd_workspace_size(int64_t B, int64_t N, int64_t H, int64_t D,
                                              int32_t w1, int32_t w2, int32_t dtype);
int simplicial_attn_det_bwd(const void* q, const void* k, const void* kp, const void* v,
                            const void* vp, const void* out, const void* dout, const float* lse,
                            void* dq, void* dk, void* dkp, void* dv, void* dvp, void* workspace,
                            size_t workspace_bytes, int64_t B, int64_t N, int64_t H, int64_t D,
                            int32_t w1, int32_t w2, float scale, int32_t dtype, void* stream);

/*
 * Backward with grouped-query attention, for the outputs of
 * simplicial_attn_fwd_gqa. Every K-side element enters the logits of all the
 * query heads of its group, so dK, dK', dV, dV' are the per-query-head
 * gradients summed over the group (bitwise deterministic). dK', dV': each
 * query head's gradient in dtype, summed in fp32 in ascending head order and
 * rounded once. dK, dV: on the MFMA kernels (bf16, D 64 or 128, w2 <= 64) the
 * key-stationary kernel reads K, K', V, V' in place and accumulates the whole
 * group in fp32 before rounding once; otherwise as dK', dV'.
 *   q, out, dout, dq        [B, N, H, D], dtype
 *   k, kp, v, vp            [B, N, Hkv, D], dtype
 *   dk, dkp, dv, dvp        [B, N, Hkv, D], dtype, fully overwritten
 *   lse                     [B, H, N] float32 from the forward
 *   workspace               at least simplicial_attn_bwd_gqa_workspace_size()
 *                           bytes, 16-byte aligned; contents on entry ignored.
 *                           For Hkv < H it holds, besides what
 *                           simplicial_attn_bwd needs, the per-query-head
 *                           dK', dV' (MFMA kernels: 2 tensors of B*N*H*D
 *                           elements), or K, K', V, V' expanded to H heads
 *                           and all four per-query-head K-side gradients
 *                           (other shapes: 8 such tensors).
 *   Hkv                     as simplicial_attn_fwd_gqa (else SA_ERR_INVALID)
 * Other arguments and errors as simplicial_attn_bwd; Hkv == H is exactly
 * simplicial_attn_bwd. The workspace size function returns 0 for arguments
 * the backward would reject.
 */
size_t simplicial_attn_bwd_gqa_workspace_size(int64_t B, int64_t N, int64_t H, int64_t Hkv,
                                              int64_t D, int32_t w1, int32_t w2, int32_t dtype);
int simplicial_attn_bwd_gqa(const void* q, const void* k, const void* kp, const void* v,
                            const void* vp, const void* out, const void* dout, const float* lse,
                            void* dq, void* dk, void* dkp, void* dv, void* dvp, void* workspace,
                            size_t workspace_bytes, int64_t B, int64_t N, int64_t H, int64_t Hkv,
                            int64_t D, int32_t w1, int32_t w2, float scale, int32_t dtype,
                            void* stream);

/*
 * The backward in three stages, for callers that schedule them themselves.
 * simplicial_attn_bwd is exactly preprocess, then query side, then key side
 * on one stream. Both sides read what preprocess wrote into `workspace` (the
 * per-query Delta); once it has run they are independent of each other.
 *   preprocess  Delta_i = <dO_i, O_i> into the workspace.
 *   query side  dQ, dK', dV' (the query-stationary kernel, Section 7's second
 *               kernel, with the k-halo reduction of Algorithm 2's role).
 *   key side    dK, dV (the key-stationary kernel, Section 7's first kernel).
 * Arguments mean what they mean for simplicial_attn_bwd; the same workspace
 * (same size rule) must be passed to all three.
 */
int simplicial_attn_bwd_preprocess(const void* out, const void* dout, void* workspace,
                                   size_t workspace_bytes, int64_t B, int64_t N, int64_t H,
                                   int64_t D, int32_t w1, int32_t w2, int32_t dtype, void* stream);
int simplicial_attn_bwd_query_side(const void* q, const void* k, const void* kp, const void* v,
                                   const void* vp, const void* dout, const float* lse, void* dq,
                                   void* dkp, void* dvp, void* workspace, size_t workspace_bytes,
                                   int64_t B, int64_t N, int64_t H, int64_t D, int32_t w1,
                                   int32_t w2, float scale, int32_t dtype, void* stream);
int simplicial_attn_bwd_key_side(const void* q, const void* k, const void* kp, const void* v,
                                 const void* vp, const void* dout, const float* lse, void* dk,
                                 void* dv, void* workspace, size_t workspace_bytes, int64_t B,
                                 int64_t N, int64_t H, int64_t D, int32_t w1, int32_t w2,
                                 float scale, int32_t dtype, void* stream);
/*
 * Fused backward: Section 7's five gradients from one computation of S and dP
 * per (row block, key block), instead of the two kernels that each recompute
 * them (12 units of matrix work per query instead of 16). A kernel owns 64
 * keys: it writes dK, dV and its partial sums of dQ, dK', dV' (fp32) to
 * `workspace`; the reduction adds the partial sums of the kernels in a fixed
 * order, so the result is bitwise deterministic (no atomics). Same gradients
 * as simplicial_attn_bwd up to the order of fp32 additions. Sequence on one
 * stream: simplicial_attn_bwd_preprocess (Delta), simplicial_attn_bwd_fused,
 * simplicial_attn_bwd_fused_reduce, all three with the same workspace of at
 * least simplicial_attn_bwd_fused_workspace_size() bytes: Delta plus
 * 4 * B * H * ceil(N / 64) * ((63 + w1) + 2 * (94 + w1)) * D bytes of
 * partial sums (7.5 GB at B=1, H=16, N=32768, D=128, w1=512).
 * Shapes: bf16, head_dim 128, w2 <= 32; the size function returns 0 and the
 * two calls SA_ERR_UNSUPPORTED for others. kp_bias, vp_bias: the K' / V'
 * constants of simplicial_attn_bwd_biased (0 for the plain operation; the
 * reduction takes none). Arguments otherwise as for the stages above.
 */
size_t simplicial_attn_bwd_fused_workspace_size(int64_t B, int64_t N, int64_t H, int64_t D, int32_t w1,
                                                int32_t w2, int32_t dtype);
int simplicial_attn_bwd_fused(const void* q, const void* k, const void* kp, const void* v,
                              const void* vp, const void* dout, const float* lse, void* dk, void* dv,
                              void* workspace, size_t workspace_bytes, int64_t B, int64_t N, int64_t H,
                              int64_t D, int32_t w1, int32_t w2, float scale, float kp_bias,
                              float vp_bias, int32_t dtype, void* stream);
int simplicial_attn_bwd_fused_reduce(void* dq, void* dkp, void* dvp, const void* workspace,
                                     size_t workspace_bytes, int64_t B, int64_t N, int64_t H, int64_t D,
                                     int32_t w1, int32_t w2, float scale, int32_t dtype, void* stream);

/* Static, NUL-terminated description of a status code ("unknown status" otherwise). */
const char* simplicial_attn_error_string(int code);

/* SIMPLICIAL_ATTN_ABI_VERSION of the loaded library. */
int simplicial_attn_abi_version(void);

/*
 * Name of the kernel path the forward (which = 0) or backward (which = 1) would
 * take for these sizes, e.g. "mfma_bf16" or "generic"; "invalid" when the
 * arguments would be rejected. Static string; no HIP call is made.
 */
const char* simplicial_attn_path_name(int32_t which, int64_t B, int64_t N, int64_t H, int64_t D,
                                      int32_t w1, int32_t w2, int32_t dtype);

#ifdef __cplusplus
}
#endif

#endif /* SIMPLICIAL_ATTN_H */
