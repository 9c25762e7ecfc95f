// C-ABI entry points of libsimplicial_attn.so: argument validation (host only,
// before any HIP call), kernel-path selection and error mapping. The
// operation and the conventions are documented in include/simplicial_attn.h.
#include "simplicial_attn.h"

#include <limits.h>
#include <math.h>

#include <initializer_list>
#include <mutex>

#include "sa_internal.h"

namespace {

using sa::BwdStage;
using sa::Shape;

enum class Path { Invalid, Generic, Mfma };

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

int check_ptrs(std::initializer_list<const void*> ptrs) {
  for (const void* p : ptrs) {
    if (!p || !aligned16(p)) return SA_ERR_INVALID;
  }
  return SA_OK;
}

// Size checks shared by every entry point. Returns SA_OK or an error code.
int check_sizes(int64_t B, int64_t N, int64_t H, int64_t D, int32_t w1, int32_t w2,
                int32_t dtype) {
  if (B <= 0 || N <= 0 || H <= 0 || D <= 0 || w1 < 1 || w2 < 1) return SA_ERR_INVALID;
  // Every grid index and per-head row count must fit in 32 bits, and element
  // offsets comfortably in 64 bits.
  if (N > INT_MAX || B > INT_MAX || H > INT_MAX || D > INT_MAX) return SA_ERR_INVALID;
  const int64_t rows = B * H;
  if (rows > INT_MAX || N > INT_MAX / rows) return SA_ERR_INVALID;
  if (D > (int64_t(1) << 40) / (N * rows)) return SA_ERR_INVALID;
  if (dtype != SA_DTYPE_F32 && dtype != SA_DTYPE_BF16) return SA_ERR_UNSUPPORTED;
  if (D != 16 && D != 32 && D != 64 && D != 128) return SA_ERR_UNSUPPORTED;
  return SA_OK;
}

Shape make_shape(int64_t B, int64_t N, int64_t H, int64_t D, int32_t w1, int32_t w2, float scale,
                 int32_t dtype) {
  Shape s;
  s.B = static_cast<int>(B);
  s.N = static_cast<int>(N);
  s.H = static_cast<int>(H);
  s.D = static_cast<int>(D);
  // Windows longer than the sequence behave exactly like the sequence length.
  s.w1 = static_cast<int>(w1 > N ? N : w1);
  s.w2 = static_cast<int>(w2 > N ? N : w2);
  s.scale = scale;
  s.dtype = dtype;
  s.Hkv = s.H;
  s.form = 0;
  s.ws_cap = 0;
  s.kp_bias = 0.f;
  s.vp_bias = 0.f;
  return s;
}

Path choose_path(int which, int64_t B, int64_t N, int64_t H, int64_t D, int32_t w1, int32_t w2,
                 int32_t dtype) {
  if (check_sizes(B, N, H, D, w1, w2, dtype) != SA_OK) return Path::Invalid;
  const Shape s = make_shape(B, N, H, D, w1, w2, 1.0f, dtype);
  if (which == 0 && sa::mfma_fwd_supported(s)) return Path::Mfma;
  if (which == 1 && sa::mfma_bwd_supported(s)) return Path::Mfma;
  return Path::Generic;
}

// Shapes the fused backward kernel takes.
bool fused_path(const Shape& s) { return sa::mfma_fused_supported(s); }

size_t workspace_bytes_for(int64_t B, int64_t N, int64_t H, int64_t D, int32_t w1, int32_t w2,
                           int32_t dtype) {
  if (check_sizes(B, N, H, D, w1, w2, dtype) != SA_OK) return 0;
  if (choose_path(1, B, N, H, D, w1, w2, dtype) == Path::Mfma)
    return sa::mfma_bwd_plan(make_shape(B, N, H, D, w1, w2, 1.0f, dtype)).bytes;
  // Delta: one float per (b, h, query), rounded up to 256 bytes.
  return ((static_cast<size_t>(B * H * N) * sizeof(float)) + 255) & ~size_t(255);
}

// Backward workspace of the determinant logits: the MFMA plan (with the dQ~
// rows) where the MFMA kernels take the shape, else Delta only.
size_t det_workspace_bytes_for(int64_t B, int64_t N, int64_t H, int64_t D, int32_t w1, int32_t w2,
                               int32_t dtype) {
  if (check_sizes(B, N, H, D, w1, w2, dtype) != SA_OK) return 0;
  Shape s = make_shape(B, N, H, D, w1, w2, 1.0f, dtype);
  s.form = 1;
  if (sa::mfma_bwd_supported(s)) return sa::mfma_bwd_plan(s).bytes;
  return ((static_cast<size_t>(B * H * N) * sizeof(float)) + 255) & ~size_t(255);
}

// Backward workspace with Hkv K-side heads: the per-head backward's workspace,
// then (Hkv < H only) per-query-head gradients of the data type, each
// [B, N, H, D]: on the MFMA path dK' and dV' (the key side sums the group
// itself), on the generic path K, K', V, V' expanded to H heads and dK, dK',
// dV, dV' before the group sum.
struct GqaLayout {
  size_t base, per_tensor, bytes;
};

// Whether the grouped-query backward takes the MFMA kernels with the K side
// read in place (no expansion).
bool gqa_native(const Shape& s) { return s.form == 0 && sa::mfma_bwd_supported(s); }

GqaLayout gqa_layout(int64_t B, int64_t N, int64_t H, int64_t Hkv, int64_t D, int32_t w1,
                     int32_t w2, int32_t dtype) {
  GqaLayout l{0, 0, 0};
  if (check_sizes(B, N, H, D, w1, w2, dtype) != SA_OK) return l;
  if (Hkv <= 0 || Hkv > H || H % Hkv != 0) return l;
  l.base = (workspace_bytes_for(B, N, H, D, w1, w2, dtype) + 255) & ~size_t(255);
  if (Hkv == H) {
    l.bytes = workspace_bytes_for(B, N, H, D, w1, w2, dtype);
    return l;
  }
  const size_t esize = dtype == SA_DTYPE_BF16 ? 2 : 4;
  l.per_tensor = (static_cast<size_t>(B * N * H * D) * esize + 255) & ~size_t(255);
  const bool native = gqa_native(make_shape(B, N, H, D, w1, w2, 1.0f, dtype));
  l.bytes = l.base + (native ? 2 : 8) * l.per_tensor;
  return l;
}

int to_status(hipError_t e) { return e == hipSuccess ? SA_OK : SA_ERR_HIP; }

// Common validation of the backward entry points (pointers checked by callers).
int check_bwd(int64_t B, int64_t N, int64_t H, int64_t D, int32_t w1, int32_t w2, float scale,
              int32_t dtype, size_t workspace_bytes) {
  if (!isfinite(scale)) return SA_ERR_INVALID;
  const int rc = check_sizes(B, N, H, D, w1, w2, dtype);
  if (rc != SA_OK) return rc;
  if (workspace_bytes < workspace_bytes_for(B, N, H, D, w1, w2, dtype)) return SA_ERR_WORKSPACE;
  return SA_OK;
}

// Forward with Hkv K/V heads (Hkv == H: the plain forward) and K'/V' bias
// constants (0: none).
int forward(const void* q, const void* k, const void* kp, const void* v, const void* vp, void* out,
            float* lse, int64_t B, int64_t N, int64_t H, int64_t Hkv, int64_t D, int32_t w1,
            int32_t w2, float scale, int32_t dtype, void* stream, float kp_bias = 0.f,
            float vp_bias = 0.f) {
  if (check_ptrs({q, k, kp, v, vp, out, lse}) != SA_OK) return SA_ERR_INVALID;
  if (!isfinite(scale) || !isfinite(kp_bias) || !isfinite(vp_bias)) return SA_ERR_INVALID;
  if (Hkv <= 0 || Hkv > H || H % Hkv != 0) return SA_ERR_INVALID;
  const int rc = check_sizes(B, N, H, D, w1, w2, dtype);
  if (rc != SA_OK) return rc;
  Shape s = make_shape(B, N, H, D, w1, w2, scale, dtype);
  s.Hkv = static_cast<int>(Hkv);
  s.kp_bias = kp_bias;
  s.vp_bias = vp_bias;
  hipStream_t st = static_cast<hipStream_t>(stream);
  switch (choose_path(0, B, N, H, D, w1, w2, dtype)) {
    case Path::Generic: return to_status(sa::generic_fwd(s, q, k, kp, v, vp, out, lse, st));
    case Path::Mfma: return to_status(sa::mfma_fwd(s, q, k, kp, v, vp, out, lse, st));
    default: return SA_ERR_UNSUPPORTED;
  }
}

int run_delta(const Shape& s, Path path, const void* out, const void* dout, void* workspace,
              hipStream_t st) {
  if (path == Path::Mfma) return to_status(sa::mfma_bwd_delta(s, out, dout, workspace, st));
  return to_status(sa::launch_delta(s, out, dout, static_cast<float*>(workspace), st));
}

int run_stage(const Shape& s, Path path, BwdStage stage, const void* q, const void* k,
              const void* kp, const void* v, const void* vp, const void* dout, const float* lse,
              void* g0, void* g1, void* g2, void* workspace, hipStream_t st) {
  if (path == Path::Mfma)
    return to_status(
        sa::mfma_bwd_stage(s, stage, q, k, kp, v, vp, dout, lse, g0, g1, g2, workspace, st));
  return to_status(sa::generic_bwd_stage(s, stage, q, k, kp, v, vp, dout, lse,
                                         static_cast<const float*>(workspace), g0, g1, g2, st));
}

// ---- device scratch of the allocation-free backward ----
//
// The workspace of simplicial_attn_bwd_noalloc is this file-scope device
// array: each GPU the library runs on holds its own copy, at its own address,
// until the process ends. In host code the name `scratch` is only a host-side
// stand-in for the symbol, so it is never passed to a kernel or a copy: the
// device address comes from hipGetSymbolAddress, taken once per device with
// that device current and kept per device.
constexpr size_t kScratchBytes = SA_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices];

// Device address of the current device's scratch array (SA_OK), or SA_ERR_HIP.
int current_device_scratch(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) {
    (void)hipGetLastError();
    return SA_ERR_HIP;
  }
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr) {
      (void)hipGetLastError();
      return SA_ERR_HIP;
    }
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return SA_OK;
}

}  // namespace

extern "C" {

int simplicial_attn_abi_version(void) { return SIMPLICIAL_ATTN_ABI_VERSION; }

const char* simplicial_attn_error_string(int code) {
  switch (code) {
    case SA_OK: return "success";
    case SA_ERR_INVALID: return "invalid argument (null/misaligned pointer, bad size or window)";
    case SA_ERR_UNSUPPORTED: return "unsupported head_dim or dtype";
    case SA_ERR_WORKSPACE: return "workspace smaller than simplicial_attn_bwd_workspace_size()";
    case SA_ERR_HIP: return "HIP runtime error while launching kernels";
    case SA_ERR_SCRATCH:
      return "problem needs more device scratch than the allocation-free backward's fixed "
             "SA_NOALLOC_SCRATCH_BYTES";
    default: return "unknown status";
  }
}

const char* simplicial_attn_path_name(int32_t which, int64_t B, int64_t N, int64_t H, int64_t D,
                                      int32_t w1, int32_t w2, int32_t dtype) {
  if (which != 0 && which != 1) return "invalid";
  switch (choose_path(which, B, N, H, D, w1, w2, dtype)) {
    case Path::Generic: return "generic";
    case Path::Mfma: return "mfma_bf16";
    default: return "invalid";
  }
}

int simplicial_attn_fwd(const void* q, const void* k, const void* kp, const void* v, const void* vp,
                        void* out, float* lse, int64_t B, int64_t N, int64_t H, int64_t D, int32_t w1,
                        int32_t w2, float scale, int32_t dtype, void* stream) {
  return forward(q, k, kp, v, vp, out, lse, B, N, H, H, D, w1, w2, scale, dtype, stream);
}

int simplicial_attn_fwd_gqa(const void* q, const void* k, const void* kp, const void* v,
                            const void* vp, void* out, float* lse, int64_t B, int64_t N, int64_t H,
                            int64_t Hkv, int64_t D, int32_t w1, int32_t w2, float scale,
                            int32_t dtype, void* stream) {
  return forward(q, k, kp, v, vp, out, lse, B, N, H, Hkv, D, w1, w2, scale, dtype, stream);
}

size_t simplicial_attn_bwd_workspace_size(int64_t B, int64_t N, int64_t H, int64_t D, int32_t w1,
                                          int32_t w2, int32_t dtype) {
  return workspace_bytes_for(B, N, H, D, w1, w2, dtype);
}

int simplicial_attn_bwd_preprocess(const void* out, const void* dout, void* workspace,
                                   size_t workspace_bytes, int64_t B, int64_t N, int64_t H,
                                   int64_t D, int32_t w1, int32_t w2, int32_t dtype, void* stream) {
  if (check_ptrs({out, dout, workspace}) != SA_OK) return SA_ERR_INVALID;
  const int rc = check_bwd(B, N, H, D, w1, w2, 1.0f, dtype, workspace_bytes);
  if (rc != SA_OK) return rc;
  const Shape s = make_shape(B, N, H, D, w1, w2, 1.0f, dtype);
  return run_delta(s, choose_path(1, B, N, H, D, w1, w2, dtype), out, dout, workspace,
                   static_cast<hipStream_t>(stream));
}

int simplicial_attn_bwd_query_side(const void* q, const void* k, const void* kp, const void* v,
                                   const void* vp, const void* dout, const float* lse, void* dq,
                                   void* dkp, void* dvp, void* workspace, size_t workspace_bytes,
                                   int64_t B, int64_t N, int64_t H, int64_t D, int32_t w1,
                                   int32_t w2, float scale, int32_t dtype, void* stream) {
  if (check_ptrs({q, k, kp, v, vp, dout, lse, dq, dkp, dvp, workspace}) != SA_OK)
    return SA_ERR_INVALID;
  const int rc = check_bwd(B, N, H, D, w1, w2, scale, dtype, workspace_bytes);
  if (rc != SA_OK) return rc;
  const Shape s = make_shape(B, N, H, D, w1, w2, scale, dtype);
  return run_stage(s, choose_path(1, B, N, H, D, w1, w2, dtype), BwdStage::Query, q, k, kp, v, vp,
                   dout, lse, dq, dkp, dvp, workspace, static_cast<hipStream_t>(stream));
}

int simplicial_attn_bwd_key_side(const void* q, const void* k, const void* kp, const void* v,
                                 const void* vp, const void* dout, const float* lse, void* dk,
                                 void* dv, void* workspace, size_t workspace_bytes, int64_t B,
                                 int64_t N, int64_t H, int64_t D, int32_t w1, int32_t w2,
                                 float scale, int32_t dtype, void* stream) {
  if (check_ptrs({q, k, kp, v, vp, dout, lse, dk, dv, workspace}) != SA_OK) return SA_ERR_INVALID;
  const int rc = check_bwd(B, N, H, D, w1, w2, scale, dtype, workspace_bytes);
  if (rc != SA_OK) return rc;
  const Shape s = make_shape(B, N, H, D, w1, w2, scale, dtype);
  return run_stage(s, choose_path(1, B, N, H, D, w1, w2, dtype), BwdStage::Key, q, k, kp, v, vp,
                   dout, lse, dk, dv, nullptr, workspace, static_cast<hipStream_t>(stream));
}

int simplicial_attn_bwd(const void* q, const void* k, const void* kp, const void* v, const void* vp,
                        const void* out, const void* dout, const float* lse, void* dq, void* dk,
                        void* dkp, void* dv, void* dvp, void* workspace, size_t workspace_bytes,
                        int64_t B, int64_t N, int64_t H, int64_t D, int32_t w1, int32_t w2,
                        float scale, int32_t dtype, void* stream) {
  return simplicial_attn_bwd_biased(q, k, kp, v, vp, out, dout, lse, dq, dk, dkp, dv, dvp,
                                    workspace, workspace_bytes, B, N, H, D, w1, w2, scale, 0.f, 0.f,
                                    dtype, stream);
}

int simplicial_attn_fwd_biased(const void* q, const void* k, const void* kp, const void* v,
                               const void* vp, void* out, float* lse, int64_t B, int64_t N,
                               int64_t H, int64_t D, int32_t w1, int32_t w2, float scale,
                               float kp_bias, float vp_bias, int32_t dtype, void* stream) {
  return forward(q, k, kp, v, vp, out, lse, B, N, H, H, D, w1, w2, scale, dtype, stream, kp_bias,
                 vp_bias);
}

int simplicial_attn_bwd_biased(const void* q, const void* k, const void* kp, const void* v,
                               const void* vp, const void* out, const void* dout, const float* lse,
                               void* dq, void* dk, void* dkp, void* dv, void* dvp, void* workspace,
                               size_t workspace_bytes, int64_t B, int64_t N, int64_t H, int64_t D,
                               int32_t w1, int32_t w2, float scale, float kp_bias, float vp_bias,
                               int32_t dtype, void* stream) {
  if (check_ptrs({q, k, kp, v, vp, out, dout, lse, dq, dk, dkp, dv, dvp, workspace}) != SA_OK)
    return SA_ERR_INVALID;
  if (!isfinite(kp_bias) || !isfinite(vp_bias)) return SA_ERR_INVALID;
  const int rc = check_bwd(B, N, H, D, w1, w2, scale, dtype, workspace_bytes);
  if (rc != SA_OK) return rc;
  Shape s = make_shape(B, N, H, D, w1, w2, scale, dtype);
  s.kp_bias = kp_bias;
  s.vp_bias = vp_bias;
  const Path path = choose_path(1, B, N, H, D, w1, w2, dtype);
  hipStream_t st = static_cast<hipStream_t>(stream);
  int r = run_delta(s, path, out, dout, workspace, st);
  if (r != SA_OK) return r;
  r = run_stage(s, path, BwdStage::Query, q, k, kp, v, vp, dout, lse, dq, dkp, dvp, workspace, st);
  if (r != SA_OK) return r;
  return run_stage(s, path, BwdStage::Key, q, k, kp, v, vp, dout, lse, dk, dv, nullptr, workspace,
                   st);
}

size_t simplicial_attn_bwd_fused_workspace_size(int64_t B, int64_t N, int64_t H, int64_t D, int32_t w1,
                                                int32_t w2, int32_t dtype) {
  if (check_sizes(B, N, H, D, w1, w2, dtype) != SA_OK) return 0;
  const Shape s = make_shape(B, N, H, D, w1, w2, 1.0f, dtype);
  return fused_path(s) ? sa::mfma_fused_plan(s).bytes : 0;
}

// Validation shared by the fused entry points.
static int check_fused(int64_t B, int64_t N, int64_t H, int64_t D, int32_t w1, int32_t w2, float scale,
                int32_t dtype, size_t workspace_bytes) {
  if (!isfinite(scale)) return SA_ERR_INVALID;
  const int rc = check_sizes(B, N, H, D, w1, w2, dtype);
  if (rc != SA_OK) return rc;
  const size_t need = simplicial_attn_bwd_fused_workspace_size(B, N, H, D, w1, w2, dtype);
  if (need == 0) return SA_ERR_UNSUPPORTED;
  return workspace_bytes < need ? SA_ERR_WORKSPACE : SA_OK;
}

int simplicial_attn_bwd_fused(const void* q, const void* k, const void* kp, const void* v,
                              const void* vp, const void* dout, const float* lse, void* dk, void* dv,
                              void* workspace, size_t workspace_bytes, int64_t B, int64_t N, int64_t H,
                              int64_t D, int32_t w1, int32_t w2, float scale, float kp_bias,
                              float vp_bias, int32_t dtype, void* stream) {
  if (check_ptrs({q, k, kp, v, vp, dout, lse, dk, dv, workspace}) != SA_OK) return SA_ERR_INVALID;
  if (!isfinite(kp_bias) || !isfinite(vp_bias)) return SA_ERR_INVALID;
  const int rc = check_fused(B, N, H, D, w1, w2, scale, dtype, workspace_bytes);
  if (rc != SA_OK) return rc;
  Shape s = make_shape(B, N, H, D, w1, w2, scale, dtype);
  s.kp_bias = kp_bias;
  s.vp_bias = vp_bias;
  return to_status(sa::mfma_bwd_fused(s, q, k, kp, v, vp, dout, lse, dk, dv, workspace,
                                      static_cast<hipStream_t>(stream)));
}

int simplicial_attn_bwd_fused_reduce(void* dq, void* dkp, void* dvp, const void* workspace,
                                     size_t workspace_bytes, int64_t B, int64_t N, int64_t H, int64_t D,
                                     int32_t w1, int32_t w2, float scale, int32_t dtype, void* stream) {
  if (check_ptrs({dq, dkp, dvp, workspace}) != SA_OK) return SA_ERR_INVALID;
  const int rc = check_fused(B, N, H, D, w1, w2, scale, dtype, workspace_bytes);
  if (rc != SA_OK) return rc;
  const Shape s = make_shape(B, N, H, D, w1, w2, scale, dtype);
  return to_status(sa::mfma_bwd_fused_reduce(s, dq, dkp, dvp, workspace, static_cast<hipStream_t>(stream)));
}

int simplicial_attn_bwd_noalloc(const void* q, const void* k, const void* kp, const void* v,
                                const void* vp, const void* out, const void* dout, const float* lse,
                                void* dq, void* dk, void* dkp, void* dv, void* dvp, int64_t B,
                                int64_t N, int64_t H, int64_t D, int32_t w1, int32_t w2, float scale,
                                int32_t dtype, void* stream) {
  if (check_ptrs({q, k, kp, v, vp, out, dout, lse, dq, dk, dkp, dv, dvp}) != SA_OK)
    return SA_ERR_INVALID;
  if (!isfinite(scale)) return SA_ERR_INVALID;
  const int rc = check_sizes(B, N, H, D, w1, w2, dtype);
  if (rc != SA_OK) return rc;
  Shape s = make_shape(B, N, H, D, w1, w2, scale, dtype);
  s.ws_cap = kScratchBytes;
  const Path path = choose_path(1, B, N, H, D, w1, w2, dtype);
  const size_t need = path == Path::Mfma ? sa::mfma_bwd_plan(s).bytes
                                         : workspace_bytes_for(B, N, H, D, w1, w2, dtype);
  if (need > kScratchBytes) return SA_ERR_SCRATCH;
  void* ws = nullptr;
  int r = current_device_scratch(&ws);
  if (r != SA_OK) return r;
  hipStream_t st = static_cast<hipStream_t>(stream);
  r = run_delta(s, path, out, dout, ws, st);
  if (r != SA_OK) return r;
  r = run_stage(s, path, BwdStage::Query, q, k, kp, v, vp, dout, lse, dq, dkp, dvp, ws, st);
  if (r != SA_OK) return r;
  return run_stage(s, path, BwdStage::Key, q, k, kp, v, vp, dout, lse, dk, dv, nullptr, ws, st);
}

int simplicial_attn_det_fwd(const void* q, const void* k, const void* kp, const void* v,
                            const void* vp, void* out, float* lse, int64_t B, int64_t N, int64_t H,
                            int64_t D, int32_t w1, int32_t w2, float scale, int32_t dtype,
                            void* stream) {
  if (check_ptrs({q, k, kp, v, vp, out, lse}) != SA_OK) return SA_ERR_INVALID;
  if (!isfinite(scale)) return SA_ERR_INVALID;
  const int rc = check_sizes(B, N, H, D, w1, w2, dtype);
  if (rc != SA_OK) return rc;
  Shape s = make_shape(B, N, H, D, w1, w2, scale, dtype);
  s.form = 1;
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (sa::mfma_fwd_supported(s)) return to_status(sa::mfma_fwd(s, q, k, kp, v, vp, out, lse, st));
  return to_status(sa::generic_fwd(s, q, k, kp, v, vp, out, lse, st));
}

size_t simplicial_attn_det_bwd_workspace_size(int64_t B, int64_t N, int64_t H, int64_t D,
                                              int32_t w1, int32_t w2, int32_t dtype) {
  return det_workspace_bytes_for(B, N, H, D, w1, w2, dtype);
}

int simplicial_attn_det_bwd(const void* q, const void* k, const void* kp, const void* v,
                            const void* vp, const void* out, const void* dout, const float* lse,
                            void* dq, void* dk, void* dkp, void* dv, void* dvp, void* workspace,
                            size_t workspace_bytes, int64_t B, int64_t N, int64_t H, int64_t D,
                            int32_t w1, int32_t w2, float scale, int32_t dtype, void* stream) {
  if (check_ptrs({q, k, kp, v, vp, out, dout, lse, dq, dk, dkp, dv, dvp, workspace}) != SA_OK)
    return SA_ERR_INVALID;
  if (!isfinite(scale)) return SA_ERR_INVALID;
  const int rc = check_sizes(B, N, H, D, w1, w2, dtype);
  if (rc != SA_OK) return rc;
  if (workspace_bytes < det_workspace_bytes_for(B, N, H, D, w1, w2, dtype)) return SA_ERR_WORKSPACE;
  Shape s = make_shape(B, N, H, D, w1, w2, scale, dtype);
  s.form = 1;
  const Path path = sa::mfma_bwd_supported(s) ? Path::Mfma : Path::Generic;
  hipStream_t st = static_cast<hipStream_t>(stream);
  int r = run_delta(s, path, out, dout, workspace, st);
  if (r != SA_OK) return r;
  r = run_stage(s, path, BwdStage::Query, q, k, kp, v, vp, dout, lse, dq, dkp, dvp, workspace, st);
  if (r != SA_OK) return r;
  return run_stage(s, path, BwdStage::Key, q, k, kp, v, vp, dout, lse, dk, dv, nullptr, workspace,
                   st);
}

size_t simplicial_attn_bwd_gqa_workspace_size(int64_t B, int64_t N, int64_t H, int64_t Hkv,
                                              int64_t D, int32_t w1, int32_t w2, int32_t dtype) {
  return gqa_layout(B, N, H, Hkv, D, w1, w2, dtype).bytes;
}

int simplicial_attn_bwd_gqa(const void* q, const void* k, const void* kp, const void* v,
                            const void* vp, const void* out, const void* dout, const float* lse,
                            void* dq, void* dk, void* dkp, void* dv, void* dvp, void* workspace,
                            size_t workspace_bytes, int64_t B, int64_t N, int64_t H, int64_t Hkv,
                            int64_t D, int32_t w1, int32_t w2, float scale, int32_t dtype,
                            void* stream) {
  if (check_ptrs({q, k, kp, v, vp, out, dout, lse, dq, dk, dkp, dv, dvp, workspace}) != SA_OK)
    return SA_ERR_INVALID;
  if (Hkv <= 0 || Hkv > H || H % Hkv != 0) return SA_ERR_INVALID;
  const int rc = check_bwd(B, N, H, D, w1, w2, scale, dtype, workspace_bytes);
  if (rc != SA_OK) return rc;
  const GqaLayout l = gqa_layout(B, N, H, Hkv, D, w1, w2, dtype);
  if (workspace_bytes < l.bytes) return SA_ERR_WORKSPACE;
  if (Hkv == H)
    return simplicial_attn_bwd(q, k, kp, v, vp, out, dout, lse, dq, dk, dkp, dv, dvp, workspace,
                               workspace_bytes, B, N, H, D, w1, w2, scale, dtype, stream);
  Shape s = make_shape(B, N, H, D, w1, w2, scale, dtype);
  s.Hkv = static_cast<int>(Hkv);
  hipStream_t st = static_cast<hipStream_t>(stream);
  char* ws = static_cast<char*>(workspace);
  if (gqa_native(s)) {
    // K side read in place: the query side writes each query head's dK', dV'
    // (summed over the group afterwards), the key side accumulates dK, dV
    // over the group's query heads itself.
    void* gkp = ws + l.base;
    void* gvp = ws + l.base + l.per_tensor;
    int r = run_delta(s, Path::Mfma, out, dout, workspace, st);
    if (r != SA_OK) return r;
    r = run_stage(s, Path::Mfma, BwdStage::Query, q, k, kp, v, vp, dout, lse, dq, gkp, gvp, workspace, st);
    if (r != SA_OK) return r;
    r = run_stage(s, Path::Mfma, BwdStage::Key, q, k, kp, v, vp, dout, lse, dk, dv, nullptr, workspace, st);
    if (r != SA_OK) return r;
    const void* gsrc[4] = {gkp, gvp, nullptr, nullptr};
    void* gdst[4] = {dkp, dvp, nullptr, nullptr};
    return to_status(sa::gqa_group_sum(s, gsrc, gdst, st, 2));
  }
  void* ex[4];  // K, K', V, V' expanded to H heads
  void* gx[4];  // per-query-head dK, dK', dV, dV'
  for (int t = 0; t < 4; ++t) {
    ex[t] = ws + l.base + t * l.per_tensor;
    gx[t] = ws + l.base + (4 + t) * l.per_tensor;
  }
  const void* src[4] = {k, kp, v, vp};
  int r = to_status(sa::gqa_expand(s, src, ex, st));
  if (r != SA_OK) return r;
  r = simplicial_attn_bwd(q, ex[0], ex[1], ex[2], ex[3], out, dout, lse, dq, gx[0], gx[1], gx[2],
                          gx[3], workspace, l.base, B, N, H, D, w1, w2, scale, dtype, stream);
  if (r != SA_OK) return r;
  const void* gsrc[4] = {gx[0], gx[1], gx[2], gx[3]};
  void* gdst[4] = {dk, dkp, dv, dvp};
  return to_status(sa::gqa_group_sum(s, gsrc, gdst, st));
}

}  // extern "C"
