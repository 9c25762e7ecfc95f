"""ctypes binding of libsimplicial_attn.so (argument marshalling only).

Every function here has the name of the C entry point it calls and does no
arithmetic of its own: tensors are checked for device, dtype, layout and shape,
outputs/workspace are allocated with torch (device memory only), and the raw
pointers plus torch's current HIP stream are handed to the library. If the
library has not been built the import of the first call raises; there is no
fallback implementation.
"""

import ctypes
import os

import torch

__all__ = [
    "SimplicialAttnError",
    "load_library",
    "simplicial_attn_fwd",
    "simplicial_attn_fwd_gqa",
    "simplicial_attn_bwd",
    "simplicial_attn_bwd_gqa",
    "simplicial_attn_bwd_noalloc",
    "simplicial_attn_fwd_biased",
    "simplicial_attn_bwd_biased",
    "simplicial_attn_det_fwd",
    "simplicial_attn_det_bwd",
    "simplicial_attn_bwd_gqa_workspace_size",
    "simplicial_attn_det_bwd_workspace_size",
    "simplicial_attn_bwd_preprocess",
    "simplicial_attn_bwd_query_side",
    "simplicial_attn_bwd_key_side",
    "simplicial_attn_bwd_fused",
    "simplicial_attn_bwd_fused_reduce",
    "simplicial_attn_bwd_fused_workspace_size",
    "simplicial_attn_bwd_workspace_size",
    "simplicial_attn_error_string",
    "simplicial_attn_abi_version",
    "simplicial_attn_path_name",
    "DTYPE_F32",
    "DTYPE_BF16",
]

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libsimplicial_attn.so")
DTYPE_F32 = 0
DTYPE_BF16 = 1
_DTYPES = {torch.float32: DTYPE_F32, torch.bfloat16: DTYPE_BF16}

_lib = None


class SimplicialAttnError(RuntimeError):
    def __init__(self, code, where):
        self.code = code
        super().__init__(f"{where} failed with status {code}: {simplicial_attn_error_string(code)}")


def load_library():
    """Load (once) and return the ctypes handle; raise if the library is missing."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(
            f"{LIB_PATH} is not built; run `python -m paper_2507_02754_amd.build` "
            "(the HIP library is required; there is no CPU fallback)")
    lib = ctypes.CDLL(LIB_PATH)
    vp, i64, i32, f32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_float
    lib.simplicial_attn_fwd.argtypes = [vp] * 7 + [i64] * 4 + [i32, i32, f32, i32, vp]
    lib.simplicial_attn_fwd.restype = ctypes.c_int
    lib.simplicial_attn_fwd_gqa.argtypes = [vp] * 7 + [i64] * 5 + [i32, i32, f32, i32, vp]
    lib.simplicial_attn_fwd_gqa.restype = ctypes.c_int
    lib.simplicial_attn_bwd.argtypes = [vp] * 14 + [ctypes.c_size_t] + [i64] * 4 + [i32, i32, f32, i32, vp]
    lib.simplicial_attn_bwd.restype = ctypes.c_int
    lib.simplicial_attn_fwd_biased.argtypes = [vp] * 7 + [i64] * 4 + [i32, i32, f32, f32, f32, i32, vp]
    lib.simplicial_attn_fwd_biased.restype = ctypes.c_int
    lib.simplicial_attn_bwd_biased.argtypes = ([vp] * 14 + [ctypes.c_size_t] + [i64] * 4 +
                                               [i32, i32, f32, f32, f32, i32, vp])
    lib.simplicial_attn_bwd_biased.restype = ctypes.c_int
    lib.simplicial_attn_bwd_noalloc.argtypes = [vp] * 13 + [i64] * 4 + [i32, i32, f32, i32, vp]
    lib.simplicial_attn_bwd_noalloc.restype = ctypes.c_int
    lib.simplicial_attn_det_fwd.argtypes = lib.simplicial_attn_fwd.argtypes
    lib.simplicial_attn_det_fwd.restype = ctypes.c_int
    lib.simplicial_attn_det_bwd.argtypes = lib.simplicial_attn_bwd.argtypes
    lib.simplicial_attn_det_bwd.restype = ctypes.c_int
    lib.simplicial_attn_bwd_gqa.argtypes = [vp] * 14 + [ctypes.c_size_t] + [i64] * 5 + [i32, i32, f32, i32, vp]
    lib.simplicial_attn_bwd_gqa.restype = ctypes.c_int
    lib.simplicial_attn_det_bwd_workspace_size.argtypes = [i64] * 4 + [i32, i32, i32]
    lib.simplicial_attn_det_bwd_workspace_size.restype = ctypes.c_size_t
    lib.simplicial_attn_bwd_gqa_workspace_size.argtypes = [i64] * 5 + [i32, i32, i32]
    lib.simplicial_attn_bwd_gqa_workspace_size.restype = ctypes.c_size_t
    lib.simplicial_attn_bwd_preprocess.argtypes = [vp] * 3 + [ctypes.c_size_t] + [i64] * 4 + [i32, i32, i32, vp]
    lib.simplicial_attn_bwd_preprocess.restype = ctypes.c_int
    lib.simplicial_attn_bwd_query_side.argtypes = [vp] * 11 + [ctypes.c_size_t] + [i64] * 4 + [i32, i32, f32, i32, vp]
    lib.simplicial_attn_bwd_query_side.restype = ctypes.c_int
    lib.simplicial_attn_bwd_key_side.argtypes = [vp] * 10 + [ctypes.c_size_t] + [i64] * 4 + [i32, i32, f32, i32, vp]
    lib.simplicial_attn_bwd_key_side.restype = ctypes.c_int
    lib.simplicial_attn_bwd_fused.argtypes = [vp] * 10 + [ctypes.c_size_t] + [i64] * 4 + [i32, i32, f32, f32, f32, i32, vp]
    lib.simplicial_attn_bwd_fused.restype = ctypes.c_int
    lib.simplicial_attn_bwd_fused_reduce.argtypes = [vp] * 4 + [ctypes.c_size_t] + [i64] * 4 + [i32, i32, f32, i32, vp]
    lib.simplicial_attn_bwd_fused_reduce.restype = ctypes.c_int
    lib.simplicial_attn_bwd_fused_workspace_size.argtypes = [i64] * 4 + [i32, i32, i32]
    lib.simplicial_attn_bwd_fused_workspace_size.restype = ctypes.c_size_t
    lib.simplicial_attn_bwd_workspace_size.argtypes = [i64] * 4 + [i32, i32, i32]
    lib.simplicial_attn_bwd_workspace_size.restype = ctypes.c_size_t
    lib.simplicial_attn_error_string.argtypes = [ctypes.c_int]
    lib.simplicial_attn_error_string.restype = ctypes.c_char_p
    lib.simplicial_attn_abi_version.argtypes = []
    lib.simplicial_attn_abi_version.restype = ctypes.c_int
    lib.simplicial_attn_path_name.argtypes = [i32] + [i64] * 4 + [i32, i32, i32]
    lib.simplicial_attn_path_name.restype = ctypes.c_char_p
    _lib = lib
    return lib


def simplicial_attn_error_string(code):
    return load_library().simplicial_attn_error_string(int(code)).decode()


def simplicial_attn_abi_version():
    return int(load_library().simplicial_attn_abi_version())


def simplicial_attn_path_name(which, B, N, H, D, w1, w2, dtype):
    """Kernel path for forward (which=0) or backward (which=1); dtype is a torch dtype or int."""
    dt = _DTYPES.get(dtype, dtype)
    return load_library().simplicial_attn_path_name(int(which), B, N, H, D, int(w1), int(w2), int(dt)).decode()


def simplicial_attn_bwd_workspace_size(B, N, H, D, w1, w2, dtype):
    dt = _DTYPES.get(dtype, dtype)
    return int(load_library().simplicial_attn_bwd_workspace_size(B, N, H, D, int(w1), int(w2), int(dt)))


def simplicial_attn_det_bwd_workspace_size(B, N, H, D, w1, w2, dtype):
    dt = _DTYPES.get(dtype, dtype)
    return int(load_library().simplicial_attn_det_bwd_workspace_size(B, N, H, D, int(w1), int(w2), int(dt)))


def simplicial_attn_bwd_gqa_workspace_size(B, N, H, Hkv, D, w1, w2, dtype):
    dt = _DTYPES.get(dtype, dtype)
    return int(load_library().simplicial_attn_bwd_gqa_workspace_size(B, N, H, Hkv, D, int(w1), int(w2),
                                                                      int(dt)))


def _check_inputs(tensors, names):
    t0 = tensors[0]
    if t0.dim() != 4:
        raise ValueError(f"{names[0]} must be [B, N, H, D], got shape {tuple(t0.shape)}")
    if t0.dtype not in _DTYPES:
        raise ValueError(f"unsupported dtype {t0.dtype}; expected float32 or bfloat16")
    for t, n in zip(tensors, names):
        if not t.is_cuda:
            raise ValueError(f"{n} must be a GPU tensor")
        if t.device != t0.device:
            raise ValueError(f"{n} is on {t.device}, expected {t0.device}")
        if t.dtype != t0.dtype:
            raise ValueError(f"{n} has dtype {t.dtype}, expected {t0.dtype}")
        if t.shape != t0.shape:
            raise ValueError(f"{n} has shape {tuple(t.shape)}, expected {tuple(t0.shape)}")
        if not t.is_contiguous():
            raise ValueError(f"{n} must be contiguous [B, N, H, D]")
    return t0.shape, _DTYPES[t0.dtype]


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr())


def _stream(device):
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def simplicial_attn_fwd(q, k, kp, v, vp, w1, w2, scale=None, out=None, lse=None):
    """O, LSE = forward(Q, K, K', V, V'); tensors [B, N, H, D] on one GPU.

    `scale` defaults to 1/sqrt(D). Returns (out [B, N, H, D], lse [B, H, N] fp32).
    """
    return _fwd("simplicial_attn_fwd", q, k, kp, v, vp, w1, w2, scale, out, lse)


def simplicial_attn_det_fwd(q, k, kp, v, vp, w1, w2, scale=1.0, out=None, lse=None):
    """Forward with the determinant logits of Section 5 (arguments and results
    as simplicial_attn_fwd). `scale` defaults to 1: Eq. (logits) has no scale
    factor."""
    return _fwd("simplicial_attn_det_fwd", q, k, kp, v, vp, w1, w2, scale, out, lse)


def simplicial_attn_fwd_biased(q, k, kp, v, vp, w1, w2, scale=None, kp_bias=0.0, vp_bias=0.0,
                               out=None, lse=None):
    """Forward with the K' / V' bias constants (K' + kp_bias, V' + vp_bias in
    place of K', V'); otherwise as simplicial_attn_fwd."""
    return _fwd("simplicial_attn_fwd_biased", q, k, kp, v, vp, w1, w2, scale, out, lse,
                biases=(float(kp_bias), float(vp_bias)))


def _fwd(entry, q, k, kp, v, vp, w1, w2, scale, out, lse, biases=()):
    (B, N, H, D), dt = _check_inputs((q, k, kp, v, vp), ("q", "k", "kp", "v", "vp"))
    if scale is None:
        scale = D ** -0.5
    if out is None:
        out = torch.empty_like(q)
    else:
        _check_inputs((q, out), ("q", "out"))
    if lse is None:
        lse = torch.empty((B, H, N), dtype=torch.float32, device=q.device)
    elif lse.shape != (B, H, N) or lse.dtype != torch.float32 or not lse.is_contiguous() \
            or lse.device != q.device:
        raise ValueError("lse must be a contiguous float32 [B, H, N] tensor on the inputs' device")
    rc = getattr(load_library(), entry)(
        _ptr(q), _ptr(k), _ptr(kp), _ptr(v), _ptr(vp), _ptr(out), _ptr(lse),
        B, N, H, D, int(w1), int(w2), float(scale), *biases, dt, _stream(q.device))
    if rc != 0:
        raise SimplicialAttnError(rc, entry)
    return out, lse


def simplicial_attn_fwd_gqa(q, k, kp, v, vp, w1, w2, scale=None, out=None, lse=None):
    """O, LSE = forward with grouped-query attention: q [B, N, H, D] and
    k, kp, v, vp [B, N, Hkv, D] (H a multiple of Hkv; query head h reads head
    h // (H // Hkv)). `scale` defaults to 1/sqrt(D). Returns (out [B, N, H, D],
    lse [B, H, N] fp32)."""
    (B, N, Hkv, D), dt = _check_inputs((k, kp, v, vp), ("k", "kp", "v", "vp"))
    _check_inputs((q,), ("q",))
    if q.dim() != 4 or q.shape[0] != B or q.shape[1] != N or q.shape[3] != D or q.dtype != k.dtype \
            or q.device != k.device:
        raise ValueError(f"q must be [B, N, H, D] = [{B}, {N}, H, {D}] with the dtype and device of k, "
                         f"got {tuple(q.shape)} {q.dtype} {q.device}")
    H = q.shape[2]
    if scale is None:
        scale = D ** -0.5
    if out is None:
        out = torch.empty_like(q)
    else:
        _check_inputs((q, out), ("q", "out"))
    if lse is None:
        lse = torch.empty((B, H, N), dtype=torch.float32, device=q.device)
    elif lse.shape != (B, H, N) or lse.dtype != torch.float32 or not lse.is_contiguous() \
            or lse.device != q.device:
        raise ValueError("lse must be a contiguous float32 [B, H, N] tensor on the inputs' device")
    rc = load_library().simplicial_attn_fwd_gqa(
        _ptr(q), _ptr(k), _ptr(kp), _ptr(v), _ptr(vp), _ptr(out), _ptr(lse),
        B, N, H, Hkv, D, int(w1), int(w2), float(scale), dt, _stream(q.device))
    if rc != 0:
        raise SimplicialAttnError(rc, "simplicial_attn_fwd_gqa")
    return out, lse


def _bwd_common(q, k, kp, v, vp, dout, lse, w1, w2, extra=(), extra_names=()):
    (B, N, H, D), dt = _check_inputs((q, k, kp, v, vp, dout, *extra),
                                     ("q", "k", "kp", "v", "vp", "dout", *extra_names))
    if lse.shape != (B, H, N) or lse.dtype != torch.float32 or not lse.is_contiguous() \
            or lse.device != q.device:
        raise ValueError("lse must be a contiguous float32 [B, H, N] tensor on the inputs' device")
    return (B, N, H, D), dt


def _workspace(workspace, B, N, H, D, w1, w2, dt, device):
    ws = simplicial_attn_bwd_workspace_size(B, N, H, D, w1, w2, dt)
    if workspace is None:
        workspace = torch.empty(max(ws, 16), dtype=torch.uint8, device=device)
    return workspace


def simplicial_attn_bwd_preprocess(out, dout, w1, w2, workspace):
    """Delta_i = <dO_i, O_i> into `workspace` (a uint8 GPU tensor of the backward's size)."""
    (B, N, H, D), dt = _check_inputs((out, dout), ("out", "dout"))
    rc = load_library().simplicial_attn_bwd_preprocess(
        _ptr(out), _ptr(dout), _ptr(workspace), ctypes.c_size_t(workspace.numel()),
        B, N, H, D, int(w1), int(w2), dt, _stream(out.device))
    if rc != 0:
        raise SimplicialAttnError(rc, "simplicial_attn_bwd_preprocess")
    return workspace


def simplicial_attn_bwd_query_side(q, k, kp, v, vp, dout, lse, w1, w2, workspace, scale=None,
                                   grads=None):
    """(dQ, dK', dV') after simplicial_attn_bwd_preprocess filled `workspace`."""
    (B, N, H, D), dt = _bwd_common(q, k, kp, v, vp, dout, lse, w1, w2)
    scale = D ** -0.5 if scale is None else scale
    grads = grads if grads is not None else tuple(torch.empty_like(q) for _ in range(3))
    _check_inputs((q, *grads), ("q", "dq", "dkp", "dvp"))
    rc = load_library().simplicial_attn_bwd_query_side(
        _ptr(q), _ptr(k), _ptr(kp), _ptr(v), _ptr(vp), _ptr(dout), _ptr(lse),
        *(_ptr(g) for g in grads), _ptr(workspace), ctypes.c_size_t(workspace.numel()),
        B, N, H, D, int(w1), int(w2), float(scale), dt, _stream(q.device))
    if rc != 0:
        raise SimplicialAttnError(rc, "simplicial_attn_bwd_query_side")
    return grads


def simplicial_attn_bwd_key_side(q, k, kp, v, vp, dout, lse, w1, w2, workspace, scale=None,
                                 grads=None):
    """(dK, dV) after simplicial_attn_bwd_preprocess filled `workspace`."""
    (B, N, H, D), dt = _bwd_common(q, k, kp, v, vp, dout, lse, w1, w2)
    scale = D ** -0.5 if scale is None else scale
    grads = grads if grads is not None else tuple(torch.empty_like(q) for _ in range(2))
    _check_inputs((q, *grads), ("q", "dk", "dv"))
    rc = load_library().simplicial_attn_bwd_key_side(
        _ptr(q), _ptr(k), _ptr(kp), _ptr(v), _ptr(vp), _ptr(dout), _ptr(lse),
        *(_ptr(g) for g in grads), _ptr(workspace), ctypes.c_size_t(workspace.numel()),
        B, N, H, D, int(w1), int(w2), float(scale), dt, _stream(q.device))
    if rc != 0:
        raise SimplicialAttnError(rc, "simplicial_attn_bwd_key_side")
    return grads


def simplicial_attn_bwd_fused_workspace_size(B, N, H, D, w1, w2, dtype):
    """Bytes of the fused backward's workspace (0: shape not supported by it)."""
    dt = _DTYPES.get(dtype, dtype)
    return int(load_library().simplicial_attn_bwd_fused_workspace_size(B, N, H, D, int(w1), int(w2), int(dt)))


def simplicial_attn_bwd_fused(q, k, kp, v, vp, dout, lse, w1, w2, workspace, scale=None, grads=None,
                              kp_bias=0.0, vp_bias=0.0):
    """(dK, dV) of the fused kernel after simplicial_attn_bwd_preprocess filled
    `workspace` (of simplicial_attn_bwd_fused_workspace_size bytes); the
    kernel also leaves the partial sums of dQ, dK', dV' there."""
    (B, N, H, D), dt = _bwd_common(q, k, kp, v, vp, dout, lse, w1, w2)
    scale = D ** -0.5 if scale is None else scale
    grads = grads if grads is not None else tuple(torch.empty_like(q) for _ in range(2))
    _check_inputs((q, *grads), ("q", "dk", "dv"))
    rc = load_library().simplicial_attn_bwd_fused(
        _ptr(q), _ptr(k), _ptr(kp), _ptr(v), _ptr(vp), _ptr(dout), _ptr(lse),
        *(_ptr(g) for g in grads), _ptr(workspace), ctypes.c_size_t(workspace.numel()),
        B, N, H, D, int(w1), int(w2), float(scale), float(kp_bias), float(vp_bias), dt, _stream(q.device))
    if rc != 0:
        raise SimplicialAttnError(rc, "simplicial_attn_bwd_fused")
    return grads


def simplicial_attn_bwd_fused_reduce(q, w1, w2, workspace, scale=None, grads=None):
    """(dQ, dK', dV') from the partial sums simplicial_attn_bwd_fused left in
    `workspace` (q gives sizes, dtype and device)."""
    (B, N, H, D), dt = _check_inputs((q,), ("q",))
    scale = D ** -0.5 if scale is None else scale
    grads = grads if grads is not None else tuple(torch.empty_like(q) for _ in range(3))
    _check_inputs((q, *grads), ("q", "dq", "dkp", "dvp"))
    rc = load_library().simplicial_attn_bwd_fused_reduce(
        *(_ptr(g) for g in grads), _ptr(workspace), ctypes.c_size_t(workspace.numel()),
        B, N, H, D, int(w1), int(w2), float(scale), dt, _stream(q.device))
    if rc != 0:
        raise SimplicialAttnError(rc, "simplicial_attn_bwd_fused_reduce")
    return grads


def simplicial_attn_bwd(q, k, kp, v, vp, out, dout, lse, w1, w2, scale=None, grads=None,
                        workspace=None):
    """(dQ, dK, dK', dV, dV') = backward(...); `out`/`lse` come from the forward."""
    return _bwd("simplicial_attn_bwd", q, k, kp, v, vp, out, dout, lse, w1, w2, scale, grads,
                workspace)


def simplicial_attn_bwd_noalloc(q, k, kp, v, vp, out, dout, lse, w1, w2, scale=None, grads=None):
    """(dQ, dK, dK', dV, dV') through the allocation-free entry point, whose
    workspace is the library's fixed device scratch array. Pass preallocated
    `grads` to keep the whole call free of allocations (otherwise torch
    allocates them here, before the entry point is called)."""
    (B, N, H, D), dt = _check_inputs((q, k, kp, v, vp, out, dout),
                                     ("q", "k", "kp", "v", "vp", "out", "dout"))
    if scale is None:
        scale = D ** -0.5
    if lse.shape != (B, H, N) or lse.dtype != torch.float32 or not lse.is_contiguous() \
            or lse.device != q.device:
        raise ValueError("lse must be a contiguous float32 [B, H, N] tensor on the inputs' device")
    if grads is None:
        grads = tuple(torch.empty_like(q) for _ in range(5))
    else:
        _check_inputs((q, *grads), ("q", "dq", "dk", "dkp", "dv", "dvp"))
    rc = load_library().simplicial_attn_bwd_noalloc(
        _ptr(q), _ptr(k), _ptr(kp), _ptr(v), _ptr(vp), _ptr(out), _ptr(dout), _ptr(lse),
        *(_ptr(g) for g in grads), B, N, H, D, int(w1), int(w2), float(scale), dt,
        _stream(q.device))
    if rc != 0:
        raise SimplicialAttnError(rc, "simplicial_attn_bwd_noalloc")
    return grads


def simplicial_attn_det_bwd(q, k, kp, v, vp, out, dout, lse, w1, w2, scale=1.0, grads=None,
                            workspace=None):
    """Backward with the determinant logits of Section 5 (arguments and results
    as simplicial_attn_bwd; `out`/`lse` from simplicial_attn_det_fwd; `scale`
    defaults to 1 as in the forward)."""
    if workspace is None:
        B, N, H, D = q.shape
        need = simplicial_attn_det_bwd_workspace_size(B, N, H, D, w1, w2, q.dtype)
        workspace = torch.empty(max(need, 16), dtype=torch.uint8, device=q.device)
    return _bwd("simplicial_attn_det_bwd", q, k, kp, v, vp, out, dout, lse, w1, w2, scale, grads,
                workspace)


def simplicial_attn_bwd_biased(q, k, kp, v, vp, out, dout, lse, w1, w2, scale=None, kp_bias=0.0,
                               vp_bias=0.0, grads=None, workspace=None):
    """Backward of simplicial_attn_fwd_biased (same constants); gradients are
    with respect to the given K' and V'."""
    return _bwd("simplicial_attn_bwd_biased", q, k, kp, v, vp, out, dout, lse, w1, w2, scale, grads,
                workspace, biases=(float(kp_bias), float(vp_bias)))


def _bwd(entry, q, k, kp, v, vp, out, dout, lse, w1, w2, scale, grads, workspace, biases=()):
    (B, N, H, D), dt = _check_inputs((q, k, kp, v, vp, out, dout),
                                     ("q", "k", "kp", "v", "vp", "out", "dout"))
    if scale is None:
        scale = D ** -0.5
    if lse.shape != (B, H, N) or lse.dtype != torch.float32 or not lse.is_contiguous() \
            or lse.device != q.device:
        raise ValueError("lse must be a contiguous float32 [B, H, N] tensor on the inputs' device")
    if grads is None:
        grads = tuple(torch.empty_like(q) for _ in range(5))
    else:
        _check_inputs((q, *grads), ("q", "dq", "dk", "dkp", "dv", "dvp"))
    workspace = _workspace(workspace, B, N, H, D, w1, w2, dt, q.device)
    rc = getattr(load_library(), entry)(
        _ptr(q), _ptr(k), _ptr(kp), _ptr(v), _ptr(vp), _ptr(out), _ptr(dout), _ptr(lse),
        *(_ptr(g) for g in grads), _ptr(workspace), ctypes.c_size_t(workspace.numel()),
        B, N, H, D, int(w1), int(w2), float(scale), *biases, dt, _stream(q.device))
    if rc != 0:
        raise SimplicialAttnError(rc, entry)
    return grads


def simplicial_attn_bwd_gqa(q, k, kp, v, vp, out, dout, lse, w1, w2, scale=None, grads=None,
                            workspace=None):
    """(dQ, dK, dK', dV, dV') for simplicial_attn_fwd_gqa: q, out, dout, dQ are
    [B, N, H, D]; k, kp, v, vp and their gradients [B, N, Hkv, D]."""
    (B, N, H, D), dt = _check_inputs((q, out, dout), ("q", "out", "dout"))
    (Bk, Nk, Hkv, Dk), dtk = _check_inputs((k, kp, v, vp), ("k", "kp", "v", "vp"))
    if (Bk, Nk, Dk) != (B, N, D) or dtk != dt or k.device != q.device:
        raise ValueError(f"k, kp, v, vp must be [B, N, Hkv, D] = [{B}, {N}, Hkv, {D}] with the dtype "
                         f"and device of q, got {tuple(k.shape)} {k.dtype} {k.device}")
    if scale is None:
        scale = D ** -0.5
    if lse.shape != (B, H, N) or lse.dtype != torch.float32 or not lse.is_contiguous() \
            or lse.device != q.device:
        raise ValueError("lse must be a contiguous float32 [B, H, N] tensor on the inputs' device")
    if grads is None:
        grads = (torch.empty_like(q), *(torch.empty_like(k) for _ in range(4)))
    else:
        _check_inputs((q, grads[0]), ("q", "dq"))
        _check_inputs((k, *grads[1:]), ("k", "dk", "dkp", "dv", "dvp"))
    need = simplicial_attn_bwd_gqa_workspace_size(B, N, H, Hkv, D, w1, w2, dt)
    if workspace is None:
        workspace = torch.empty(max(need, 16), dtype=torch.uint8, device=q.device)
    rc = load_library().simplicial_attn_bwd_gqa(
        _ptr(q), _ptr(k), _ptr(kp), _ptr(v), _ptr(vp), _ptr(out), _ptr(dout), _ptr(lse),
        *(_ptr(g) for g in grads), _ptr(workspace), ctypes.c_size_t(workspace.numel()),
        B, N, H, Hkv, D, int(w1), int(w2), float(scale), dt, _stream(q.device))
    if rc != 0:
        raise SimplicialAttnError(rc, "simplicial_attn_bwd_gqa")
    return grads
