"""The C-ABI library: it builds, loads, exports every declared symbol, and rejects
invalid arguments on the host before any HIP call (so these run without a GPU).
"""

import ctypes
import os
import re
import subprocess

import pytest

from paper_2507_02754_amd import binding

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "simplicial_attn.h")

# Fake device addresses for calls that must be rejected before any launch. They
# are only used where the validation must fail; on a machine with a GPU these
# tests are skipped so a validation bug can never launch on them.
A = 0x10000  # 16-byte aligned
MISALIGNED = 0x10008


def _no_gpu():
    import torch
    return torch.cuda.device_count() == 0


only_without_gpu = pytest.mark.skipif(not _no_gpu(), reason="fake-pointer checks run only where no GPU is visible")


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(binding.LIB_PATH):
        from paper_2507_02754_amd import build
        build.build()
    return binding.load_library()


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(simplicial_attn_\w+)\s*\(", src)))


def test_header_declares_the_expected_entry_points():
    assert declared_functions() == sorted([
        "simplicial_attn_fwd", "simplicial_attn_fwd_gqa", "simplicial_attn_bwd",
        "simplicial_attn_bwd_workspace_size", "simplicial_attn_bwd_gqa",
        "simplicial_attn_bwd_gqa_workspace_size", "simplicial_attn_det_fwd", "simplicial_attn_det_bwd",
        "simplicial_attn_error_string", "simplicial_attn_abi_version", "simplicial_attn_path_name",
        "simplicial_attn_bwd_preprocess", "simplicial_attn_bwd_query_side",
        "simplicial_attn_bwd_key_side", "simplicial_attn_bwd_noalloc",
        "simplicial_attn_fwd_biased", "simplicial_attn_bwd_biased",
        "simplicial_attn_det_bwd_workspace_size", "simplicial_attn_bwd_fused",
        "simplicial_attn_bwd_fused_reduce", "simplicial_attn_bwd_fused_workspace_size",
    ])


def test_library_exports_every_declared_symbol(lib):
    out = subprocess.run(["nm", "-D", "--defined-only", binding.LIB_PATH],
                         capture_output=True, text=True, check=True).stdout
    exported = set(re.findall(r"\bT (simplicial_attn_\w+)", out))
    for name in declared_functions():
        assert name in exported, name
        assert hasattr(lib, name)


def test_abi_version_matches_header(lib):
    m = re.search(r"#define SIMPLICIAL_ATTN_ABI_VERSION (\d+)", open(HEADER).read())
    assert binding.simplicial_attn_abi_version() == int(m.group(1))


def test_error_strings(lib):
    for code in range(6):
        s = binding.simplicial_attn_error_string(code)
        assert s and s != "unknown status"
    assert binding.simplicial_attn_error_string(99) == "unknown status"


def _fwd(lib, ptrs=None, B=1, N=64, H=2, D=128, w1=16, w2=8, scale=0.1, dtype=1):
    ptrs = ptrs or [A] * 7
    return lib.simplicial_attn_fwd(*[ctypes.c_void_p(p) for p in ptrs], B, N, H, D, w1, w2,
                                   ctypes.c_float(scale), dtype, None)


def _bwd(lib, ptrs=None, ws_bytes=1 << 30, B=1, N=64, H=2, D=128, w1=16, w2=8, scale=0.1, dtype=1):
    ptrs = ptrs or [A] * 14
    return lib.simplicial_attn_bwd(*[ctypes.c_void_p(p) for p in ptrs], ctypes.c_size_t(ws_bytes),
                                   B, N, H, D, w1, w2, ctypes.c_float(scale), dtype, None)


@only_without_gpu
def test_forward_rejects_invalid_arguments(lib):
    for i in range(7):
        ptrs = [A] * 7
        ptrs[i] = 0
        assert _fwd(lib, ptrs) == 1, f"null pointer {i}"
        ptrs[i] = MISALIGNED
        assert _fwd(lib, ptrs) == 1, f"misaligned pointer {i}"
    assert _fwd(lib, B=0) == 1
    assert _fwd(lib, N=0) == 1
    assert _fwd(lib, H=-1) == 1
    assert _fwd(lib, D=0) == 1
    assert _fwd(lib, w1=0) == 1
    assert _fwd(lib, w2=-3) == 1
    assert _fwd(lib, scale=float("nan")) == 1
    assert _fwd(lib, scale=float("inf")) == 1
    assert _fwd(lib, N=1 << 31) == 1          # does not fit a 32-bit index
    assert _fwd(lib, B=1 << 20, N=1 << 20, H=1 << 10) == 1  # overflow
    assert _fwd(lib, D=48) == 2
    assert _fwd(lib, D=256) == 2
    assert _fwd(lib, dtype=2) == 2
    assert _fwd(lib, dtype=-1) == 2


def _fwd_gqa(lib, ptrs=None, B=1, N=64, H=4, Hkv=2, D=128, w1=16, w2=8, scale=0.1, dtype=1):
    ptrs = ptrs or [A] * 7
    return lib.simplicial_attn_fwd_gqa(*[ctypes.c_void_p(p) for p in ptrs], B, N, H, Hkv, D, w1, w2,
                                       ctypes.c_float(scale), dtype, None)


@only_without_gpu
def test_gqa_forward_rejects_invalid_arguments(lib):
    for i in range(7):
        ptrs = [A] * 7
        ptrs[i] = 0
        assert _fwd_gqa(lib, ptrs) == 1, f"null pointer {i}"
        ptrs[i] = MISALIGNED
        assert _fwd_gqa(lib, ptrs) == 1, f"misaligned pointer {i}"
    assert _fwd_gqa(lib, Hkv=0) == 1
    assert _fwd_gqa(lib, Hkv=-2) == 1
    assert _fwd_gqa(lib, H=4, Hkv=8) == 1   # more K-side heads than query heads
    assert _fwd_gqa(lib, H=6, Hkv=4) == 1   # not a multiple
    assert _fwd_gqa(lib, w1=0) == 1
    assert _fwd_gqa(lib, scale=float("nan")) == 1
    assert _fwd_gqa(lib, D=48) == 2
    assert _fwd_gqa(lib, dtype=5) == 2


def _bwd_gqa(lib, ptrs=None, ws_bytes=1 << 40, B=1, N=64, H=4, Hkv=2, D=128, w1=16, w2=8, scale=0.1,
             dtype=1):
    ptrs = ptrs or [A] * 14
    return lib.simplicial_attn_bwd_gqa(*[ctypes.c_void_p(p) for p in ptrs], ctypes.c_size_t(ws_bytes),
                                       B, N, H, Hkv, D, w1, w2, ctypes.c_float(scale), dtype, None)


@only_without_gpu
def test_gqa_backward_rejects_invalid_arguments(lib):
    for i in range(14):
        ptrs = [A] * 14
        ptrs[i] = 0
        assert _bwd_gqa(lib, ptrs) == 1, f"null pointer {i}"
        ptrs[i] = MISALIGNED
        assert _bwd_gqa(lib, ptrs) == 1, f"misaligned pointer {i}"
    assert _bwd_gqa(lib, Hkv=0) == 1
    assert _bwd_gqa(lib, H=4, Hkv=8) == 1
    assert _bwd_gqa(lib, H=6, Hkv=4) == 1
    assert _bwd_gqa(lib, w2=0) == 1
    assert _bwd_gqa(lib, scale=float("inf")) == 1
    assert _bwd_gqa(lib, D=40) == 2
    need = binding.simplicial_attn_bwd_gqa_workspace_size(1, 64, 4, 2, 128, 16, 8, 1)
    assert _bwd_gqa(lib, ws_bytes=need - 1) == 3
    assert _bwd_gqa(lib, ws_bytes=0) == 3


def test_gqa_workspace_size(lib):
    f = binding.simplicial_attn_bwd_gqa_workspace_size
    plain = binding.simplicial_attn_bwd_workspace_size
    assert f(1, 64, 4, 3, 128, 16, 8, 1) == 0      # Hkv does not divide H
    assert f(1, 64, 4, 0, 128, 16, 8, 1) == 0
    assert f(1, 64, 4, 2, 48, 16, 8, 1) == 0
    # Hkv == H: the plain backward's workspace
    assert f(2, 8192, 8, 8, 128, 512, 32, 1) == plain(2, 8192, 8, 128, 512, 32, 1)
    # Hkv < H: plus [B, N, H, D] tensors of the data type, two where the MFMA
    # kernels read the K side in place (bf16, D 64/128, w2 <= 64), else eight
    for (b, n, h, hkv, d, w1, w2, dt, es, nt) in [(1, 64, 4, 2, 128, 16, 8, 1, 2, 2),
                                                  (1, 64, 4, 2, 64, 16, 64, 1, 2, 2),
                                                  (1, 200, 4, 2, 128, 16, 65, 1, 2, 8),
                                                  (1, 64, 4, 2, 128, 16, 8, 0, 4, 8),
                                                  (2, 100, 6, 1, 32, 9, 5, 0, 4, 8)]:
        ws = f(b, n, h, hkv, d, w1, w2, dt)
        assert ws >= plain(b, n, h, d, w1, w2, dt) + nt * b * n * h * d * es
        assert ws <= plain(b, n, h, d, w1, w2, dt) + nt * (b * n * h * d * es + 255) + 255


@only_without_gpu
def test_determinant_entry_points_reject_invalid_arguments(lib):
    fd = lambda ptrs=None, B=1, N=64, H=2, D=128, w1=16, w2=8, scale=0.1, dtype=1: \
        lib.simplicial_attn_det_fwd(*[ctypes.c_void_p(p) for p in (ptrs or [A] * 7)], B, N, H, D, w1,
                                    w2, ctypes.c_float(scale), dtype, None)
    bd = lambda ptrs=None, ws=1 << 30, D=128, w1=16: lib.simplicial_attn_det_bwd(
        *[ctypes.c_void_p(p) for p in (ptrs or [A] * 14)], ctypes.c_size_t(ws), 1, 64, 2, D, w1, 8,
        ctypes.c_float(0.1), 1, None)
    for i in range(7):
        ptrs = [A] * 7
        ptrs[i] = 0
        assert fd(ptrs) == 1
    for i in range(14):
        ptrs = [A] * 14
        ptrs[i] = MISALIGNED
        assert bd(ptrs) == 1
    assert fd(w1=0) == 1 and fd(scale=float("nan")) == 1 and fd(D=48) == 2 and fd(dtype=3) == 2
    assert bd(w1=0) == 1 and bd(D=40) == 2 and bd(ws=0) == 3


@only_without_gpu
def test_backward_rejects_invalid_arguments(lib):
    for i in range(14):
        ptrs = [A] * 14
        ptrs[i] = 0
        assert _bwd(lib, ptrs) == 1, f"null pointer {i}"
        ptrs[i] = MISALIGNED
        assert _bwd(lib, ptrs) == 1, f"misaligned pointer {i}"
    assert _bwd(lib, w1=0) == 1
    assert _bwd(lib, D=40) == 2
    need = binding.simplicial_attn_bwd_workspace_size(1, 64, 2, 128, 16, 8, 1)
    assert need > 0
    assert _bwd(lib, ws_bytes=need - 1) == 3
    assert _bwd(lib, ws_bytes=0) == 3


@only_without_gpu
def test_backward_stages_reject_invalid_arguments(lib):
    size = ctypes.c_size_t
    args = [1, 64, 2, 128, 16, 8]
    pre = lambda ptrs, ws=1 << 30, dtype=1, a=args: lib.simplicial_attn_bwd_preprocess(
        *[ctypes.c_void_p(p) for p in ptrs], size(ws), *a, dtype, None)
    assert pre([0, A, A]) == 1
    assert pre([A, MISALIGNED, A]) == 1
    assert pre([A, A, A], ws=0) == 3
    assert pre([A, A, A], dtype=3) == 2
    assert pre([A, A, A], a=[1, 64, 2, 128, 0, 8]) == 1
    for fn, n in ((lib.simplicial_attn_bwd_query_side, 11), (lib.simplicial_attn_bwd_key_side, 10)):
        call = lambda ptrs, ws=1 << 30, scale=0.1, a=args, dtype=1: fn(
            *[ctypes.c_void_p(p) for p in ptrs], size(ws), *a, ctypes.c_float(scale), dtype, None)
        for i in range(n):
            ptrs = [A] * n
            ptrs[i] = 0
            assert call(ptrs) == 1
            ptrs[i] = MISALIGNED
            assert call(ptrs) == 1
        assert call([A] * n, ws=16) == 3
        assert call([A] * n, scale=float("nan")) == 1
        assert call([A] * n, a=[1, 64, 2, 96, 16, 8]) == 2


def test_workspace_size(lib):
    f = binding.simplicial_attn_bwd_workspace_size
    assert f(0, 64, 2, 128, 16, 8, 1) == 0
    assert f(1, 64, 2, 128, 16, 8, 7) == 0
    assert f(1, 64, 2, 128, 0, 8, 1) == 0
    # at least one float of Delta per (b, h, query), 256-byte granular
    for shape in [(1, 64, 2, 128, 16, 8, 1), (2, 8192, 8, 128, 512, 32, 1), (1, 128, 1, 64, 16, 8, 0)]:
        ws = f(*shape)
        b, n, h = shape[0], shape[1], shape[2]
        assert ws >= 4 * b * h * n and ws % 256 == 0


def test_path_names(lib):
    f = binding.simplicial_attn_path_name
    assert f(0, 1, 128, 1, 64, 16, 8, 0) == "generic"
    assert f(1, 1, 128, 1, 64, 16, 8, 0) == "generic"
    assert f(0, 1, 128, 1, 48, 16, 8, 0) == "invalid"
    assert f(2, 1, 128, 1, 64, 16, 8, 0) == "invalid"
    for which in (0, 1):
        assert f(which, 1, 32768, 16, 128, 512, 32, 1) == "mfma_bf16"
    assert f(1, 1, 4096, 8, 128, 512, 32, 0) == "generic"


def test_fused_workspace_holds_the_partial_sums(lib):
    """The fused backward's workspace: Delta, then per workgroup of 64 keys the
    dq partials of 63 + w1 queries and the dk', dv' partials of 94 + w1
    k-rows (fp32, D each); at least the split backward's workspace (the
    preprocess stage checks that size). 0 for shapes it does not take."""
    f = binding.simplicial_attn_bwd_fused_workspace_size
    for B, N, H, w1, w2 in [(1, 32768, 16, 512, 32), (2, 8192, 8, 512, 32), (1, 100, 2, 7, 5), (1, 1, 1, 1, 1)]:
        njb = -(-N // 64)
        need = 4 * (B * H * N + B * H * njb * ((63 + w1) + 2 * (94 + w1)) * 128)
        ws = f(B, N, H, 128, w1, w2, 1)
        assert ws >= need and ws >= binding.simplicial_attn_bwd_workspace_size(B, N, H, 128, w1, w2, 1)
    assert f(1, 4096, 8, 128, 512, 64, 1) == 0  # w2 > 32
    assert f(1, 4096, 8, 64, 512, 32, 1) == 0   # head_dim 64
    assert f(1, 4096, 8, 128, 512, 32, 0) == 0  # fp32
    assert f(0, 4096, 8, 128, 512, 32, 1) == 0  # invalid


@only_without_gpu
def test_fused_stages_reject_invalid_arguments(lib):
    size = ctypes.c_size_t
    args = [1, 64, 2, 128, 16, 8]
    fused = lambda ptrs, ws=1 << 30, scale=0.1, a=args, dtype=1, kb=0.0: lib.simplicial_attn_bwd_fused(
        *[ctypes.c_void_p(p) for p in ptrs], size(ws), *a, ctypes.c_float(scale), ctypes.c_float(kb),
        ctypes.c_float(0.0), dtype, None)
    red = lambda ptrs, ws=1 << 30, scale=0.1, a=args, dtype=1: lib.simplicial_attn_bwd_fused_reduce(
        *[ctypes.c_void_p(p) for p in ptrs], size(ws), *a, ctypes.c_float(scale), dtype, None)
    for call, n in ((fused, 10), (red, 4)):
        for i in range(n):
            ptrs = [A] * n
            ptrs[i] = 0
            assert call(ptrs) == 1
            ptrs[i] = MISALIGNED
            assert call(ptrs) == 1
        assert call([A] * n, ws=16) == 3
        assert call([A] * n, scale=float("nan")) == 1
        assert call([A] * n, a=[1, 64, 2, 64, 16, 8]) == 2   # head_dim 64: split path only
        assert call([A] * n, a=[1, 64, 2, 128, 16, 40]) == 2  # w2 > 32
        assert call([A] * n, dtype=0) == 2                     # fp32
    assert fused([A] * 10, kb=float("inf")) == 1


@only_without_gpu
def test_biased_entry_points_reject_invalid_arguments(lib):
    f32 = ctypes.c_float

    def fwd(kb=0.5, vb=0.5, ptrs=None, D=128):
        ptrs = ptrs or [A] * 7
        return lib.simplicial_attn_fwd_biased(*[ctypes.c_void_p(p) for p in ptrs], 1, 64, 2, D, 16, 8,
                                              f32(0.1), f32(kb), f32(vb), 1, None)

    def bwd(kb=0.5, vb=0.5, ws=1 << 30, ptrs=None):
        ptrs = ptrs or [A] * 14
        return lib.simplicial_attn_bwd_biased(*[ctypes.c_void_p(p) for p in ptrs], ctypes.c_size_t(ws),
                                              1, 64, 2, 128, 16, 8, f32(0.1), f32(kb), f32(vb), 1, None)

    for kb, vb in [(float("nan"), 0.0), (0.0, float("inf")), (float("-inf"), 1.0)]:
        assert fwd(kb, vb) == 1
        assert bwd(kb, vb) == 1
    ptrs = [A] * 7
    ptrs[3] = 0
    assert fwd(ptrs=ptrs) == 1
    assert fwd(D=48) == 2
    assert bwd(ws=16) == 3
