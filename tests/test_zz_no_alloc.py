"""The allocation-free backward (simplicial_attn_bwd_noalloc, workspace in the
library's fixed device scratch array) against the workspace backward
(simplicial_attn_bwd) through the C ABI."""

import ctypes

import pytest
import torch

import parity as P
from paper_2507_02754_amd import (load_library, simplicial_attn_bwd, simplicial_attn_bwd_noalloc,
                                  simplicial_attn_bwd_workspace_size, simplicial_attn_fwd)
from paper_2507_02754_amd.workloads import WORKLOADS, draw, make_inputs

SCRATCH = 64 << 20
SA_ERR_SCRATCH = 5


@pytest.mark.skipif(torch.cuda.device_count() > 0,
                    reason="fake-pointer checks run only where no GPU is visible")
def test_noalloc_rejects_sizes_beyond_the_scratch_before_any_hip_call():
    """Host-only: a problem whose Delta alone exceeds the 64 MiB array is
    rejected with SA_ERR_SCRATCH (fake device pointers are never touched)."""
    lib = load_library()
    fake = ctypes.c_void_p(1 << 20)
    B, N, H, D = 1, 1 << 20, 64, 128  # Delta: 256 MiB
    rc = lib.simplicial_attn_bwd_noalloc(*([fake] * 13), B, N, H, D, 512, 32, 0.088, 1, None)
    assert rc == SA_ERR_SCRATCH
    assert "scratch" in lib.simplicial_attn_error_string(rc).decode()
    # generic path (fp32): same limit
    rc = lib.simplicial_attn_bwd_noalloc(*([fake] * 13), B, N, H, 64, 16, 8, 0.125, 0, None)
    assert rc == SA_ERR_SCRATCH
    # arguments are still validated first
    rc = lib.simplicial_attn_bwd_noalloc(*([fake] * 12), None, 1, 16, 1, 128, 16, 8, 0.1, 1, None)
    assert rc == 1


def _inputs(case):
    if isinstance(case, str):
        w = WORKLOADS[case]
        return make_inputs(w), w.w1, w.w2, w.scale
    b, h, n, d, w1, w2, dt = case
    tdt = torch.bfloat16 if dt == "bf16" else torch.float32
    return draw((b, n, h, d), seed=40 + n, dtype=tdt), w1, w2, d ** -0.5


@pytest.mark.gpu
def test_noalloc_matches_workspace_backward():
    """Calls in a row on one GPU, larger first: the benchmark shape (its
    workspace exceeds the array, so the query side walks longer chunks), then
    sizes whose workspace fits (bitwise equal to simplicial_attn_bwd), the
    w2 = 64 path and the plain fp32 path. Each call is checked against the
    workspace backward on the same inputs at the parity bar."""
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    cases = ["long_bf16_n32k", (2, 8, 8192, 128, 512, 32, "bf16"), (1, 2, 700, 128, 256, 32, "bf16"),
             (1, 1, 300, 64, 40, 64, "bf16"), (1, 2, 100, 64, 7, 5, "fp32")]
    for case in cases:
        inputs, w1, w2, scale = _inputs(case)
        b, n, h, d = inputs[0].shape
        dt = inputs[0].dtype
        need = simplicial_attn_bwd_workspace_size(b, n, h, d, w1, w2, dt)
        print(f"\n[noalloc] {case} workspace {need} bytes ({'fits' if need <= SCRATCH else 'capped'})",
              flush=True)
        x = [t.cuda() for t in inputs]
        o, lse = simplicial_attn_fwd(*x[:5], w1, w2, scale)
        ref = simplicial_attn_bwd(*x[:5], o, x[5], lse, w1, w2, scale)
        grads = tuple(torch.full_like(x[0], float("nan")) for _ in range(5))
        got = simplicial_attn_bwd_noalloc(*x[:5], o, x[5], lse, w1, w2, scale, grads=grads)
        torch.cuda.synchronize()
        if need <= SCRATCH:
            for name, a, c in zip(P.GRAD_NAMES, got, ref):
                assert torch.equal(a, c), f"{case}: {name} differs from simplicial_attn_bwd"
        idx = torch.arange(0, n, max(1, n // 4096), device=x[0].device)
        P.check_grads([P.to64(g_[:, idx]) for g_ in got], [P.to64(g_[:, idx]) for g_ in ref],
                      "fp32" if dt == torch.float32 else "bf16", f"noalloc {case}")
        del x, o, lse, ref, grads, got
