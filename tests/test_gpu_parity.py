"""GPU parity: the HIP path (through the C ABI) against the CPU oracle on the
same seeded inputs. Small shapes compare every element; the full workload
shapes compare sampled rows that the oracle computes exactly."""

import numpy as np
import pytest
import torch

import oracle as orc
from paper_2507_02754_amd import (load_library, simplicial_attn_bwd, simplicial_attn_bwd_fused_workspace_size,
                                  simplicial_attn_bwd_key_side, simplicial_attn_fwd_biased,
                                  simplicial_attn_bwd_preprocess, simplicial_attn_bwd_query_side,
                                  simplicial_attn_bwd_workspace_size, simplicial_attn_fwd,
                                  simplicial_attn_path_name)
from paper_2507_02754_amd.workloads import WORKLOADS, draw, make_inputs

import parity as P

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    load_library()


def _announce(label):
    print(f"\n[parity] {label}", flush=True)


def test_tiny_fp32_workload_full():
    w = WORKLOADS["tiny_fp32"]
    _announce(f"{w.name} {w.shape()} w1={w.w1} w2={w.w2}")
    inputs = make_inputs(w)
    o, lse = P.gpu_forward(inputs, w.w1, w.w2, w.scale)
    grads = P.gpu_backward(inputs, o, lse, w.w1, w.w2, w.scale)
    o_ref, lse_ref, g_ref = P.full_oracle(inputs, w.w1, w.w2, w.scale)
    P.check_forward(P.to64(o), P.to64(lse), o_ref, lse_ref, "fp32", w.name)
    P.check_grads([P.to64(g) for g in grads], g_ref, "fp32", w.name)


SMALL = [
    # (B, H, N, D, w1, w2, dtype)
    (1, 2, 300, 128, 64, 32, "bf16"),    # several query tiles and a ragged tail
    (2, 1, 200, 64, 40, 32, "bf16"),     # head_dim 64
    (1, 1, 333, 128, 96, 64, "bf16"),    # w2 = 64
    (1, 1, 150, 128, 16, 32, "bf16"),    # w1 < w2
    (1, 1, 20, 128, 512, 32, "bf16"),    # both windows longer than the sequence
    (1, 3, 1, 128, 512, 32, "bf16"),     # a single query
    (1, 1, 129, 128, 33, 7, "bf16"),     # w2 not a multiple of 32
    (1, 1, 100, 64, 7, 5, "fp32"),
    (2, 2, 70, 32, 9, 3, "fp32"),
    (1, 1, 70, 16, 9, 3, "bf16"),
]


@pytest.mark.parametrize("shape", SMALL, ids=[str(s) for s in SMALL])
def test_small_shapes_full(shape):
    b, h, n, d, w1, w2, dt = shape
    _announce(f"small {shape} fwd={simplicial_attn_path_name(0, b, n, h, d, w1, w2, 1 if dt == 'bf16' else 0)}")
    inputs = draw((b, n, h, d), seed=100 + n, dtype=torch.float32 if dt == "fp32" else torch.bfloat16)
    scale = d ** -0.5
    o, lse = P.gpu_forward(inputs, w1, w2, scale)
    grads = P.gpu_backward(inputs, o, lse, w1, w2, scale)
    o_ref, lse_ref, g_ref = P.full_oracle(inputs, w1, w2, scale)
    P.check_forward(P.to64(o), P.to64(lse), o_ref, lse_ref, dt, str(shape))
    if n == 1 and dt == "bf16":
        # one pair per query: dQ, dK, dK' vanish exactly (bounded instead)
        P.check_grads([P.to64(g) for g in grads[3:]], g_ref[3:], dt, str(shape))
        P.check_single_pair_grads([P.to64(g) for g in grads[:3]],
                                  [x.to(torch.float64).numpy() for x in inputs], scale, str(shape))
    else:
        P.check_grads([P.to64(g) for g in grads], g_ref, dt, str(shape))


@pytest.mark.parametrize("d", [128, 64])
def test_running_max_raised_mid_window(d):
    """Keys alternate, 32 at a time, between blocks whose logits sit near -24
    and blocks with logits ~N(0, 1): a window whose first block is a low one
    sets the running maximum there and must raise it (by ~35 in log2 units,
    rescaling the partial sums) when the next block arrives. The low blocks'
    weights are ~e^-24 next to a normal block, so the bf16 rounding of their
    large logits barely reaches the result."""
    b, h, n, w1, w2 = 1, 2, 257, 96, 32
    _announce(f"running max raised mid-window N={n} D={d} w1={w1} w2={w2}")
    g = torch.Generator(device="cpu").manual_seed(7 + d)
    shape = (b, n, h, d)
    q = 1 + 0.1 * torch.randn(shape, generator=g)
    kp = 1 + 0.1 * torch.randn(shape, generator=g)
    k = torch.randn(shape, generator=g)
    low = ((torch.arange(n) // 32) % 2 == 0).view(1, n, 1, 1)
    k = torch.where(low, torch.full_like(k, -2.1 * (128 / d) ** 0.5), k)
    v, vp, do = (torch.randn(shape, generator=g) for _ in range(3))
    inputs = tuple(x.to(torch.bfloat16).contiguous() for x in (q, k, kp, v, vp, do))
    scale = d ** -0.5
    o, lse = P.gpu_forward(inputs, w1, w2, scale)
    grads = P.gpu_backward(inputs, o, lse, w1, w2, scale)
    o_ref, lse_ref, g_ref = P.full_oracle(inputs, w1, w2, scale)
    assert lse_ref.min() < -15  # some queries see only low blocks
    P.check_forward(P.to64(o), P.to64(lse), o_ref, lse_ref, "bf16", f"mid-window max D={d}")
    P.check_grads([P.to64(g_) for g_ in grads], g_ref, "bf16", f"mid-window max D={d}")


@pytest.mark.parametrize("d,w1,w2", [(64, 200, 32), (128, 230, 32), (64, 300, 32), (128, 230, 17)])
def test_forward_tile_runs(d, w1, w2):
    """The forward's XCD-aware tile order over 3 heads of 4096 queries (one
    XCD's contiguous run of 4-query tiles crosses a head boundary), with
    w1 = 200, 230, 300 giving 7, 8 and 10 key blocks per tile: the v' rows
    issued in iteration 0 are covered by the ring waits (>= 7 blocks) and the
    K/V ring stages wrap at different points. Sampled rows of every head, the
    first rows of each head included."""
    b, h, n = 1, 3, 4096
    _announce(f"forward tile runs N={n} H={h} D={d} w1={w1} w2={w2} "
              f"fwd={simplicial_attn_path_name(0, b, n, h, d, w1, w2, 1)}")
    inputs = draw((b, n, h, d), seed=11 + d + w1 + w2, dtype=torch.bfloat16)
    scale = d ** -0.5
    o, lse = P.gpu_forward(inputs, w1, w2, scale)
    rows = P.sample_rows(n, w1, w2, extra=40, seed=w1)
    heads = [(0, x) for x in range(h)]
    P.sampled_forward_check(inputs[:5], o, lse, w1, w2, scale, "bf16", heads, rows,
                            f"tile runs D={d} w1={w1} w2={w2}")


GQA = [
    # (B, H, Hkv, N, D, w1, w2, dtype)
    (1, 4, 2, 300, 128, 64, 32, "bf16"),   # MFMA path, two query heads per K-side head
    (2, 8, 1, 200, 64, 40, 32, "bf16"),    # head_dim 64, all query heads on one K-side head (head-folded)
    (1, 4, 2, 333, 128, 96, 64, "bf16"),   # w2 = 64 (two wavefronts per query)
    (1, 6, 3, 100, 64, 7, 5, "fp32"),      # generic path
    (1, 3, 3, 129, 128, 33, 7, "bf16"),    # Hkv == H
    (1, 64, 1, 96, 64, 40, 32, "bf16"),    # 64 query heads per K-side head (Section 6's ratio)
    (1, 8, 2, 257, 128, 100, 17, "bf16"),  # head-folded, w1 and w2 not multiples of 32
    (2, 16, 1, 70, 128, 512, 32, "bf16"),  # head-folded, windows longer than the sequence
    (1, 4, 1, 1, 128, 512, 32, "bf16"),    # head-folded, a single query
    (1, 6, 2, 150, 128, 64, 32, "bf16"),   # three query heads per K-side head (odd group)
    (2, 6, 3, 97, 64, 40, 64, "bf16"),     # w2 = 64 and head_dim 64, ragged length, two batches
]


def _head_folded(h, hkv, d, w2, dt):
    """Shapes the forward runs with query heads folded into one tile."""
    return dt == "bf16" and d in (64, 128) and w2 <= 32 and hkv < h and (h // hkv) % 4 == 0


def _gqa_inputs(b, h, hkv, n, d, dt, seed):
    tdt = torch.float32 if dt == "fp32" else torch.bfloat16
    g = torch.Generator(device="cpu").manual_seed(seed)
    q = torch.randn((b, n, h, d), generator=g).to(tdt)
    kv = [torch.randn((b, n, hkv, d), generator=g).to(tdt) for _ in range(4)]
    do = torch.randn((b, n, h, d), generator=g).to(tdt)
    return q, kv, do


@pytest.mark.parametrize("shape", GQA, ids=[str(s) for s in GQA])
def test_gqa_forward(shape):
    """Grouped-query forward against the oracle (query head h reads K-side head
    h // (H // Hkv)), and, where query heads are not folded into one tile, bit
    for bit against the plain forward on K, K', V, V' repeated per query head
    (folded tiles walk each query's own key window, a different block
    alignment, so only the oracle comparison applies)."""
    from paper_2507_02754_amd import simplicial_attn_fwd_gqa

    b, h, hkv, n, d, w1, w2, dt = shape
    _announce(f"gqa {shape}")
    tdt = torch.float32 if dt == "fp32" else torch.bfloat16
    g = torch.Generator(device="cpu").manual_seed(500 + n + h)
    q = torch.randn((b, n, h, d), generator=g).to(tdt)
    kv = [torch.randn((b, n, hkv, d), generator=g).to(tdt) for _ in range(4)]
    scale = d ** -0.5
    o, lse = simplicial_attn_fwd_gqa(q.cuda(), *(x.cuda() for x in kv), w1, w2, scale)
    torch.cuda.synchronize()
    rep = [x.repeat_interleave(h // hkv, dim=2).contiguous() for x in kv]
    o_m, lse_m = simplicial_attn_fwd(q.cuda(), *(x.cuda() for x in rep), w1, w2, scale)
    torch.cuda.synchronize()
    if not _head_folded(h, hkv, d, w2, dt):
        assert torch.equal(o, o_m) and torch.equal(lse, lse_m), "GQA forward differs from repeated K/V"
    ref = P.gqa_oracle_forward(q, kv, w1, w2, scale)
    o_ref = np.stack([np.stack([ref[(bb, hh)][0] for hh in range(h)], axis=1) for bb in range(b)])
    lse_ref = np.stack([np.stack([ref[(bb, hh)][1] for hh in range(h)]) for bb in range(b)])
    P.check_forward(P.to64(o), P.to64(lse), o_ref, lse_ref, dt, f"gqa {shape}")


@pytest.mark.parametrize("shape", GQA, ids=[str(s) for s in GQA])
def test_gqa_backward(shape):
    """Grouped-query backward against the oracle (chain rule over the shared
    K-side heads) and against the per-head backward on repeated K, K', V, V'
    with each group's K-side gradients summed in fp32: bit for bit, except dK
    and dV of the MFMA path, which sums the group before rounding (within the
    rounding bound of check_gqa_against_composite)."""
    from paper_2507_02754_amd import simplicial_attn_bwd_gqa, simplicial_attn_fwd_gqa

    b, h, hkv, n, d, w1, w2, dt = shape
    _announce(f"gqa backward {shape}")
    q, kv, do = _gqa_inputs(b, h, hkv, n, d, dt, 900 + n + h)
    scale = d ** -0.5
    qc, kvc, doc = q.cuda(), [x.cuda() for x in kv], do.cuda()
    o, lse = simplicial_attn_fwd_gqa(qc, *kvc, w1, w2, scale)
    grads = simplicial_attn_bwd_gqa(qc, *kvc, o, doc, lse, w1, w2, scale)
    torch.cuda.synchronize()
    assert grads[0].shape == q.shape and all(g_.shape == kv[0].shape for g_ in grads[1:])
    comp, mags = P.gqa_composite_backward(qc, kvc, o, doc, lse, w1, w2, scale, with_abs=True)
    P.check_gqa_against_composite(grads, comp, mags, P.gqa_native(h, hkv, d, w2, dt),
                                  f"gqa backward {shape}")
    dq_ref, dkv_ref = P.gqa_oracle_backward(q, kv, do, w1, w2, scale)
    got = [P.to64(g_) for g_ in grads]
    if n == 1:
        # one pair per query: dQ, dK, dK' vanish exactly; on the GPU each query
        # head's term is off by at most the operand-rounding error of
        # check_single_pair_grads, and the K-side gradients sum H / Hkv of them
        P.check_grads(got[3:], dkv_ref[2:], dt, f"gqa backward {shape} dv")
        g = h // hkv
        q64, do64 = q.double().numpy(), do.double().numpy()
        k64, kp64, v64, vp64 = (x.double().numpy().repeat(g, axis=2) for x in kv)
        eps = 2.0 ** -8 * np.abs(do64 * v64 * vp64).sum(axis=-1, keepdims=True)
        terms = [2 * scale * eps * np.abs(x * y) for x, y in [(k64, kp64), (q64, kp64), (q64, k64)]]
        bounds = [terms[0]] + [t.reshape(b, n, hkv, g, d).sum(axis=3) for t in terms[1:]]
        for name, g_, bd in zip(("dq", "dk", "dkp"), got[:3], bounds):
            assert np.all(np.abs(g_) <= bd + 1e-6), (name, float(np.max(np.abs(g_) - bd)))
    else:
        P.check_grads(got, [dq_ref, *dkv_ref], dt, f"gqa backward {shape}")


def test_gqa_backward_full_size_sampled():
    """16 query heads on 2 K-side heads, N = 4096, w1 = 512, w2 = 32: the whole
    backward against the per-head composite (dQ, dK', dV' bit for bit, dK and
    dV within the rounding bound), and sampled rows of K-side head 0 (all 8 of
    its query heads) against the oracle."""
    from paper_2507_02754_amd import simplicial_attn_bwd_gqa, simplicial_attn_fwd_gqa

    b, h, hkv, n, d, w1, w2 = 1, 16, 2, 4096, 128, 512, 32
    _announce(f"gqa backward full size B={b} H={h} Hkv={hkv} N={n} D={d} w1={w1} w2={w2}")
    q, kv, do = _gqa_inputs(b, h, hkv, n, d, "bf16", 78)
    q = torch.nn.functional.normalize(q.float(), dim=-1).mul(d ** 0.5).to(torch.bfloat16)
    kv[0] = torch.nn.functional.normalize(kv[0].float(), dim=-1).mul(d ** 0.5).to(torch.bfloat16)
    scale = d ** -0.5
    qc, kvc, doc = q.cuda(), [x.cuda() for x in kv], do.cuda()
    o, lse = simplicial_attn_fwd_gqa(qc, *kvc, w1, w2, scale)
    grads = simplicial_attn_bwd_gqa(qc, *kvc, o, doc, lse, w1, w2, scale)
    torch.cuda.synchronize()
    comp, mags = P.gqa_composite_backward(qc, kvc, o, doc, lse, w1, w2, scale, with_abs=True)
    P.check_gqa_against_composite(grads, comp, mags, True, "gqa backward full size")
    q_rows = P.sample_rows(n, w1, w2, extra=2, seed=5)
    key_rows = [0, 1, w2, w1 - 1, n // 2, n - 1]
    queries = set(q_rows)
    for r in key_rows:
        queries.update(range(r, min(n, r + w1)))
    dq_ref, dkv_ref = P.gqa_oracle_backward(q, kv, do, w1, w2, scale, b_heads=[(0, 0)],
                                            queries=sorted(queries))
    got = [P.to64(grads[0])[0][q_rows][:, :h // hkv]] + \
          [P.to64(g_)[0][key_rows][:, 0] for g_ in grads[1:]]
    ref = [dq_ref[0][q_rows][:, :h // hkv]] + [r_[0][key_rows][:, 0] for r_ in dkv_ref]
    P.check_grads(got, ref, "bf16", "gqa backward full size")


def test_autograd_gqa():
    """torch.autograd with fewer K-side heads routes to the GQA entry points:
    gradients equal the direct GQA backward bit for bit."""
    from paper_2507_02754_amd import (simplicial_attention, simplicial_attn_bwd_gqa,
                                      simplicial_attn_fwd_gqa)

    b, h, hkv, n, d, w1, w2 = 1, 4, 2, 200, 128, 64, 32
    _announce("autograd gqa")
    q, kv, do = _gqa_inputs(b, h, hkv, n, d, "bf16", 31)
    scale = d ** -0.5
    leaves = [x.cuda().requires_grad_(True) for x in (q, *kv)]
    o = simplicial_attention(*leaves, w1, w2, scale)
    (o.float() * do.cuda().float()).sum().backward()
    o_d, lse_d = simplicial_attn_fwd_gqa(q.cuda(), *(x.cuda() for x in kv), w1, w2, scale)
    direct = simplicial_attn_bwd_gqa(q.cuda(), *(x.cuda() for x in kv), o_d, do.cuda(), lse_d,
                                     w1, w2, scale)
    assert torch.equal(o.detach(), o_d)
    for name, lf, g2 in zip(P.GRAD_NAMES, leaves, direct):
        assert torch.equal(lf.grad, g2), f"{name}: autograd differs from the direct GQA backward"


DET = [
    # (B, H, N, D, w1, w2, dtype): determinant logits (Section 5), plain fp32 kernels
    (1, 2, 100, 16, 7, 5, "fp32"),      # 5 chunks + 1 unused component
    (1, 2, 130, 64, 33, 7, "fp32"),     # 21 chunks + 1
    (2, 1, 77, 32, 20, 32, "bf16"),     # w2 longer than w1
    (1, 2, 150, 128, 40, 16, "bf16"),   # 42 chunks + 2 (MFMA forward)
    (1, 2, 300, 128, 64, 32, "bf16"),   # MFMA forward, several tiles
    (1, 3, 257, 64, 100, 17, "bf16"),   # MFMA forward, head_dim 64 (21 chunks + 1)
    (2, 1, 100, 64, 7, 5, "bf16"),      # MFMA forward, short windows
    (1, 1, 40, 16, 1, 1, "fp32"),       # unit windows
    (1, 1, 1, 64, 8, 8, "fp32"),        # one query
]


@pytest.mark.parametrize("shape", DET, ids=[str(s) for s in DET])
def test_determinant_form(shape):
    """simplicial_attn_det_fwd / _bwd against the determinant oracle, every element."""
    from oracle import determinant_oracle as dor
    from paper_2507_02754_amd import simplicial_attn_det_bwd, simplicial_attn_det_fwd

    b, h, n, d, w1, w2, dt = shape
    _announce(f"determinant form {shape}")
    inputs = draw((b, n, h, d), seed=700 + n + d, dtype=torch.float32 if dt == "fp32" else torch.bfloat16)
    scale = d ** -0.5
    dev = [x.cuda() for x in inputs]
    o, lse = simplicial_attn_det_fwd(*dev[:5], w1, w2, scale)
    grads = simplicial_attn_det_bwd(*dev[:5], o, dev[5], lse, w1, w2, scale)
    torch.cuda.synchronize()
    o_ref = np.zeros((b, n, h, d))
    lse_ref = np.zeros((b, h, n))
    g_ref = [np.zeros((b, n, h, d)) for _ in range(5)]
    for bb in range(b):
        for hh in range(h):
            arrs = P.head_arrays(inputs, bb, hh)
            o_ref[bb, :, hh], lse_ref[bb, hh] = dor.forward(*arrs[:5], w1, w2, scale)
            for t, g_ in enumerate(dor.backward(*arrs, w1, w2, scale)):
                g_ref[t][bb, :, hh] = g_
    P.check_forward(P.to64(o), P.to64(lse), o_ref, lse_ref, dt, f"det {shape}")
    P.check_grads([P.to64(g_) for g_ in grads], g_ref, dt, f"det {shape}")
    # the D mod 3 trailing components get no Q, K, K' gradient
    tail = 3 * (d // 3)
    for g_ in grads[:3]:
        assert torch.count_nonzero(g_[..., tail:]) == 0


def test_determinant_forward_full_size_sampled():
    """Determinant forward on the MFMA kernel at B=1, H=4, N=8192, D=128,
    w1=512, w2=32: sampled rows of every head against the determinant oracle."""
    from oracle import determinant_oracle as dor
    from paper_2507_02754_amd import simplicial_attn_det_fwd

    b, h, n, d, w1, w2 = 1, 4, 8192, 128, 512, 32
    _announce(f"determinant forward full size B={b} H={h} N={n} D={d} w1={w1} w2={w2}")
    inputs = draw((b, n, h, d), seed=808, dtype=torch.bfloat16)
    scale = d ** -0.5
    o, lse = simplicial_attn_det_fwd(*(x.cuda() for x in inputs[:5]), w1, w2, scale)
    torch.cuda.synchronize()
    rows = P.sample_rows(n, w1, w2, extra=6, seed=9)
    o64, l64 = P.to64(o), P.to64(lse)
    got_o, got_l, ref_o, ref_l = [], [], [], []
    for hh in range(h):
        arrs = P.head_arrays(inputs, 0, hh)
        ro, rl = dor.forward(*arrs[:5], w1, w2, scale, queries=rows)
        got_o.append(o64[0, rows, hh])
        got_l.append(l64[0, hh, rows])
        ref_o.append(ro[rows])
        ref_l.append(rl[rows])
    P.check_forward(np.concatenate(got_o), np.concatenate(got_l), np.concatenate(ref_o),
                    np.concatenate(ref_l), "bf16", "determinant full size")


def test_determinant_backward_full_size_sampled():
    """Determinant backward on the MFMA kernels at B=1, H=2, N=8192, D=128,
    w1=512, w2=32 (with the dQ~ rows through the workspace): dQ every 64
    queries, dK / dV and dK' / dV' on rows spread over the sequence, both heads,
    against the determinant oracle (every query touching a checked row)."""
    from oracle import determinant_oracle as dor
    from paper_2507_02754_amd import simplicial_attn_det_bwd, simplicial_attn_det_fwd

    b, h, n, d, w1, w2 = 1, 2, 8192, 128, 512, 32
    _announce(f"determinant backward full size B={b} H={h} N={n} D={d} w1={w1} w2={w2} "
              f"bwd={simplicial_attn_path_name(1, b, n, h, d, w1, w2, 1)}")
    inputs = draw((b, n, h, d), seed=809, dtype=torch.bfloat16)
    scale = d ** -0.5
    x = [t.cuda() for t in inputs]
    o, lse = simplicial_attn_det_fwd(*x[:5], w1, w2, scale)
    grads = simplicial_attn_det_bwd(*x[:5], o, x[5], lse, w1, w2, scale)
    torch.cuda.synchronize()
    q_rows = sorted(set(range(0, n, 64)) | {1, 2, 31, 32, n - 2, n - 1})
    k_rows = sorted({0, 1, 300, 511, n // 2, n - 700, n - 1})
    kp_rows = sorted(set(range(5, n, 509)) | {0, 30, n - 1})
    queries = set(q_rows)
    for r in k_rows:
        queries.update(range(r, min(n, r + w1)))
    for r in kp_rows:
        queries.update(range(r, min(n, r + w2)))
    rows = [q_rows, k_rows, kp_rows, k_rows, kp_rows]
    got = [[] for _ in range(5)]
    ref = [[] for _ in range(5)]
    import oracle_pool
    for hh in range(h):
        arrs = P.head_arrays(inputs, 0, hh)
        g_ref = oracle_pool.backward(*arrs, w1, w2, scale, sorted(queries), rows,
                                     module="oracle.determinant_oracle")
        for t in range(5):
            got[t].append(P.to64(grads[t][0, :, hh][torch.tensor(rows[t], device="cuda")]))
            ref[t].append(g_ref[t])
    P.check_grads([np.concatenate(g_) for g_ in got], [np.concatenate(r_) for r_ in ref], "bf16",
                  "determinant backward full size")


def test_gqa_forward_full_size_sampled():
    """16 query heads on 2 K-side heads, N = 8192, w1 = 512, w2 = 32: sampled rows
    of every query head against the oracle."""
    from paper_2507_02754_amd import simplicial_attn_fwd_gqa

    b, h, hkv, n, d, w1, w2 = 1, 16, 2, 8192, 128, 512, 32
    _announce(f"gqa full size B={b} H={h} Hkv={hkv} N={n} D={d} w1={w1} w2={w2}")
    g = torch.Generator(device="cpu").manual_seed(77)
    q = torch.randn((b, n, h, d), generator=g).to(torch.bfloat16)
    kv = [torch.randn((b, n, hkv, d), generator=g).to(torch.bfloat16) for _ in range(4)]
    scale = d ** -0.5
    o, lse = simplicial_attn_fwd_gqa(q.cuda(), *(x.cuda() for x in kv), w1, w2, scale)
    torch.cuda.synchronize()
    rows = P.sample_rows(n, w1, w2, extra=6, seed=3)
    heads = [(0, hh) for hh in range(h)]
    ref = P.gqa_oracle_forward(q, kv, w1, w2, scale, heads=heads, rows=rows)
    o64, l64 = P.to64(o), P.to64(lse)
    P.check_forward(np.concatenate([o64[0, rows, hh, :] for (_, hh) in heads]),
                    np.concatenate([l64[0, hh, rows] for (_, hh) in heads]),
                    np.concatenate([ref[k_][0][rows] for k_ in heads]),
                    np.concatenate([ref[k_][1][rows] for k_ in heads]), "bf16", "gqa full size")


def _is_fast(w, which):
    return simplicial_attn_path_name(which, w.B, w.N, w.H, w.D, w.w1, w.w2, 1) != "generic"


# Full-size forward: whole heads compared element by element (every query),
# other heads on sampled rows. Oracle time (one CPU thread, ~0.8 ms per query
# at w1 = 512, w2 = 32 and ~1.8 ms at 1024, 64) is spread over worker processes.
FULL_FWD = {
    "fwd_bf16_n4k": ([(0, h) for h in range(8)], []),
    "fb_bf16_n8k": ([(0, 0), (1, 7)], [(0, 3)]),
    "long_bf16_n32k": ([(0, 0)], [(0, 15)]),
    "wide_bf16_n16k": ([(0, 0)], [(3, 15)]),
}


def _spread_rows(n, stride, phase, w1, w2, seed):
    """Rows every `stride` (with a moving offset inside each stride, so that
    different positions within a kernel tile are hit) plus the edge rows."""
    rows = set(P.sample_rows(n, w1, w2, seed=seed))
    rows.update((t * stride + (t * phase) % stride) for t in range(n // stride))
    return sorted(r for r in rows if 0 <= r < n)


@pytest.mark.parametrize("name", list(FULL_FWD))
def test_full_size_forward(name):
    import oracle_pool

    w = WORKLOADS[name]
    if not _is_fast(w, 0):
        pytest.skip("full-size shapes are only run on the MFMA path")
    full, sampled = FULL_FWD[name]
    _announce(f"{w.name} forward {w.shape()} w1={w.w1} w2={w.w2}: whole heads {full}, sampled {sampled}, "
              f"{oracle_pool.workers()} oracle workers")
    inputs = make_inputs(w)
    o, lse = P.gpu_forward(inputs, w.w1, w.w2, w.scale)
    rows_s = _spread_rows(w.N, 97, 31, w.w1, w.w2, w.seed)
    for (b, h) in full + sampled:
        rows = list(range(w.N)) if (b, h) in full else rows_s
        arrs = P.head_arrays(inputs[:5], b, h)
        o_ref, l_ref = oracle_pool.forward(*arrs, w.w1, w.w2, w.scale, rows)
        idx = torch.tensor(rows, device=o.device)
        P.check_forward(P.to64(o[b, :, h][idx]), P.to64(lse[b, h][idx]), o_ref, l_ref, w.dtype,
                        f"{w.name} head {(b, h)} {'all' if (b, h) in full else len(rows)} queries")


# Full-size backward: per head, dQ on every 16th query, dK / dV on key rows
# spread over the sequence (one per `kstride`, a different position inside each
# 128-key tile of the key-side kernel every time), dK' / dV' on one row per
# `kpstride`, plus the edge rows. The oracle runs every query that touches a
# checked row, so each checked row is exact.
FULL_BWD = {
    # name: [(head, kstride, kpstride), ...]
    "fb_bf16_n8k": [((0, 0), 256, 64), ((1, 7), 256, 64)],
    "long_bf16_n32k": [((0, 0), 512, 128), ((0, 15), 2048, 256)],
    "wide_bf16_n16k": [((0, 0), 2048, 256), ((3, 15), 2048, 256)],
}


@pytest.mark.parametrize("name", list(FULL_BWD))
def test_full_size_backward(name):
    import oracle_pool

    w = WORKLOADS[name]
    if not (_is_fast(w, 0) and _is_fast(w, 1)):
        pytest.skip("full-size shapes are only run on the MFMA path")
    _announce(f"{w.name} backward {w.shape()} w1={w.w1} w2={w.w2}: {FULL_BWD[name]}, "
              f"{oracle_pool.workers()} oracle workers")
    inputs = make_inputs(w)
    o, lse = P.gpu_forward(inputs, w.w1, w.w2, w.scale)
    grads = P.gpu_backward(inputs, o, lse, w.w1, w.w2, w.scale)
    n = w.N
    edges = [0, 1, w.w2 - 1, w.w1 - 1, n // 2, n - 2, n - 1]
    for (b, h), kstride, kpstride in FULL_BWD[name]:
        q_rows = _spread_rows(n, 16, 5, w.w1, w.w2, w.seed)
        k_rows = sorted(set(edges) | set(_spread_rows(n, kstride, 37, 1, 1, w.seed)))
        kp_rows = sorted(set(edges) | set(_spread_rows(n, kpstride, 13, 1, 1, w.seed)))
        queries = set(q_rows)
        for r in k_rows:
            queries.update(range(r, min(n, r + w.w1)))
        for r in kp_rows:
            queries.update(range(r, min(n, r + w.w2)))
        rows = [q_rows, k_rows, kp_rows, k_rows, kp_rows]
        arrs = P.head_arrays(inputs, b, h)
        ref = oracle_pool.backward(*arrs, w.w1, w.w2, w.scale, sorted(queries), rows)
        got = [P.to64(g[b, :, h][torch.tensor(r, device=g.device)]) for g, r in zip(grads, rows)]
        P.check_grads(got, ref, w.dtype,
                      f"{w.name} head {(b, h)}: dq {len(q_rows)} rows, dk/dv {len(k_rows)}, "
                      f"dk'/dv' {len(kp_rows)} ({len(queries)} oracle queries)")


@pytest.mark.parametrize("shape", [(1, 2, 300, 128, 64, 32, "bf16"), (1, 1, 100, 64, 7, 5, "fp32")],
                         ids=["bf16", "fp32"])
def test_autograd_function(shape):
    """Gradients through torch.autograd (loss = sum(O * dO)) equal the direct
    backward call bit for bit and match the oracle; LSE carries no gradient."""
    from paper_2507_02754_amd import simplicial_attention

    b, h, n, d, w1, w2, dt = shape
    _announce(f"autograd {shape}")
    inputs = draw((b, n, h, d), seed=300 + n, dtype=torch.float32 if dt == "fp32" else torch.bfloat16)
    scale = d ** -0.5
    leaves = [x.to("cuda").requires_grad_(True) for x in inputs[:5]]
    do = inputs[5].to("cuda")
    o = simplicial_attention(*leaves, w1, w2, scale)
    (o.float() * do.float()).sum().backward()
    auto = [x.grad for x in leaves]
    o_d, lse_d = P.gpu_forward(inputs, w1, w2, scale)
    direct = P.gpu_backward(inputs, o_d, lse_d, w1, w2, scale)
    assert torch.equal(o.detach(), o_d), "autograd forward differs from the direct call"
    for name, g1, g2 in zip(("dq", "dk", "dkp", "dv", "dvp"), auto, direct):
        assert torch.equal(g1, g2), f"{name}: autograd differs from the direct backward"
    o_ref, lse_ref, g_ref = P.full_oracle(inputs, w1, w2, scale)
    P.check_forward(P.to64(o.detach()), P.to64(lse_d), o_ref, lse_ref, dt, f"autograd {shape}")
    P.check_grads([P.to64(g) for g in auto], g_ref, dt, f"autograd {shape}")


def test_unit_windows_through_gpu():
    """w1 = w2 = 1: each query sees only the pair (i, i), so O = V o V',
    dV = dO o V' and dV' = dO o V (checked at the usual tolerance), while dQ, dK
    and dK' vanish in exact arithmetic. On the GPU they equal
    scale * (dP_i - Delta_i) * (x_i o y_i), where dP_i is a product of bf16-rounded
    operands and Delta_i uses the bf16 output; each is off by at most
    2^-9 * sum_d |dO_id v_id v'_id|, which bounds them (with a factor 2 margin)."""
    b, h, n, d = 1, 1, 100, 128
    _announce("unit windows")
    inputs = draw((b, n, h, d), seed=200)
    scale = d ** -0.5
    o, lse = P.gpu_forward(inputs, 1, 1, scale)
    grads = P.gpu_backward(inputs, o, lse, 1, 1, scale)
    o_ref, lse_ref, g_ref = P.full_oracle(inputs, 1, 1, scale)
    P.check_forward(P.to64(o), P.to64(lse), o_ref, lse_ref, "bf16", "unit windows")
    dgrads = [P.to64(g) for g in grads]
    P.check_grads(dgrads[3:], g_ref[3:], "bf16", "unit windows dv")
    P.check_single_pair_grads(dgrads[:3], [x.to(torch.float64).numpy() for x in inputs], scale,
                              "unit windows")


def test_backward_is_deterministic():
    shape = (1, 2, 400, 128, 128, 32)
    b, h, n, d, w1, w2 = shape
    _announce(f"determinism {shape}")
    inputs = [x.cuda() for x in draw((b, n, h, d), seed=7)]
    o, lse = simplicial_attn_fwd(*inputs[:5], w1, w2)
    runs = []
    for _ in range(3):
        g = simplicial_attn_bwd(*inputs[:5], o, inputs[5], lse, w1, w2)
        torch.cuda.synchronize()
        runs.append([x.clone() for x in g])
    for r in runs[1:]:
        for a, c in zip(runs[0], r):
            assert torch.equal(a.view(torch.int16), c.view(torch.int16))


@pytest.mark.parametrize("d,w1", [(128, 230), (64, 200)])
def test_forward_is_deterministic(d, w1):
    """The forward has no atomics and a fixed order of operations: repeated
    calls on the same inputs (3 heads of 4096 queries, w2 = 32) must agree
    bit for bit."""
    b, h, n, w2 = 1, 3, 4096, 32
    _announce(f"forward determinism N={n} H={h} D={d} w1={w1} w2={w2}")
    inputs = [x.cuda() for x in draw((b, n, h, d), seed=11 + d + w1 + w2)[:5]]
    o0, l0 = simplicial_attn_fwd(*inputs, w1, w2)
    torch.cuda.synchronize()
    o0, l0 = o0.clone(), l0.clone()
    differing = 0
    for _ in range(8):
        o, lse = simplicial_attn_fwd(*inputs, w1, w2)
        torch.cuda.synchronize()
        if not (torch.equal(o.view(torch.int16), o0.view(torch.int16)) and torch.equal(lse, l0)):
            differing += 1
    assert differing == 0, f"{differing} of 8 repeated forwards differ from the first"


@pytest.mark.parametrize("shape", [(1, 2, 700, 128, 256, 32), (1, 1, 300, 64, 40, 64),
                                   (1, 1, 90, 64, 7, 5)])
def test_staged_backward_matches_composite(shape):
    """preprocess + query side + key side (the three stage entry points) give
    bitwise the same gradients as simplicial_attn_bwd; where the fused
    backward takes the shape, its gradients agree with them at the parity
    bar (both are checked against the oracle by other tests)."""
    b, h, n, d, w1, w2 = shape
    _announce(f"staged backward {shape}")
    dt = torch.bfloat16 if (w1, w2) != (7, 5) else torch.float32
    x = [t.cuda() for t in draw((b, n, h, d), seed=12, dtype=dt)]
    o, lse = simplicial_attn_fwd(*x[:5], w1, w2)
    ref = simplicial_attn_bwd(*x[:5], o, x[5], lse, w1, w2)
    ws = torch.empty(simplicial_attn_bwd_workspace_size(b, n, h, d, w1, w2, dt), dtype=torch.uint8,
                     device="cuda")
    simplicial_attn_bwd_preprocess(o, x[5], w1, w2, ws)
    dq, dkp, dvp = simplicial_attn_bwd_query_side(*x[:5], x[5], lse, w1, w2, ws)
    dk, dv = simplicial_attn_bwd_key_side(*x[:5], x[5], lse, w1, w2, ws)
    torch.cuda.synchronize()
    for a, c in zip(ref, (dq, dk, dkp, dv, dvp)):
        assert torch.equal(a, c)
    if simplicial_attn_bwd_fused_workspace_size(b, n, h, d, w1, w2, dt):
        fused = P.gpu_backward_fused(x, o, lse, w1, w2, d ** -0.5)
        P.check_grads([P.to64(g) for g in fused], [P.to64(g) for g in ref], "bf16", f"fused vs split {shape}")


# ---- fused backward (one computation of S and dP; Section 7's gradients) ----

FUSED = [
    # (B, H, N, D, w1, w2)
    (1, 2, 300, 128, 64, 32),    # several 64-key blocks and a ragged tail
    (1, 1, 150, 128, 16, 32),    # w1 < w2
    (1, 1, 20, 128, 512, 32),    # both windows longer than the sequence
    (1, 2, 65, 128, 64, 17),     # a second key block with one key
    (2, 1, 190, 128, 100, 31),   # w2 = 31
    (1, 1, 129, 128, 33, 7),     # w2 not a multiple of 32, k-rows outside the window inside the tile
    (2, 2, 640, 128, 300, 32),   # key blocks past the edge of every window
]


@pytest.mark.parametrize("shape", FUSED, ids=[str(s) for s in FUSED])
def test_fused_backward_small_full(shape):
    b, h, n, d, w1, w2 = shape
    _announce(f"fused backward {shape}")
    inputs = draw((b, n, h, d), seed=200 + n)
    scale = d ** -0.5
    o, lse = P.gpu_forward(inputs, w1, w2, scale)
    grads = P.gpu_backward_fused(inputs, o, lse, w1, w2, scale)
    _, _, g_ref = P.full_oracle(inputs, w1, w2, scale)
    P.check_grads([P.to64(g) for g in grads], g_ref, "bf16", f"fused {shape}")


def test_fused_backward_single_pair_edges():
    """N = 1 and unit windows: one pair per query, so dQ, dK, dK' vanish
    exactly (bounded by the operand rounding) and dV, dV' are exact products."""
    for (b, h, n, d, w1, w2) in [(1, 3, 1, 128, 512, 32), (1, 2, 130, 128, 1, 1)]:
        _announce(f"fused backward single pair {(b, h, n, d, w1, w2)}")
        inputs = draw((b, n, h, d), seed=300 + n)
        o, lse = P.gpu_forward(inputs, w1, w2, d ** -0.5)
        grads = P.gpu_backward_fused(inputs, o, lse, w1, w2, d ** -0.5)
        _, _, g_ref = P.full_oracle(inputs, w1, w2, d ** -0.5)
        P.check_grads([P.to64(g) for g in grads[3:]], g_ref[3:], "bf16", f"fused single pair {n}")
        P.check_single_pair_grads([P.to64(g) for g in grads[:3]], [t.double().numpy() for t in inputs],
                                  d ** -0.5, f"fused single pair {n}")


def test_fused_backward_with_bias_constants():
    b, h, n, d, w1, w2 = 1, 2, 300, 128, 64, 32
    kb, vb = 0.75, -0.5
    _announce("fused backward with K'/V' constants")
    inputs = draw((b, n, h, d), seed=71)
    scale = d ** -0.5
    q, k, kp, v, vp = (t.cuda() for t in inputs[:5])
    o, lse = simplicial_attn_fwd_biased(q, k, kp, v, vp, w1, w2, scale, kb, vb)
    grads = P.gpu_backward_fused(inputs, o, lse, w1, w2, scale, kp_bias=kb, vp_bias=vb)
    shifted = [t.double() for t in inputs]
    shifted[2] = shifted[2] + kb
    shifted[4] = shifted[4] + vb
    _, _, g_ref = P.full_oracle(shifted, w1, w2, scale)
    P.check_grads([P.to64(g) for g in grads], g_ref, "bf16", "fused biased")


def test_fused_backward_is_deterministic():
    b, h, n, d, w1, w2 = 1, 4, 2000, 128, 512, 32
    _announce("fused backward determinism")
    inputs = draw((b, n, h, d), seed=81)
    o, lse = P.gpu_forward(inputs, w1, w2, d ** -0.5)
    g0 = P.gpu_backward_fused(inputs, o, lse, w1, w2, d ** -0.5)
    for _ in range(3):
        g1 = P.gpu_backward_fused(inputs, o, lse, w1, w2, d ** -0.5)
        for a, c in zip(g0, g1):
            assert torch.equal(a.view(torch.int16), c.view(torch.int16))


@pytest.mark.parametrize("name", ["fb_bf16_n8k", "long_bf16_n32k"])
def test_fused_backward_full_size(name):
    """At full size: two heads, dQ every 16 queries, dK / dV and dK' / dV' rows
    spread over the sequence (and the edges), each against the oracle run on
    every query that touches them."""
    import oracle_pool

    w = WORKLOADS[name]
    _announce(f"fused backward {w.name} {w.shape()} w1={w.w1} w2={w.w2}")
    inputs = make_inputs(w)
    o, lse = P.gpu_forward(inputs, w.w1, w.w2, w.scale)
    grads = P.gpu_backward_fused(inputs, o, lse, w.w1, w.w2, w.scale)
    n = w.N
    edges = [0, 1, w.w2 - 1, w.w1 - 1, 63, 64, n // 2, n - 2, n - 1]
    for (b, h), kstride, kpstride in FULL_BWD[name]:
        q_rows = _spread_rows(n, 16, 7, w.w1, w.w2, w.seed)
        k_rows = sorted(set(edges) | set(_spread_rows(n, kstride, 41, 1, 1, w.seed)))
        kp_rows = sorted(set(edges) | set(_spread_rows(n, kpstride, 11, 1, 1, w.seed)))
        queries = set(q_rows)
        for r in k_rows:
            queries.update(range(r, min(n, r + w.w1)))
        for r in kp_rows:
            queries.update(range(r, min(n, r + w.w2)))
        rows = [q_rows, k_rows, kp_rows, k_rows, kp_rows]
        arrs = P.head_arrays(inputs, b, h)
        ref = oracle_pool.backward(*arrs, w.w1, w.w2, w.scale, sorted(queries), rows)
        got = [P.to64(g[b, :, h][torch.tensor(r, device=g.device)]) for g, r in zip(grads, rows)]
        P.check_grads(got, ref, w.dtype, f"fused {w.name} head {(b, h)}: dq {len(q_rows)} rows, "
                      f"dk/dv {len(k_rows)}, dk'/dv' {len(kp_rows)} ({len(queries)} oracle queries)")


def test_unit_values_through_gpu():
    """V = V' = 1 gives O = 1 and zero key/query gradients (exact identities)."""
    b, h, n, d, w1, w2 = 1, 2, 260, 128, 64, 32
    _announce("unit values")
    q, k, kp, _, _, do = draw((b, n, h, d), seed=8)
    ones = torch.ones_like(q)
    dev = [x.cuda() for x in (q, k, kp, ones, ones, do)]
    o, lse = simplicial_attn_fwd(*dev[:5], w1, w2)
    dq, dk, dkp, dv, dvp = simplicial_attn_bwd(*dev[:5], o, dev[5], lse, w1, w2)
    torch.cuda.synchronize()
    assert torch.allclose(o.float(), torch.ones_like(o, dtype=torch.float32), atol=8e-3)
    # dv_j = sum_{i,k} P_ijk dO_i: compare with the oracle; dq, dk, dkp vanish.
    for g in (dq, dk, dkp):
        assert g.float().abs().max().item() <= 5e-3 * max(1.0, dv.float().abs().max().item())


def test_guard_bands_untouched_and_no_stray_reads():
    """Tensors live inside NaN-filled allocations; outputs must be finite and the
    guard regions around every output must still be NaN afterwards."""
    b, h, n, d, w1, w2 = 1, 2, 190, 128, 64, 32
    _announce("guard bands")
    inputs = draw((b, n, h, d), seed=9)
    numel = b * n * h * d
    pad = 4096

    def guarded(x=None, dtype=torch.bfloat16, count=numel):
        buf = torch.full((count + 2 * pad,), float("nan"), dtype=dtype, device="cuda")
        view = buf[pad:pad + count]
        if x is not None:
            view.copy_(x.reshape(-1))
        return buf, view

    bufs = [guarded(x) for x in inputs]
    t = [v.view(b, n, h, d) for _, v in bufs]
    ob, ov = guarded()
    lb, lv = guarded(dtype=torch.float32, count=b * h * n)
    o, lse = simplicial_attn_fwd(*t[:5], w1, w2, out=ov.view(b, n, h, d), lse=lv.view(b, h, n))
    gbufs = [guarded() for _ in range(5)]
    grads = tuple(v.view(b, n, h, d) for _, v in gbufs)
    simplicial_attn_bwd(*t[:5], o, t[5], lse, w1, w2, grads=grads)
    torch.cuda.synchronize()
    for buf, view in [(ob, ov), (lb, lv), *gbufs]:
        assert torch.isfinite(view.float()).all()
        assert torch.isnan(buf[:pad].float()).all() and torch.isnan(buf[-pad:].float()).all()
    o_ref, lse_ref, g_ref = P.full_oracle(inputs, w1, w2, d ** -0.5)
    P.check_forward(P.to64(o), P.to64(lse), o_ref, lse_ref, "bf16", "guard")
    P.check_grads([P.to64(g) for g in grads], g_ref, "bf16", "guard")
