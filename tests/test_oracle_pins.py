"""Pins of the CPU oracle against facts fixed by the paper and by mathematics.

None of these compares the oracle with itself: each checks it against a
different formulation (Algorithm 1 executed densely), a library routine
(torch's scaled-dot-product attention, torch autograd), a closed form derived
by hand, an exact identity, or central finite differences.
"""

import math

import numpy as np
import pytest
import torch

import oracle as orc

RNG = np.random.default_rng(12345)


def rand_heads(b, n, h, d, count=5, rng=RNG, scale=1.0):
    return [rng.standard_normal((b, n, h, d)) * scale for _ in range(count)]


SHAPES = [
    # (B, N, H, D, w1, w2)
    (1, 7, 2, 4, 3, 2),
    (2, 16, 1, 8, 5, 7),     # w1 < w2
    (1, 12, 1, 6, 20, 20),   # windows wider than the sequence: plain causal Algorithm 1
    (1, 1, 1, 4, 3, 3),      # a single query
    (1, 10, 1, 5, 1, 1),     # w1 = w2 = 1
    (1, 9, 2, 3, 4, 1),      # w2 = 1
    (1, 13, 1, 4, 1, 6),     # w1 = 1
    (1, 24, 1, 16, 9, 4),
]


@pytest.mark.parametrize("shape", SHAPES)
def test_windowed_matches_algorithm1_brute_force(shape):
    """Section 4, Algorithm 1: the dense N^3 einsum with the window mask."""
    b, n, h, d, w1, w2 = shape
    q, k, kp, v, vp = rand_heads(b, n, h, d)
    scale = d ** -0.5
    o_bf, lse_bf, p_bf = orc.brute_force_forward(q, k, kp, v, vp, w1, w2, scale)
    o, lse = orc.forward_batched(q, k, kp, v, vp, w1, w2, scale)
    np.testing.assert_allclose(o, o_bf, rtol=0, atol=1e-12)
    np.testing.assert_allclose(lse, lse_bf, rtol=0, atol=1e-12)
    # The probabilities of one query agree entry by entry inside the window and
    # the dense tensor is exactly zero outside it.
    for i in range(n):
        _, _, p, (j0, j1), (k0, k1) = orc.query_forward(
            q[0, :, 0], k[0, :, 0], kp[0, :, 0], v[0, :, 0], vp[0, :, 0], i, w1, w2, scale)
        dense = p_bf[0, 0, i]
        np.testing.assert_allclose(dense[j0:j1, k0:k1], p, rtol=0, atol=1e-14)
        assert dense.sum() == pytest.approx(1.0, abs=1e-13)
        outside = dense.copy()
        outside[j0:j1, k0:k1] = 0.0
        assert np.all(outside == 0.0)


def _sdpa_fp64(q, k, v, w, scale):
    """Causal sliding-window softmax attention by torch's library routine (fp64, CPU)."""
    n = q.shape[0]
    i = torch.arange(n)[:, None]
    j = torch.arange(n)[None, :]
    mask = (j <= i) & (j > i - w)
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a))[None, None]
    out = torch.nn.functional.scaled_dot_product_attention(
        t(q), t(k), t(v), attn_mask=mask[None, None], scale=scale)
    logits = (t(q) @ t(k).transpose(-1, -2))[0, 0] * scale
    lse = torch.logsumexp(logits.masked_fill(~mask, float("-inf")), dim=-1)
    return out[0, 0].numpy(), lse.numpy()


@pytest.mark.parametrize("n,d,w1,w2", [(40, 8, 7, 5), (33, 16, 40, 3), (25, 4, 1, 9)])
def test_reduces_to_sliding_window_attention(n, d, w1, w2):
    """K' = 1 and V' = 1: the trilinear form becomes <q_i, k_j>, constant in k,
    so the joint softmax marginalises to standard sliding-window attention over
    w1 keys (Section 4, Eqs. 1-3 for the 1-simplex); the w2 count only shifts the
    log-sum-exp by log(#k)."""
    rng = np.random.default_rng(7)
    q, k, v = (rng.standard_normal((n, d)) for _ in range(3))
    ones = np.ones((n, d))
    scale = 0.37
    o, lse = orc.forward(q, k, ones, v, ones, w1, w2, scale)
    o_ref, lse_ref = _sdpa_fp64(q, k, v, w1, scale)
    np.testing.assert_allclose(o, o_ref, rtol=0, atol=1e-12)
    nk = np.minimum(np.arange(n) + 1, w2)
    np.testing.assert_allclose(lse, lse_ref + np.log(nk), rtol=0, atol=1e-12)


def test_w2_one_reduces_to_attention_on_modulated_queries():
    """w2 = 1: only k = i survives, so o_i = v'_i o SWA(q_i o k'_i; K, V)."""
    rng = np.random.default_rng(8)
    n, d, w1 = 30, 8, 6
    q, k, kp, v, vp = (rng.standard_normal((n, d)) for _ in range(5))
    scale = d ** -0.5
    o, _ = orc.forward(q, k, kp, v, vp, w1, 1, scale)
    swa, _ = _sdpa_fp64(q * kp, k, v, w1, scale)
    np.testing.assert_allclose(o, vp * swa, rtol=0, atol=1e-12)


def test_swap_symmetry_forward_and_backward():
    """Swapping (K, V, w1) with (K', V', w2) leaves the output unchanged and swaps
    the gradients (the trilinear form and the Hadamard product are symmetric;
    Listing 2 exploits it with its role flip)."""
    rng = np.random.default_rng(9)
    n, d, w1, w2 = 21, 6, 8, 3
    q, k, kp, v, vp, do = (rng.standard_normal((n, d)) for _ in range(6))
    s = 0.3
    o1, l1 = orc.forward(q, k, kp, v, vp, w1, w2, s)
    o2, l2 = orc.forward(q, kp, k, vp, v, w2, w1, s)
    np.testing.assert_allclose(o1, o2, atol=1e-12)
    np.testing.assert_allclose(l1, l2, atol=1e-12)
    g1 = orc.backward(q, k, kp, v, vp, do, w1, w2, s)
    g2 = orc.backward(q, kp, k, vp, v, do, w2, w1, s)
    for a, b in zip(g1, (g2[0], g2[2], g2[1], g2[4], g2[3])):
        np.testing.assert_allclose(a, b, atol=1e-12)


def test_query_zero_closed_form():
    """Query 0 sees exactly one pair (0, 0): o_0 = v_0 o v'_0, lse_0 = scale <q0,k0,k'0>."""
    rng = np.random.default_rng(10)
    n, d = 6, 5
    q, k, kp, v, vp = (rng.standard_normal((n, d)) for _ in range(5))
    o, lse = orc.forward(q, k, kp, v, vp, 4, 3, 0.7)
    np.testing.assert_allclose(o[0], v[0] * vp[0], atol=1e-15)
    assert lse[0] == pytest.approx(0.7 * float(np.sum(q[0] * k[0] * kp[0])), abs=1e-14)


def test_degenerate_unit_windows():
    """w1 = w2 = 1: P = 1 on (i, i, i); O = V o V', dV = dO o V', dV' = dO o V and
    dQ = dK = dK' = 0 (the softmax of a single logit has zero derivative)."""
    rng = np.random.default_rng(11)
    n, d = 9, 4
    q, k, kp, v, vp, do = (rng.standard_normal((n, d)) for _ in range(6))
    o, lse = orc.forward(q, k, kp, v, vp, 1, 1, 0.5)
    np.testing.assert_allclose(o, v * vp, atol=1e-15)
    np.testing.assert_allclose(lse, 0.5 * np.sum(q * k * kp, axis=1), atol=1e-14)
    dq, dk, dkp, dv, dvp = orc.backward(q, k, kp, v, vp, do, 1, 1, 0.5)
    np.testing.assert_allclose(dv, do * vp, atol=1e-15)
    np.testing.assert_allclose(dvp, do * v, atol=1e-15)
    for g in (dq, dk, dkp):
        np.testing.assert_allclose(g, 0.0, atol=1e-15)


def test_unit_values_give_unit_output_and_no_key_gradients():
    """V = V' = 1: every v_j o v'_k is the ones vector, so O = 1 whatever the
    probabilities; then dP = <dO_i, 1> is constant in (j, k), dS = 0 and
    dQ = dK = dK' = 0."""
    rng = np.random.default_rng(12)
    n, d, w1, w2 = 17, 6, 5, 4
    q, k, kp, do = (rng.standard_normal((n, d)) for _ in range(4))
    ones = np.ones((n, d))
    o, _ = orc.forward(q, k, kp, ones, ones, w1, w2, 0.4)
    np.testing.assert_allclose(o, 1.0, atol=1e-14)
    dq, dk, dkp, dv, dvp = orc.backward(q, k, kp, ones, ones, do, w1, w2, 0.4)
    for g in (dq, dk, dkp):
        np.testing.assert_allclose(g, 0.0, atol=1e-13)


def test_bilinearity_in_values():
    rng = np.random.default_rng(13)
    n, d = 15, 4
    q, k, kp, v, vp = (rng.standard_normal((n, d)) for _ in range(5))
    o, _ = orc.forward(q, k, kp, v, vp, 6, 3, 0.5)
    o2, _ = orc.forward(q, k, kp, 2.5 * v, -0.75 * vp, 6, 3, 0.5)
    np.testing.assert_allclose(o2, -1.875 * o, atol=1e-13)


def test_hand_worked_example():
    """A 2-token, D = 1 example worked by hand from Eqs. (3d-attention), (softmax)
    and (attenval) with scale 1 and w1 = w2 = 2.

    q_1 = 1, k = (0, ln 3), k' = (1, 1): the four logits of query 1 are
    (0, 0, ln 3, ln 3), so the weights are 1, 1, 3, 3 over a total of 8:
    lse_1 = ln 8 and, with v = (1, 2), v' = (1, 1), o_1 = (2*1 + 6*2)/8 = 1.75.
    Query 0: o_0 = v_0 v'_0 = 1, lse_0 = q_0 k_0 k'_0 = 0.
    """
    q = np.array([[5.0], [1.0]])
    k = np.array([[0.0], [math.log(3.0)]])
    kp = np.ones((2, 1))
    v = np.array([[1.0], [2.0]])
    vp = np.ones((2, 1))
    o, lse = orc.forward(q, k, kp, v, vp, 2, 2, 1.0)
    assert o[1, 0] == pytest.approx(1.75, abs=1e-15)
    assert lse[1] == pytest.approx(math.log(8.0), abs=1e-15)
    assert o[0, 0] == pytest.approx(1.0, abs=1e-15)
    assert lse[0] == pytest.approx(0.0, abs=1e-15)


def test_delta_identity():
    """sum_{jk} P dP = <dO_i, O_i>: the backward's softmax correction term
    equals the row dot product the GPU path computes from the stored output."""
    rng = np.random.default_rng(14)
    n, d, w1, w2 = 19, 5, 7, 4
    q, k, kp, v, vp, do = (rng.standard_normal((n, d)) for _ in range(6))
    o, _ = orc.forward(q, k, kp, v, vp, w1, w2, 0.45)
    for i in range(n):
        _, _, p, (j0, j1), (k0, k1) = orc.query_forward(q, k, kp, v, vp, i, w1, w2, 0.45)
        dp = np.einsum("d,jd,kd->jk", do[i], v[j0:j1], vp[k0:k1])
        assert (p * dp).sum() == pytest.approx(float(do[i] @ o[i]), abs=1e-13)


def _loss(arrs, do, w1, w2, scale):
    o, _ = orc.forward(*arrs, w1, w2, scale)
    return float(np.sum(o * do))


@pytest.mark.parametrize("n,d,w1,w2", [(11, 4, 4, 3), (9, 3, 2, 5), (8, 4, 20, 20)])
def test_backward_matches_central_finite_differences(n, d, w1, w2):
    """fp64 central differences of L = sum(O * dO) against the analytic backward."""
    rng = np.random.default_rng(15 + n)
    arrs = [rng.standard_normal((n, d)) for _ in range(5)]
    do = rng.standard_normal((n, d))
    scale = 0.6
    grads = orc.backward(*arrs, do, w1, w2, scale)
    eps = 1e-6
    for t in range(5):
        for _ in range(8):
            i, c = rng.integers(n), rng.integers(d)
            plus = [a.copy() for a in arrs]
            minus = [a.copy() for a in arrs]
            plus[t][i, c] += eps
            minus[t][i, c] -= eps
            fd = (_loss(plus, do, w1, w2, scale) - _loss(minus, do, w1, w2, scale)) / (2 * eps)
            assert grads[t][i, c] == pytest.approx(fd, abs=2e-8, rel=1e-6), (t, i, c)


def test_backward_matches_torch_autograd_of_algorithm1():
    """torch autograd (fp64, CPU) differentiating Algorithm 1's dense form pins the
    hand-written backward independently of its equations."""
    rng = np.random.default_rng(16)
    b, n, h, d, w1, w2 = 1, 14, 2, 4, 5, 3
    arrs = [rng.standard_normal((b, n, h, d)) for _ in range(5)]
    do = rng.standard_normal((b, n, h, d))
    scale = 0.5
    ts = [torch.tensor(a, requires_grad=True) for a in arrs]
    q, k, kp, v, vp = ts
    logits = scale * torch.einsum("btnh,bsnh,brnh->bntsr", q, k, kp)
    t_ = torch.arange(n)[:, None, None]
    s_ = torch.arange(n)[None, :, None]
    r_ = torch.arange(n)[None, None, :]
    mask = (s_ <= t_) & (s_ > t_ - w1) & (r_ <= t_) & (r_ > t_ - w2)
    logits = logits.masked_fill(~mask, float("-inf"))
    p = torch.softmax(logits.flatten(-2), dim=-1).view_as(logits)
    out = torch.einsum("bntsr,bsnh,brnh->btnh", p, v, vp)
    (out * torch.tensor(do)).sum().backward()
    grads = orc.backward_batched(*arrs, do, w1, w2, scale)
    for g, t in zip(grads, ts):
        np.testing.assert_allclose(g, t.grad.numpy(), rtol=0, atol=1e-12)


def test_query_subset_backward_completes_rows():
    """Restricting the backward to the queries that touch a row reproduces that
    row exactly (the sampled-row mode used by the full-size GPU parity tests)."""
    rng = np.random.default_rng(17)
    n, d, w1, w2 = 40, 4, 9, 5
    arrs = [rng.standard_normal((n, d)) for _ in range(6)]
    full = orc.backward(*arrs, w1, w2, 0.5)
    row = 17
    part_k = orc.backward(*arrs, w1, w2, 0.5, queries=range(row, min(n, row + w1)))
    part_kp = orc.backward(*arrs, w1, w2, 0.5, queries=range(row, min(n, row + w2)))
    part_q = orc.backward(*arrs, w1, w2, 0.5, queries=[row])
    np.testing.assert_allclose(part_q[0][row], full[0][row], atol=1e-14)
    for t in (1, 3):
        np.testing.assert_allclose(part_k[t][row], full[t][row], atol=1e-13)
    for t in (2, 4):
        np.testing.assert_allclose(part_kp[t][row], full[t][row], atol=1e-13)
