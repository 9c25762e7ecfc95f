"""Pins of the determinant-form oracle (Section 5, Eqs. (det) and (logits)):
against numpy's determinant, the rotation invariance that motivates the form,
antisymmetry, torch autograd through torch.linalg.det, and finite differences."""

import numpy as np
import pytest
import torch

from oracle import determinant_oracle as dor


def _rand(shape, seed):
    return np.random.default_rng(seed).standard_normal(shape)


def _rotation(rng, proper=True):
    a = rng.standard_normal((3, 3))
    qm, r = np.linalg.qr(a)
    qm = qm * np.sign(np.diag(r))
    if (np.linalg.det(qm) > 0) != proper:
        qm[:, 0] = -qm[:, 0]
    return qm


def test_levi_civita_values():
    e = dor.levi_civita()
    assert e[0, 1, 2] == 1 and e[1, 2, 0] == 1 and e[2, 0, 1] == 1
    assert e[0, 2, 1] == -1 and e[2, 1, 0] == -1 and e[1, 0, 2] == -1
    assert np.count_nonzero(e) == 6


def test_hand_worked_determinant():
    # unit basis vectors: det = +1 for (e0, e1, e2), -1 after swapping two rows
    q = np.array([1.0, 0, 0, 2.0, 0, 0])
    k = np.array([[0, 1.0, 0, 0, 3.0, 0]])
    kp = np.array([[0, 0, 1.0, 0, 0, 5.0]])
    assert dor.det_logits(q, k, kp, 1.0)[0, 0] == pytest.approx(1.0 + 30.0)
    assert dor.det_logits(q, kp, k, 1.0)[0, 0] == pytest.approx(-31.0)


@pytest.mark.parametrize("d", [3, 7, 16, 64])
def test_logits_match_numpy_det(d):
    q, k, kp = _rand(d, 1), _rand((4, d), 2), _rand((5, d), 3)
    got = dor.det_logits(q, k, kp, 0.3)
    p = d // 3
    for j in range(4):
        for kk in range(5):
            ref = sum(np.linalg.det(np.stack([q[3 * l:3 * l + 3], k[j, 3 * l:3 * l + 3],
                                              kp[kk, 3 * l:3 * l + 3]])) for l in range(p))
            assert got[j, kk] == pytest.approx(0.3 * ref, rel=1e-12, abs=1e-12)


def test_rotation_invariance_and_reflection_sign():
    rng = np.random.default_rng(4)
    d, n = 12, 9
    q, k, kp, v, vp = (_rand((n, d), s) for s in range(10, 15))
    rots = [_rotation(rng) for _ in range(d // 3)]
    refl = [_rotation(rng, proper=False) for _ in range(d // 3)]

    def apply(x, mats):
        xc = dor.chunks(x).copy()
        for l, r in enumerate(mats):
            xc[..., l, :] = xc[..., l, :] @ r.T
        return xc.reshape(x.shape)

    a0 = dor.det_logits(q[5], k, kp, 1.0)
    a_rot = dor.det_logits(apply(q, rots)[5], apply(k, rots), apply(kp, rots), 1.0)
    a_ref = dor.det_logits(apply(q, refl)[5], apply(k, refl), apply(kp, refl), 1.0)
    np.testing.assert_allclose(a_rot, a0, rtol=1e-10, atol=1e-10)
    np.testing.assert_allclose(a_ref, -a0, rtol=1e-10, atol=1e-10)
    # the whole forward is invariant under rotations of Q, K, K' (V, V' untouched)
    o0, l0 = dor.forward(q, k, kp, v, vp, 4, 3, 0.5)
    o1, l1 = dor.forward(apply(q, rots), apply(k, rots), apply(kp, rots), v, vp, 4, 3, 0.5)
    np.testing.assert_allclose(o1, o0, rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(l1, l0, rtol=1e-10, atol=1e-12)


def test_trailing_components_are_inert():
    d, n = 8, 7  # two chunks, components 6 and 7 unused
    q, k, kp, v, vp, do = (_rand((n, d), s) for s in range(20, 26))
    o0, l0 = dor.forward(q, k, kp, v, vp, 5, 3, 0.4)
    q2, k2, kp2 = q.copy(), k.copy(), kp.copy()
    q2[:, 6:] += 3.0
    k2[:, 6:] -= 1.0
    kp2[:, 7] *= 5.0
    o1, l1 = dor.forward(q2, k2, kp2, v, vp, 5, 3, 0.4)
    np.testing.assert_array_equal(o1, o0)
    np.testing.assert_array_equal(l1, l0)
    g = dor.backward(q, k, kp, v, vp, do, 5, 3, 0.4)
    for t in range(3):
        assert np.all(g[t][:, 6:] == 0)


def _torch_forward(q, k, kp, v, vp, w1, w2, scale):
    """Dense masked reference through torch.linalg.det (Eq. (logits) with each
    3 x 3 determinant taken by the library), windows of Section 6."""
    n, d = q.shape
    p = d // 3
    qc, kc, kpc = (x[:, : 3 * p].reshape(n, p, 3) for x in (q, k, kp))
    m = torch.stack([qc[:, None, None].expand(n, n, n, p, 3), kc[None, :, None].expand(n, n, n, p, 3),
                     kpc[None, None, :].expand(n, n, n, p, 3)], dim=-2)  # [i, j, k, l, 3 rows, 3]
    a = scale * torch.linalg.det(m).sum(-1)
    idx = torch.arange(n)
    dj = idx[:, None] - idx[None, :]
    mj = (dj >= 0) & (dj < w1)
    mk = (dj >= 0) & (dj < w2)
    mask = mj[:, :, None] & mk[:, None, :]
    a = a.masked_fill(~mask, float("-inf"))
    pr = torch.softmax(a.reshape(n, -1), dim=-1).reshape(n, n, n)
    return torch.einsum("ijk,jd,kd->id", pr, v, vp)


def test_backward_matches_torch_autograd_through_linalg_det():
    n, d, w1, w2, scale = 6, 7, 4, 3, 0.6
    arrs = [_rand((n, d), s) for s in range(30, 36)]
    ts = [torch.tensor(a, requires_grad=True) for a in arrs[:5]]
    out = _torch_forward(*ts, w1, w2, scale)
    o_ref, _ = dor.forward(*arrs[:5], w1, w2, scale)
    np.testing.assert_allclose(o_ref, out.detach().numpy(), rtol=1e-10, atol=1e-12)
    (out * torch.tensor(arrs[5])).sum().backward()
    got = dor.backward(*arrs, w1, w2, scale)
    for name, g, t in zip(("dq", "dk", "dkp", "dv", "dvp"), got, ts):
        np.testing.assert_allclose(g, t.grad.numpy(), rtol=1e-9, atol=1e-11, err_msg=name)


def test_backward_matches_central_finite_differences():
    n, d, w1, w2, scale = 5, 6, 3, 2, 0.8
    arrs = [_rand((n, d), s) for s in range(40, 46)]
    g = dor.backward(*arrs, w1, w2, scale)
    eps = 1e-6
    rng = np.random.default_rng(7)
    for t in range(5):
        for _ in range(6):
            r, c = int(rng.integers(n)), int(rng.integers(d))
            plus = [a.copy() for a in arrs[:5]]
            minus = [a.copy() for a in arrs[:5]]
            plus[t][r, c] += eps
            minus[t][r, c] -= eps
            fp = float(np.sum(dor.forward(*plus, w1, w2, scale)[0] * arrs[5]))
            fm = float(np.sum(dor.forward(*minus, w1, w2, scale)[0] * arrs[5]))
            num = (fp - fm) / (2 * eps)
            assert abs(num - g[t][r, c]) <= 1e-6 * max(1.0, abs(num)), (t, r, c, num, g[t][r, c])


def test_scale_one_is_the_papers_unscaled_form():
    """Eq. (logits) carries no scale factor: at scale = 1 the oracle's logits are
    the plain sum of chunk determinants, and its forward is the joint softmax of
    exactly those logits over the windows (dense brute force with numpy's det)."""
    n, d, w1, w2 = 7, 9, 4, 3
    q, k, kp, v, vp = (_rand((n, d), s) for s in range(50, 55))
    o, lse = dor.forward(q, k, kp, v, vp, w1, w2, 1.0)
    for i in range(n):
        js = range(max(0, i - w1 + 1), i + 1)
        ks = range(max(0, i - w2 + 1), i + 1)
        a = np.array([[sum(np.linalg.det(np.stack([q[i, 3 * l:3 * l + 3], k[j, 3 * l:3 * l + 3],
                                                    kp[kk, 3 * l:3 * l + 3]])) for l in range(d // 3))
                       for kk in ks] for j in js])
        assert np.allclose(dor.det_logits(q[i], k[js[0]:i + 1], kp[ks[0]:i + 1], 1.0), a,
                           rtol=1e-12, atol=1e-12)
        p = np.exp(a - a.max())
        z = p.sum()
        ref_o = np.einsum("jk,jd,kd->d", p / z, v[js[0]:i + 1], vp[ks[0]:i + 1])
        np.testing.assert_allclose(o[i], ref_o, rtol=1e-11, atol=1e-12)
        assert lse[i] == pytest.approx(a.max() + np.log(z), rel=1e-12, abs=1e-12)
