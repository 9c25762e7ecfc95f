"""Pins of the grouped-query composition of the oracle (tests/parity.py):
query head h reads K-side head h // (H // Hkv) (Section 6's shared K/V heads),
and the K-side gradients are the sums over each group's query heads. Checked
against central finite differences of the composed forward (CPU, fp64)."""

import numpy as np
import torch

import oracle as orc
import parity as P


def _inputs(b, h, hkv, n, d, seed):
    g = torch.Generator().manual_seed(seed)
    q = torch.randn((b, n, h, d), generator=g, dtype=torch.float64)
    kv = [torch.randn((b, n, hkv, d), generator=g, dtype=torch.float64) for _ in range(4)]
    do = torch.randn((b, n, h, d), generator=g, dtype=torch.float64)
    return q, kv, do


def _loss(q, kv, do, w1, w2, scale):
    res = P.gqa_oracle_forward(q, kv, w1, w2, scale)
    return sum(float(np.sum(o * do[b, :, h, :].numpy())) for (b, h), (o, _) in res.items())


def test_gqa_forward_reads_the_group_head():
    q, kv, _ = _inputs(1, 6, 2, 9, 4, 1)
    res = P.gqa_oracle_forward(q, kv, 4, 3, 0.5)
    for h in range(6):
        o, lse = orc.forward(q[0, :, h].numpy(), *(x[0, :, h // 3].numpy() for x in kv), 4, 3, 0.5)
        assert np.array_equal(res[(0, h)][0], o) and np.array_equal(res[(0, h)][1], lse)
        # a different K-side head gives a different result
        o2, _ = orc.forward(q[0, :, h].numpy(), *(x[0, :, 1 - h // 3].numpy() for x in kv), 4, 3, 0.5)
        assert not np.allclose(o, o2)


def test_gqa_backward_matches_finite_differences():
    b, h, hkv, n, d, w1, w2, scale = 2, 4, 2, 6, 3, 3, 2, 0.7
    q, kv, do = _inputs(b, h, hkv, n, d, 2)
    dq, dkv = P.gqa_oracle_backward(q, kv, do, w1, w2, scale)
    eps = 1e-6
    rng = np.random.default_rng(0)
    # every K-side tensor, sampled elements of both K-side heads, and dQ
    for t in range(4):
        for _ in range(8):
            idx = (int(rng.integers(b)), int(rng.integers(n)), int(rng.integers(hkv)), int(rng.integers(d)))
            plus = [x.clone() for x in kv]
            minus = [x.clone() for x in kv]
            plus[t][idx] += eps
            minus[t][idx] -= eps
            num = (_loss(q, plus, do, w1, w2, scale) - _loss(q, minus, do, w1, w2, scale)) / (2 * eps)
            assert abs(num - dkv[t][idx]) <= 1e-6 * max(1.0, abs(num)), (t, idx, num, dkv[t][idx])
    for _ in range(8):
        idx = (int(rng.integers(b)), int(rng.integers(n)), int(rng.integers(h)), int(rng.integers(d)))
        qp, qm = q.clone(), q.clone()
        qp[idx] += eps
        qm[idx] -= eps
        num = (_loss(qp, kv, do, w1, w2, scale) - _loss(qm, kv, do, w1, w2, scale)) / (2 * eps)
        assert abs(num - dq[idx]) <= 1e-6 * max(1.0, abs(num)), (idx, num, dq[idx])


def test_gqa_backward_with_one_query_head_per_group_is_the_plain_backward():
    q, kv, do = _inputs(1, 3, 3, 7, 4, 3)
    dq, dkv = P.gqa_oracle_backward(q, kv, do, 5, 2, 0.5)
    for h in range(3):
        g = orc.backward(q[0, :, h].numpy(), *(x[0, :, h].numpy() for x in kv), do[0, :, h].numpy(),
                         5, 2, 0.5)
        assert np.array_equal(dq[0, :, h], g[0])
        for t in range(4):
            assert np.array_equal(dkv[t][0, :, h], g[1 + t])
