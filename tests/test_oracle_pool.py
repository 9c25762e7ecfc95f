"""The process-pool runner of the oracle (used by the full-size GPU parity
tests) returns exactly what direct oracle calls return."""

import numpy as np
import torch

import oracle as orc
import oracle_pool
from paper_2507_02754_amd.workloads import draw


def test_pooled_oracle_equals_direct_calls():
    n, d, w1, w2, scale = 300, 32, 40, 9, 0.2
    arrs = [x[0, :, 0].to(torch.float64).numpy() for x in draw((1, n, 1, d), seed=21)]
    queries = list(range(3, n, 2))
    o, lse = oracle_pool.forward(*arrs[:5], w1, w2, scale, queries)
    o_ref, lse_ref = orc.forward(*arrs[:5], w1, w2, scale, queries=queries)
    assert np.array_equal(o, o_ref[queries]) and np.array_equal(lse, lse_ref[queries])
    rows = [[0, 7, 299], [0, 100, 260], [1, 290], [5, 299], [0, 42]]
    got = oracle_pool.backward(*arrs, w1, w2, scale, range(n), rows)
    ref = orc.backward(*arrs, w1, w2, scale)
    for g, r, sel in zip(got, ref, rows):
        np.testing.assert_allclose(g, r[sel], rtol=1e-12, atol=1e-14)
    from oracle import determinant_oracle as dor
    got = oracle_pool.backward(*arrs, w1, w2, scale, range(n), rows, module="oracle.determinant_oracle")
    ref = dor.backward(*arrs, w1, w2, scale)
    for g, r, sel in zip(got, ref, rows):
        np.testing.assert_allclose(g, r[sel], rtol=1e-12, atol=1e-14)
    oracle_pool.shutdown()
