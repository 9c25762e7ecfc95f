"""Host-side structure of the 2-simplicial layer and the interleaved stack
(no kernel calls)."""

import pytest
import torch

from paper_2507_02754_amd import InterleavedStack, SimplicialAttention


def test_every_fourth_layer_is_two_simplicial():
    m = InterleavedStack(vocab=32, d_model=64, n_layers=8, n_heads=2, head_dim=64, w1=16, w2=8)
    assert m.simplicial_layers() == [3, 7]
    m = InterleavedStack(vocab=32, d_model=64, n_layers=6, n_heads=2, head_dim=64, w1=16, w2=8, every=2)
    assert m.simplicial_layers() == [1, 3, 5]


def test_projection_shapes_and_options():
    a = SimplicialAttention(d_model=96, n_heads=4, head_dim=64, w1=32, w2=16, kv_heads=2)
    assert a.wq.weight.shape == (4 * 64, 96)
    for lin in (a.wk, a.wv, a.wkp, a.wvp):
        assert lin.weight.shape == (2 * 64, 96)
    assert a.wo.weight.shape == (96, 4 * 64)
    assert a.scale == pytest.approx(64 ** -0.5)
    with pytest.raises(ValueError):
        SimplicialAttention(96, 4, 64, 32, 16, kv_heads=3)
    with pytest.raises(ValueError):
        SimplicialAttention(96, 4, 64, 32, 16, kv_heads=2, kp_bias=1.0)
