"""GPU tests of the K' / V' bias constants (the _biased entry points) and of
the layer built around the kernels, against the oracle."""

import copy

import numpy as np
import pytest
import torch

import parity as P
from paper_2507_02754_amd import (InterleavedStack, SimplicialAttention, load_library,
                                  simplicial_attn_bwd, simplicial_attn_bwd_biased,
                                  simplicial_attn_fwd, simplicial_attn_fwd_biased,
                                  simplicial_attn_path_name)
from paper_2507_02754_amd.workloads import draw

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    load_library()


def _announce(label):
    print(f"\n[layer] {label}", flush=True)


BIASED = [
    # (B, H, N, D, w1, w2, dtype, kp_bias, vp_bias)
    (1, 2, 300, 128, 64, 32, "bf16", 0.75, -0.5),   # MFMA path, several tiles
    (1, 1, 129, 128, 33, 7, "bf16", -1.0, 0.5),     # rows outside the w2 window stay excluded
    (2, 1, 200, 64, 40, 32, "bf16", 0.5, 0.5),      # head_dim 64
    (1, 1, 333, 128, 96, 64, "bf16", 0.3, -0.7),    # w2 = 64 (two wavefronts per query)
    (1, 2, 100, 64, 7, 5, "fp32", 1.5, -0.25),      # plain kernels
]


@pytest.mark.parametrize("shape", BIASED, ids=[str(s) for s in BIASED])
def test_biased_entry_points_match_oracle_on_shifted_inputs(shape):
    """The _biased pair equals the oracle run on K' + kp_bias and V' + vp_bias
    (the definition of the constants), every element; gradients are those of
    the given K', V'."""
    b, h, n, d, w1, w2, dt, kb, vb = shape
    _announce(f"biased {shape} fwd={simplicial_attn_path_name(0, b, n, h, d, w1, w2, 1 if dt == 'bf16' else 0)}")
    inputs = draw((b, n, h, d), seed=60 + n, dtype=torch.float32 if dt == "fp32" else torch.bfloat16)
    scale = d ** -0.5
    x = [t.cuda() for t in inputs]
    o, lse = simplicial_attn_fwd_biased(*x[:5], w1, w2, scale, kb, vb)
    grads = simplicial_attn_bwd_biased(*x[:5], o, x[5], lse, w1, w2, scale, kb, vb)
    torch.cuda.synchronize()
    shifted = list(inputs)
    shifted[2] = inputs[2].double() + kb
    shifted[4] = inputs[4].double() + vb
    o_ref, lse_ref, g_ref = P.full_oracle([t.double() for t in shifted], w1, w2, scale)
    P.check_forward(P.to64(o), P.to64(lse), o_ref, lse_ref, dt, f"biased {shape}")
    P.check_grads([P.to64(g) for g in grads], g_ref, dt, f"biased {shape}")


def test_zero_bias_constants_give_the_plain_results_bitwise():
    b, h, n, d, w1, w2 = 1, 2, 300, 128, 64, 32
    _announce("zero bias constants")
    x = [t.cuda() for t in draw((b, n, h, d), seed=61)]
    o1, l1 = simplicial_attn_fwd(*x[:5], w1, w2)
    o2, l2 = simplicial_attn_fwd_biased(*x[:5], w1, w2, None, 0.0, 0.0)
    g1 = simplicial_attn_bwd(*x[:5], o1, x[5], l1, w1, w2)
    g2 = simplicial_attn_bwd_biased(*x[:5], o1, x[5], l1, w1, w2, None, 0.0, 0.0)
    torch.cuda.synchronize()
    assert torch.equal(o1, o2) and torch.equal(l1, l2)
    for a, c in zip(g1, g2):
        assert torch.equal(a, c)


def _reference_layer(layer):
    """float64 CPU copy of a SimplicialAttention layer whose attention is the
    oracle (same weights)."""
    ref = copy.deepcopy(layer).to("cpu", torch.float64)

    def forward(x):
        b, n, _ = x.shape
        h, hk, d = ref.n_heads, ref.kv_heads, ref.head_dim
        q = ref.wq(x).view(b, n, h, d)
        k, v = ref.wk(x).view(b, n, hk, d), ref.wv(x).view(b, n, hk, d)
        kp, vp = ref.wkp(x).view(b, n, hk, d), ref.wvp(x).view(b, n, hk, d)
        g = h // hk
        k, v, kp, vp = (t.repeat_interleave(g, dim=2) for t in (k, v, kp, vp))
        o = P.OracleAttention.apply(q, k, kp, v, vp, ref.w1, ref.w2, ref.scale, ref.kp_bias, ref.vp_bias)
        return ref.wo(o.reshape(b, n, h * d))

    return ref, forward


@pytest.mark.parametrize("kv_heads,kb,vb", [(2, 0.5, -0.3), (1, 0.0, 0.0)], ids=["mha_biased", "gqa"])
def test_layer_matches_float64_reference(kv_heads, kb, vb):
    """Output, input gradient and every projection's weight gradient of the
    layer (fp32 projections, bf16 attention on the MFMA kernels) against the
    same layer in float64 on the CPU with the oracle as its attention."""
    torch.manual_seed(5)
    d_model, h, d, w1, w2, b, n = 256, 2, 128, 48, 32, 2, 200
    _announce(f"layer kv_heads={kv_heads} biases=({kb}, {vb})")
    layer = SimplicialAttention(d_model, h, d, w1, w2, kv_heads=kv_heads, kp_bias=kb, vp_bias=vb,
                                device="cuda", dtype=torch.float32)
    with torch.no_grad():
        for p_ in layer.parameters():
            p_.normal_(0.0, d_model ** -0.5)
    x = torch.randn(b, n, d_model, device="cuda", requires_grad=True)
    dy = torch.randn(b, n, d_model)
    y = layer(x)
    (y * dy.cuda()).sum().backward()
    ref, ref_forward = _reference_layer(layer)
    xr = x.detach().cpu().double().requires_grad_(True)
    yr = ref_forward(xr)
    (yr * dy.double()).sum().backward()
    P.check_forward(P.to64(y), np.zeros(1), yr.detach().numpy(), np.zeros(1), "bf16", "layer output")
    names = ["dx"] + [nm for nm, _ in layer.named_parameters()]
    got = [P.to64(x.grad)] + [P.to64(p_.grad) for _, p_ in layer.named_parameters()]
    want = [xr.grad.numpy()] + [p_.grad.numpy() for _, p_ in ref.named_parameters()]
    for nm, g_, r_ in zip(names, got, want):
        P.check_grads([g_], [r_], "bf16", f"layer {nm}")


def test_interleaved_stack_training_steps():
    """Four blocks (layer 3 2-simplicial, with bias constants) on synthetic
    tokens: AdamW steps on one batch lower the loss, and every parameter of the
    2-simplicial layer receives a finite, non-zero gradient."""
    torch.manual_seed(3)
    vocab, b, n = 512, 2, 256
    model = InterleavedStack(vocab=vocab, d_model=256, n_layers=4, n_heads=2, head_dim=128, w1=64, w2=32,
                             kp_bias=0.25, vp_bias=0.5, device="cuda", dtype=torch.float32)
    assert model.simplicial_layers() == [3]
    tokens = torch.randint(0, vocab, (b, n + 1), device="cuda")
    opt = torch.optim.AdamW(model.parameters(), lr=3e-3, weight_decay=0.0125)
    losses = []
    for step in range(6):
        opt.zero_grad(set_to_none=True)
        loss = model.loss(tokens)
        loss.backward()
        if step == 0:
            attn = model.layers[3].attn
            for nm, p_ in attn.named_parameters():
                assert p_.grad is not None and torch.isfinite(p_.grad).all(), nm
                assert p_.grad.abs().max().item() > 0, nm
        opt.step()
        losses.append(loss.item())
    _announce(f"losses {[round(v, 4) for v in losses]}")
    assert all(np.isfinite(losses))
    assert losses[-1] < losses[0] - 0.5
