"""torch.autograd wrapper of the library's forward and backward entry points.

No arithmetic of its own: the forward is `simplicial_attn_fwd`, the backward
is `simplicial_attn_bwd` (Section 7's split backward: Delta, the key-side and
the query-side kernels), both called through the ctypes binding. Tensors are
[B, N, H, D] on one GPU, bf16 or fp32; when K, K', V, V' have fewer heads
(Hkv dividing H: grouped-query attention) the `_gqa` entry points are used.
The window lengths, the scale and the K' / V' bias constants are plain
Python numbers (not differentiated); non-zero bias constants use the `_biased`
entry points.
"""

import torch

from .binding import (simplicial_attn_bwd, simplicial_attn_bwd_biased, simplicial_attn_bwd_gqa,
                      simplicial_attn_fwd, simplicial_attn_fwd_biased, simplicial_attn_fwd_gqa)

__all__ = ["SimplicialAttnFunction", "simplicial_attention"]


class SimplicialAttnFunction(torch.autograd.Function):
    """(O, LSE) = 2-simplicial attention of (Q, K, K', V, V') with windows
    (w1, w2) and logit scale `scale`; LSE is returned without a gradient."""

    @staticmethod
    def forward(ctx, q, k, kp, v, vp, w1, w2, scale, kp_bias=0.0, vp_bias=0.0):
        q, k, kp, v, vp = (x.contiguous() for x in (q, k, kp, v, vp))
        biased = kp_bias != 0.0 or vp_bias != 0.0
        if biased:
            if k.shape[2] != q.shape[2]:
                raise ValueError("bias constants are supported with as many K-side heads as query heads")
            out, lse = simplicial_attn_fwd_biased(q, k, kp, v, vp, w1, w2, scale, kp_bias, vp_bias)
        else:
            fwd = simplicial_attn_fwd if k.shape[2] == q.shape[2] else simplicial_attn_fwd_gqa
            out, lse = fwd(q, k, kp, v, vp, w1, w2, scale)
        ctx.save_for_backward(q, k, kp, v, vp, out, lse)
        ctx.windows = (w1, w2, scale, kp_bias, vp_bias)
        ctx.mark_non_differentiable(lse)
        return out, lse

    @staticmethod
    @torch.autograd.function.once_differentiable
    def backward(ctx, dout, _dlse):
        q, k, kp, v, vp, out, lse = ctx.saved_tensors
        w1, w2, scale, kp_bias, vp_bias = ctx.windows
        if dout is None:
            dout = torch.zeros_like(out)
        dout = dout.to(out.dtype).contiguous()
        if kp_bias != 0.0 or vp_bias != 0.0:
            grads = simplicial_attn_bwd_biased(q, k, kp, v, vp, out, dout, lse, w1, w2, scale,
                                               kp_bias, vp_bias)
        else:
            bwd = simplicial_attn_bwd if k.shape[2] == q.shape[2] else simplicial_attn_bwd_gqa
            grads = bwd(q, k, kp, v, vp, out, dout, lse, w1, w2, scale)
        return (*grads, None, None, None, None, None)


def simplicial_attention(q, k, kp, v, vp, w1, w2, scale=None, kp_bias=0.0, vp_bias=0.0):
    """O = 2-simplicial attention(Q, K, K', V, V') with autograd support.

    q is [B, N, H, D]; k, kp, v, vp are [B, N, H, D] or, for grouped-query
    attention, [B, N, Hkv, D] with H a multiple of Hkv. `scale` defaults to
    1/sqrt(D). kp_bias / vp_bias are constants added to every element of K' /
    V' inside the kernels (0: none; non-zero needs Hkv == H).
    """
    if scale is None:
        scale = q.shape[-1] ** -0.5
    out, _ = SimplicialAttnFunction.apply(q, k, kp, v, vp, int(w1), int(w2), float(scale),
                                          float(kp_bias), float(vp_bias))
    return out
