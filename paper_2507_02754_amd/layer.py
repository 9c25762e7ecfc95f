"""The 2-simplicial attention layer and a small interleaved stack around it.

Section 4 builds the layer from the input X ([B, N, d_model]) with the usual
projections Q = X W_Q, K = X W_K, V = X W_V plus two more, K' = X W_K' and
V' = X W_V'; the attention is the windowed trilinear attention of the library
(`simplicial_attention`: the HIP kernels, autograd through the library's
backward), followed by an output projection. The K' / V' bias constants of the
paper's Appendix B kernels are layer options passed to the kernels. With fewer
K-side heads than query heads (grouped-query attention, Section 6) W_K, W_K',
W_V, W_V' project to `kv_heads` heads.

Section 8 interleaves such layers with ordinary attention: every fourth layer
is 2-simplicial. `InterleavedStack` does that with pre-norm residual blocks
(RMSNorm, attention, SiLU MLP); the other layers use causal dot-product
attention. The projections, norms and MLPs are plain torch modules (library
GEMMs); only the 2-simplicial attention runs in this package's kernels. The
paper's mixture-of-experts feed-forward layers and its training data are not
part of this package.
"""

import torch
import torch.nn.functional as F
from torch import nn

from .autograd import simplicial_attention

__all__ = ["SimplicialAttention", "DotProductAttention", "Block", "InterleavedStack"]


class SimplicialAttention(nn.Module):
    """2-simplicial attention layer (Section 4) over sliding windows (w1, w2).

    x [B, N, d_model] -> [B, N, d_model]. Attention runs in `attn_dtype`
    (bf16: the MFMA kernels for head_dim 64/128 and w2 <= 64; fp32: the plain
    kernels); the projections run in the dtype of the module's parameters.
    """

    def __init__(self, d_model, n_heads, head_dim, w1, w2, kv_heads=None, kp_bias=0.0, vp_bias=0.0,
                 scale=None, attn_dtype=torch.bfloat16, device=None, dtype=None):
        super().__init__()
        kv_heads = kv_heads or n_heads
        if n_heads % kv_heads:
            raise ValueError("n_heads must be a multiple of kv_heads")
        if (kp_bias or vp_bias) and kv_heads != n_heads:
            raise ValueError("bias constants need as many K-side heads as query heads")
        fk = dict(device=device, dtype=dtype, bias=False)
        self.n_heads, self.kv_heads, self.head_dim = n_heads, kv_heads, head_dim
        self.w1, self.w2 = int(w1), int(w2)
        self.kp_bias, self.vp_bias = float(kp_bias), float(vp_bias)
        self.scale = head_dim ** -0.5 if scale is None else float(scale)
        self.attn_dtype = attn_dtype
        self.wq = nn.Linear(d_model, n_heads * head_dim, **fk)
        self.wk = nn.Linear(d_model, kv_heads * head_dim, **fk)
        self.wv = nn.Linear(d_model, kv_heads * head_dim, **fk)
        self.wkp = nn.Linear(d_model, kv_heads * head_dim, **fk)  # W_K'
        self.wvp = nn.Linear(d_model, kv_heads * head_dim, **fk)  # W_V'
        self.wo = nn.Linear(n_heads * head_dim, d_model, **fk)

    def forward(self, x):
        b, n, _ = x.shape
        h, hk, d = self.n_heads, self.kv_heads, self.head_dim

        def heads(t, nh):
            return t.view(b, n, nh, d).to(self.attn_dtype).contiguous()

        q = heads(self.wq(x), h)
        k, v = heads(self.wk(x), hk), heads(self.wv(x), hk)
        kp, vp = heads(self.wkp(x), hk), heads(self.wvp(x), hk)
        o = simplicial_attention(q, k, kp, v, vp, self.w1, self.w2, self.scale, self.kp_bias, self.vp_bias)
        return self.wo(o.reshape(b, n, h * d).to(x.dtype))


class DotProductAttention(nn.Module):
    """Causal dot-product attention (the layers between the 2-simplicial ones).
    The attention itself is computed in fp32."""

    def __init__(self, d_model, n_heads, head_dim, device=None, dtype=None):
        super().__init__()
        fk = dict(device=device, dtype=dtype, bias=False)
        self.n_heads, self.head_dim = n_heads, head_dim
        self.wqkv = nn.Linear(d_model, 3 * n_heads * head_dim, **fk)
        self.wo = nn.Linear(n_heads * head_dim, d_model, **fk)

    def forward(self, x):
        b, n, _ = x.shape
        q, k, v = self.wqkv(x).float().view(b, n, 3, self.n_heads, self.head_dim).permute(2, 0, 3, 1, 4)
        o = F.scaled_dot_product_attention(q.contiguous(), k.contiguous(), v.contiguous(), is_causal=True)
        return self.wo(o.transpose(1, 2).reshape(b, n, -1).to(x.dtype))


class RMSNorm(nn.Module):
    def __init__(self, d, eps=1e-6, device=None, dtype=None):
        super().__init__()
        self.eps = eps
        self.weight = nn.Parameter(torch.ones(d, device=device, dtype=dtype))

    def forward(self, x):
        xf = x.float()
        return (xf * torch.rsqrt(xf.pow(2).mean(-1, keepdim=True) + self.eps)).to(x.dtype) * self.weight


class Block(nn.Module):
    """Pre-norm residual block: x + attn(norm(x)), then + mlp(norm(x))."""

    def __init__(self, attn, d_model, d_ff, device=None, dtype=None):
        super().__init__()
        fk = dict(device=device, dtype=dtype)
        self.norm1, self.norm2 = RMSNorm(d_model, **fk), RMSNorm(d_model, **fk)
        self.attn = attn
        self.up = nn.Linear(d_model, d_ff, bias=False, **fk)
        self.down = nn.Linear(d_ff, d_model, bias=False, **fk)

    def forward(self, x):
        x = x + self.attn(self.norm1(x))
        return x + self.down(F.silu(self.up(self.norm2(x))))


class InterleavedStack(nn.Module):
    """Token embedding, `n_layers` blocks in which layer l (0-based) is
    2-simplicial when (l + 1) % every == 0 (every fourth layer for every = 4,
    as in Section 8) and causal dot-product attention otherwise, a final norm
    and an output head. forward(tokens [B, N] int64) -> logits [B, N, vocab]."""

    def __init__(self, vocab, d_model, n_layers, n_heads, head_dim, w1, w2, every=4, d_ff=None,
                 kv_heads=None, kp_bias=0.0, vp_bias=0.0, attn_dtype=torch.bfloat16, device=None,
                 dtype=None):
        super().__init__()
        fk = dict(device=device, dtype=dtype)
        d_ff = d_ff or 4 * d_model
        self.embed = nn.Embedding(vocab, d_model, **fk)
        layers = []
        for l in range(n_layers):
            if (l + 1) % every == 0:
                attn = SimplicialAttention(d_model, n_heads, head_dim, w1, w2, kv_heads, kp_bias, vp_bias,
                                           attn_dtype=attn_dtype, **fk)
            else:
                attn = DotProductAttention(d_model, n_heads, head_dim, **fk)
            layers.append(Block(attn, d_model, d_ff, **fk))
        self.layers = nn.ModuleList(layers)
        self.norm = RMSNorm(d_model, **fk)
        self.head = nn.Linear(d_model, vocab, bias=False, **fk)

    def simplicial_layers(self):
        return [i for i, blk in enumerate(self.layers) if isinstance(blk.attn, SimplicialAttention)]

    def forward(self, tokens):
        x = self.embed(tokens)
        for blk in self.layers:
            x = blk(x)
        return self.head(self.norm(x))

    def loss(self, tokens):
        """Next-token cross-entropy of the tokens (mean over positions)."""
        logits = self(tokens[:, :-1])
        return F.cross_entropy(logits.float().reshape(-1, logits.shape[-1]), tokens[:, 1:].reshape(-1))
