"""Seeded synthetic workloads for 2-simplicial sliding-window attention.

This module only draws random inputs and names workload shapes; it holds none
of the attention arithmetic. Both the HIP path's tests/benchmark and the CPU
oracle consume the tensors it returns (the oracle after promotion to float64),
so it is the one piece they share.

Recipe (identical for every workload): one CPU ``torch.Generator`` seeded with
the workload's seed; draw order Q, K, K', V, V', dO, each an fp32 standard
normal of shape [B, N, H, D]; then the workload's transform; then a cast to the
workload dtype (round-to-nearest-even for bf16). The paper trains on text
corpora that are not available here; these shapes stand in for its training
activations (head dim 128, windows (w1, w2) = (512, 32) as chosen in Section 6).
"""

from dataclasses import dataclass, field

import torch

__all__ = ["Workload", "WORKLOADS", "make_inputs", "draw"]


@dataclass(frozen=True)
class Workload:
    name: str
    B: int
    H: int
    N: int
    D: int
    w1: int
    w2: int
    dtype: str  # "fp32" or "bf16"
    seed: int
    backward: bool = True
    transform: str = "none"  # "none" | "l2norm_qk" | "scale_half"
    note: str = field(default="", compare=False)

    @property
    def scale(self) -> float:
        return self.D ** -0.5

    @property
    def torch_dtype(self):
        return torch.float32 if self.dtype == "fp32" else torch.bfloat16

    def shape(self):
        return (self.B, self.N, self.H, self.D)


WORKLOADS = {
    w.name: w
    for w in [
        Workload("tiny_fp32", 1, 1, 128, 64, 16, 8, "fp32", seed=1,
                 note="fp32 forward+backward, iid N(0,1)"),
        Workload("fwd_bf16_n4k", 1, 8, 4096, 128, 512, 32, "bf16", seed=2, backward=False,
                 note="bf16 forward only, iid N(0,1)"),
        Workload("fb_bf16_n8k", 2, 8, 8192, 128, 512, 32, "bf16", seed=3,
                 note="bf16 forward+backward, iid N(0,1)"),
        Workload("long_bf16_n32k", 1, 16, 32768, 128, 512, 32, "bf16", seed=4,
                 transform="l2norm_qk",
                 note="bf16 forward+backward; Q and K rows L2-normalised then scaled by sqrt(D)"),
        Workload("wide_bf16_n16k", 4, 16, 16384, 128, 1024, 64, "bf16", seed=5,
                 transform="scale_half",
                 note="bf16 forward+backward; inputs iid N(0, 0.5^2), dO iid N(0,1)"),
    ]
}


def draw(shape, seed, dtype=torch.bfloat16, transform="none"):
    """Return (q, k, kp, v, vp, do) CPU tensors of `shape` = (B, N, H, D).

    Drawn in fp32 in the fixed order above, transformed, then cast to `dtype`.
    """
    g = torch.Generator(device="cpu").manual_seed(int(seed))
    ts = [torch.randn(shape, generator=g, dtype=torch.float32) for _ in range(6)]
    q, k, kp, v, vp, do = ts
    d = shape[-1]
    if transform == "l2norm_qk":
        q = q / q.norm(dim=-1, keepdim=True) * d ** 0.5
        k = k / k.norm(dim=-1, keepdim=True) * d ** 0.5
    elif transform == "scale_half":
        q, k, kp, v, vp = (x * 0.5 for x in (q, k, kp, v, vp))
    elif transform != "none":
        raise ValueError(f"unknown transform {transform!r}")
    return tuple(x.to(dtype).contiguous() for x in (q, k, kp, v, vp, do))


def make_inputs(w: Workload):
    """Inputs of a named workload: (q, k, kp, v, vp, do) as CPU tensors in its dtype."""
    return draw(w.shape(), w.seed, w.torch_dtype, w.transform)
