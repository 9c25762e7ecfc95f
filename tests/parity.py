"""Shared helpers of the GPU parity tests: run the HIP path through the C ABI,
run the oracle on the same seeded inputs (whole tensors or sampled rows), and
measure the differences.

Tolerances (the bar each parity test asserts), with the arithmetic behind them:

* fp32 data: max |x - ref| / max |ref| <= 1e-5 per tensor. The GPU computes in
  fp32 with fp32 products; with D <= 128 terms per logit and <= w1*w2 pairs per
  query, the relative rounding error stays near 1e-6.
* bf16 data, forward: max |O - O_ref| <= 2e-2 (absolute) and, because |O| is
  itself only ~1e-2 at the benchmark shapes, also the normwise
  ||O - O_ref|| / ||O_ref|| <= 1e-2. Where max |O_ref| exceeds 1 (a query
  seeing a single pair has O_i = v_i o v'_i; constants added to V' scale all
  of O) the absolute bar is 2e-2 * max |O_ref|: bf16 resolves |x| in [8, 16)
  only to 0.0625, so no bf16 result can meet a fixed 2e-2 there. The kernels round the modulated query
  q_i o k'_k, the probabilities P and the output to bf16 (unit roundoff
  2^-9 = 2e-3 each), which gives a normwise error of a few 1e-3.
  LSE (fp32 output): |LSE - ref| <= 2e-2; the bf16 rounding of the modulated
  query perturbs each logit by ~2^-9 |logit|.
* bf16 data, backward: per gradient max |g - ref| / max |ref| <= 5e-2 and
  normwise <= 2e-2, each gradient on its own scale (P, dS and the modulated
  operands are rounded to bf16 before each matrix product, and the result is
  rounded to bf16). Gradients that vanish in exact arithmetic (dQ, dK, dK' with
  unit windows or unit values) have no scale of their own; the tests of those
  identities bound them explicitly instead of calling check_grads on them.
"""

import json
import os

import numpy as np
import torch

import oracle as orc
from paper_2507_02754_amd import (simplicial_attn_bwd, simplicial_attn_bwd_fused, simplicial_attn_bwd_fused_reduce,
                                  simplicial_attn_bwd_fused_workspace_size, simplicial_attn_bwd_preprocess,
                                  simplicial_attn_fwd)

TOL = {
    "fp32": dict(o_maxrel=1e-5, lse_abs=1e-5, g_maxrel=1e-5, o_norm=1e-5, g_norm=1e-5),
    "bf16": dict(o_abs=2e-2, o_norm=1e-2, lse_abs=2e-2, g_maxrel=5e-2, g_norm=2e-2),
}

GRAD_NAMES = ("dq", "dk", "dkp", "dv", "dvp")


def _names_for(n):
    return GRAD_NAMES[len(GRAD_NAMES) - n:]


def to64(t):
    return t.detach().to("cpu", torch.float64).numpy()


def gpu_forward(inputs, w1, w2, scale, device="cuda"):
    q, k, kp, v, vp = (x.to(device) for x in inputs[:5])
    out, lse = simplicial_attn_fwd(q, k, kp, v, vp, w1, w2, scale)
    torch.cuda.synchronize()
    return out, lse


def gpu_backward(inputs, out, lse, w1, w2, scale, device="cuda"):
    q, k, kp, v, vp, do = (x.to(device) for x in inputs)
    grads = simplicial_attn_bwd(q, k, kp, v, vp, out, do, lse, w1, w2, scale)
    torch.cuda.synchronize()
    return grads


def gpu_backward_fused(inputs, out, lse, w1, w2, scale, kp_bias=0.0, vp_bias=0.0, device="cuda"):
    """The fused backward through its three C-ABI calls (Delta, fused kernel,
    reduction); gradients in the order dq, dk, dk', dv, dv'."""
    q, k, kp, v, vp, do = (x.to(device) for x in inputs)
    b, n, h, d = q.shape
    ws = torch.empty(simplicial_attn_bwd_fused_workspace_size(b, n, h, d, w1, w2, q.dtype), dtype=torch.uint8,
                     device=device)
    simplicial_attn_bwd_preprocess(out, do, w1, w2, ws)
    dk, dv = simplicial_attn_bwd_fused(q, k, kp, v, vp, do, lse, w1, w2, ws, scale, kp_bias=kp_bias,
                                       vp_bias=vp_bias)
    dq, dkp, dvp = simplicial_attn_bwd_fused_reduce(q, w1, w2, ws, scale)
    torch.cuda.synchronize()
    return dq, dk, dkp, dv, dvp


def head_arrays(inputs, b, h):
    """fp64 [N, D] arrays of head (b, h) from [B, N, H, D] tensors."""
    return [x[b, :, h, :].to(torch.float64).numpy() for x in inputs]


def err(x, ref):
    x = np.asarray(x, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    diff = np.abs(x - ref)
    mref = float(np.max(np.abs(ref))) if ref.size else 0.0
    nref = float(np.linalg.norm(ref))
    return dict(
        max_abs=float(diff.max()) if diff.size else 0.0,
        max_rel=float(diff.max()) / mref if mref > 0 else float(diff.max() if diff.size else 0.0),
        norm_rel=float(np.linalg.norm(x - ref)) / nref if nref > 0 else float(np.linalg.norm(x - ref)),
        finite=bool(np.all(np.isfinite(x))),
    )


def report(kind, label, metrics):
    """Append one JSON line per check to $PARITY_REPORT (if set)."""
    path = os.environ.get("PARITY_REPORT")
    if path:
        with open(path, "a") as f:
            f.write(json.dumps({"kind": kind, "case": label, **metrics}) + "\n")


def check_forward(o, lse, o_ref, lse_ref, dtype, label=""):
    t = TOL[dtype]
    eo, el = err(o, o_ref), err(lse, lse_ref)
    report("fwd", label, {"o": eo, "lse": el})
    assert eo["finite"] and el["finite"], f"{label}: non-finite output"
    if dtype == "fp32":
        assert eo["max_rel"] <= t["o_maxrel"], f"{label}: O {eo}"
    else:
        o_scale = max(1.0, float(np.max(np.abs(o_ref)))) if np.size(o_ref) else 1.0
        assert eo["max_abs"] <= t["o_abs"] * o_scale, f"{label}: O {eo} (bar scaled by {o_scale:.3g})"
        assert eo["norm_rel"] <= t["o_norm"], f"{label}: O {eo}"
    assert el["max_abs"] <= t["lse_abs"], f"{label}: LSE {el}"
    return eo, el


def check_grads(grads, refs, dtype, label="", rows=None):
    """grads/refs: sequences of 5 arrays; rows: optional per-gradient row index lists."""
    t = TOL[dtype]
    out = {}
    pairs = []
    for idx, (name, g, r) in enumerate(zip(_names_for(len(grads)), grads, refs)):
        if rows is not None:
            sel = rows[idx]
            if len(sel) == 0:
                continue
            g, r = g[sel], r[sel]
        pairs.append((name, np.asarray(g, np.float64), np.asarray(r, np.float64)))
    for name, g, r in pairs:
        e = err(g, r)
        out[name] = e
        assert e["finite"], f"{label}: {name} non-finite"
        assert e["max_rel"] <= t["g_maxrel"], f"{label}: {name} {e}"
        assert e["norm_rel"] <= t["g_norm"], f"{label}: {name} {e}"
    report("bwd", label, out)
    return out


def check_single_pair_grads(dgrads, arrs, scale, label=""):
    """dQ, dK, dK' when every query sees exactly one (j, k) pair (unit windows
    or a one-token sequence): then P = 1 and dS = dP - Delta = 0 in exact
    arithmetic, so the three gradients vanish. On the GPU dP is a product of
    bf16-rounded operands and Delta comes from the bf16 output, so each is off
    by at most 2^-9 * sum_d |dO_id v_id v'_id|; with scale * (x o y) on top this
    bounds the gradients (a factor 2 of margin). dgrads: dq, dk, dkp as fp64
    [.., N, H, D] arrays; arrs: q, k, kp, v, vp, do in the same layout."""
    q, k, kp, v, vp, do = arrs
    eps = 2.0 ** -8 * np.abs(do * v * vp).sum(axis=-1, keepdims=True)
    out = {}
    for name, g, (x, y) in zip(("dq", "dk", "dkp"), dgrads, [(k, kp), (q, kp), (q, k)]):
        bound = 2 * scale * eps * np.abs(x * y) + 1e-6
        excess = float(np.max(np.abs(g) - bound))
        out[name] = {"max_abs": float(np.max(np.abs(g))), "excess_over_bound": excess}
        assert np.all(np.abs(g) <= bound), f"{label}: {name} exceeds the rounding bound by {excess}"
    report("bwd_single_pair", label, out)


def full_oracle(inputs, w1, w2, scale, backward=True):
    """Oracle on whole tensors (small shapes only)."""
    arrs = [x.to(torch.float64).numpy() for x in inputs]
    o, lse = orc.forward_batched(*arrs[:5], w1, w2, scale)
    grads = orc.backward_batched(*arrs, w1, w2, scale) if backward else None
    return o, lse, grads


def gqa_oracle_forward(q, kv, w1, w2, scale, heads=None, rows=None):
    """Oracle forward with grouped-query attention: q [B, N, H, D], kv = (k, kp,
    v, vp) each [B, N, Hkv, D]; query head h reads K-side head h // (H // Hkv).
    Returns {(b, h): (o [N, D], lse [N])} for the requested heads (all if None),
    computed on the given query rows (all if None)."""
    B, N, H, D = q.shape
    Hkv = kv[0].shape[2]
    g = H // Hkv
    heads = heads if heads is not None else [(b, h) for b in range(B) for h in range(H)]
    res = {}
    for (b, h) in heads:
        qa = q[b, :, h, :].to(torch.float64).numpy()
        ka = [x[b, :, h // g, :].to(torch.float64).numpy() for x in kv]
        res[(b, h)] = orc.forward(qa, *ka, w1, w2, scale, queries=rows)
    return res


def gqa_oracle_backward(q, kv, do, w1, w2, scale, b_heads=None, queries=None):
    """Oracle backward with grouped-query attention (chain rule over shared
    K-side heads): per query head h, the oracle's gradients with K-side head
    h // G; dQ stays per query head, dK, dK', dV, dV' of K-side head hk are the
    fp64 sums over query heads hk*G .. hk*G + G - 1. `b_heads` restricts the
    work to the listed (b, hk) K-side heads (all if None; others stay 0),
    `queries` to the listed query rows (as the oracle's backward).
    Returns dq [B, N, H, D] and dk, dkp, dv, dvp [B, N, Hkv, D] (fp64)."""
    B, N, H, D = q.shape
    Hkv = kv[0].shape[2]
    g = H // Hkv
    b_heads = b_heads if b_heads is not None else [(b, hk) for b in range(B) for hk in range(Hkv)]
    dq = np.zeros((B, N, H, D))
    dkv = [np.zeros((B, N, Hkv, D)) for _ in range(4)]
    for (b, hk) in b_heads:
        ka = [x[b, :, hk, :].to(torch.float64).numpy() for x in kv]
        for h in range(hk * g, hk * g + g):
            qa = q[b, :, h, :].to(torch.float64).numpy()
            da = do[b, :, h, :].to(torch.float64).numpy()
            gr = orc.backward(qa, *ka, da, w1, w2, scale, queries=queries)
            dq[b, :, h, :] = gr[0]
            for t in range(4):
                dkv[t][b, :, hk, :] += gr[1 + t]
    return dq, dkv


def gqa_composite_backward(q, kv, out, do, lse, w1, w2, scale, with_abs=False):
    """The grouped-query backward composed from the library's per-head entry
    point on the GPU: K, K', V, V' repeated per query head, the plain backward,
    then each group's K-side gradients summed in fp32 in ascending head order
    and rounded once. with_abs: also return, per K-side gradient, the fp32 sum
    over each group of the per-query-head magnitudes (a bound's scale)."""
    H, Hkv = q.shape[2], kv[0].shape[2]
    g = H // Hkv
    rep = [x.repeat_interleave(g, dim=2).contiguous() for x in kv]
    grads = simplicial_attn_bwd(q, *rep, out, do, lse, w1, w2, scale)
    torch.cuda.synchronize()
    summed, mags = [], []
    for t in range(1, 5):
        x = grads[t].unflatten(2, (Hkv, g))
        acc = x[:, :, :, 0].float()
        mag = acc.abs()
        for j in range(1, g):
            acc = acc + x[:, :, :, j].float()
            mag = mag + x[:, :, :, j].float().abs()
        summed.append(acc.to(grads[t].dtype).contiguous())
        mags.append(mag)
    comp = (grads[0], *summed)
    return (comp, [None, *mags]) if with_abs else comp


def gqa_native(h, hkv, d, w2, dtype):
    """Shapes whose grouped-query backward reads K, K', V, V' in place (MFMA
    kernels): the key side sums dK, dV over a group's query heads in fp32
    before rounding once, where the composite rounds each head's share first."""
    return dtype == "bf16" and d in (64, 128) and w2 <= 64 and hkv < h


def check_gqa_against_composite(grads, comp, mags, native, label=""):
    """dQ, dK', dV' equal the composite bit for bit (same kernels, same group
    sum). dK, dV on the native path: the composite rounds each query head's
    share to bf16 (relative error 2^-9 each) and then the sum, the native path
    rounds the fp32 sum once, so the two differ by at most
    2^-9 (sum_h |g_h| + |S| + |comp|) <= 2^-8 (sum_h |g_h| + |comp|) per element.
    Both sides also add each head's thousands of products in fp32 in different
    orders (one accumulator for the whole group against one per head); where
    those products cancel, that difference is set by their size, not by the
    result's, hence an absolute allowance of 2^-12 of the tensor's largest
    magnitude (a wrong or missing head's share is of the order of the largest
    values and still fails)."""
    for t, (name, g1, g2) in enumerate(zip(GRAD_NAMES, grads, comp)):
        if native and t in (1, 3):
            diff = (g1.float() - g2.float()).abs()
            bound = 2.0 ** -8 * (mags[t] + g2.float().abs()) + 2.0 ** -12 * float(g2.float().abs().max())
            worst = float((diff - bound).max())
            assert worst <= 0, f"{label}: {name} exceeds the rounding bound by {worst}"
        else:
            assert torch.equal(g1, g2), f"{label}: {name} differs from the per-head composite"


def sample_rows(n, w1, w2, extra=4, seed=0):
    """Query rows spanning the clipped start, window edges, tile edges, middle and end."""
    cand = {0, 1, 2, w2 - 1, w2, w1 - 2, w1 - 1, w1, w1 + 1, 63, 64, 255, 256,
            n // 2, n // 2 + 1, n - 2, n - 1}
    rng = np.random.default_rng(seed)
    cand.update(int(x) for x in rng.integers(0, n, size=extra))
    return sorted(c for c in cand if 0 <= c < n)


def sampled_forward_check(inputs, o_gpu, lse_gpu, w1, w2, scale, dtype, heads, rows, label=""):
    o_gpu = to64(o_gpu)
    lse_gpu = to64(lse_gpu)
    os_, ors, ls, lrs = [], [], [], []
    for (b, h) in heads:
        q, k, kp, v, vp = head_arrays(inputs[:5], b, h)
        o_ref, lse_ref = orc.forward(q, k, kp, v, vp, w1, w2, scale, queries=rows)
        os_.append(o_gpu[b, rows, h, :])
        ors.append(o_ref[rows])
        ls.append(lse_gpu[b, h, rows])
        lrs.append(lse_ref[rows])
    return check_forward(np.concatenate(os_), np.concatenate(ls), np.concatenate(ors),
                         np.concatenate(lrs), dtype, label)


def sampled_backward_check(inputs, grads_gpu, w1, w2, scale, dtype, heads, q_rows, key_rows,
                           label=""):
    """dQ at q_rows; dK/dV and dK'/dV' at key_rows (the oracle runs every query
    touching those rows, so the sampled rows are exact)."""
    n = inputs[0].shape[1]
    w1c, w2c = min(w1, n), min(w2, n)
    queries = set(q_rows)
    for r in key_rows:
        queries.update(range(r, min(n, r + max(w1c, w2c))))
    queries = sorted(queries)
    g_gpu = [to64(g) for g in grads_gpu]
    got = [[] for _ in range(5)]
    ref = [[] for _ in range(5)]
    for (b, h) in heads:
        arrs = head_arrays(inputs, b, h)
        g_ref = orc.backward(*arrs, w1, w2, scale, queries=queries)
        for t in range(5):
            rows = q_rows if t == 0 else key_rows
            got[t].append(g_gpu[t][b, rows, h, :])
            ref[t].append(g_ref[t][rows])
    return check_grads([np.concatenate(x) for x in got], [np.concatenate(x) for x in ref],
                       dtype, label)


class OracleAttention(torch.autograd.Function):
    """The oracle's attention as a CPU float64 autograd function, for references
    of modules built around the kernels: forward = oracle.forward_batched,
    backward = oracle.backward_batched (tensors [B, N, H, D] float64 on the CPU;
    K' and V' enter with the bias constants added, as the kernels take them)."""

    @staticmethod
    def forward(ctx, q, k, kp, v, vp, w1, w2, scale, kp_bias, vp_bias):
        arrs = [x.detach().numpy() for x in (q, k, kp, v, vp)]
        arrs[2] = arrs[2] + kp_bias
        arrs[4] = arrs[4] + vp_bias
        o, _ = orc.forward_batched(*arrs, w1, w2, scale)
        ctx.arrs, ctx.cfg = arrs, (w1, w2, scale)
        return torch.from_numpy(o)

    @staticmethod
    def backward(ctx, do):
        w1, w2, scale = ctx.cfg
        g = orc.backward_batched(*ctx.arrs, do.detach().numpy(), w1, w2, scale)
        return (*(torch.from_numpy(x) for x in g), None, None, None, None, None)
