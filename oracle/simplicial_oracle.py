"""Plain CPU oracle for causal sliding-window 2-simplicial (trilinear) attention.

TEST INFRASTRUCTURE. This module is the checker, not the product: only the test
suite, the smoke check and the benchmark's CPU-baseline leg may import it. It
shares no code with the HIP path (no kernels, headers, helpers or constants) and
imports nothing from the package.

Everything here is float64 NumPy, written to be checked against the paper by
eye. Citations refer to arXiv 2507.02754, "Fast and Simplex: 2-Simplicial
Attention in Triton":

* Section 4, Eq. (3d-attention): trilinear logits
  A_ijk = (1/sqrt(d)) * sum_l Q_il K_jl K'_kl  (the 1/sqrt(d) is `scale`).
* Section 4, Eq. (softmax): S_ijk = exp(A_ijk) / sum_{j,k} exp(A_ijk), one joint
  softmax per query over all (j, k) pairs.
* Section 4, Eq. (attenval): out_i = sum_{j,k} S_ijk (v_j o v'_k), o = Hadamard.
* Section 4, Algorithm 1: the dense einsum form with a causal mask; used here
  as the brute-force definition (`brute_force_forward`).
* Section 6 (Model design): the sliding windows. Query i sees w1 keys of K/V
  and w2 keys of K'/V'. Read here as j in (i-w1, i] and k in (i-w2, i],
  clipped at 0, the diagonal included (the window masks of Listing 1).
* Section 7 (Kernel optimization), the backward equations for dV, dV', dP,
  dS = dsoftmax(dP), dK, dK', dQ. Read with P for the probabilities, the
  factor `scale` on dQ, dK, dK' (none on dV, dV'), and dK' summed over (i, j).
  dsoftmax is the Jacobian-vector product of the joint softmax:
  dS = P * (dP - sum_{jk} P dP).

Layout of every public function: a single head, arrays [N, D]; the batched
helpers take [B, N, H, D] and return O as [B, N, H, D], LSE as [B, H, N].
LSE is the natural-log log-sum-exp of the query's logits (the saved softmax
statistic, Listing 1's M).
"""

import numpy as np

__all__ = [
    "window",
    "query_forward",
    "forward",
    "backward",
    "forward_batched",
    "backward_batched",
    "brute_force_forward",
]


def window(i, w):
    """Index range [lo, hi) of the causal window (i-w, i], clipped at 0 (Section 6)."""
    return max(0, i - w + 1), i + 1


def query_forward(q, k, kp, v, vp, i, w1, w2, scale):
    """Forward pass of one query i (Section 4 equations over the Section 6 windows).

    Returns (o_i [D], lse_i, P [nj, nk], (j0, j1), (k0, k1)).
    """
    j0, j1 = window(i, w1)
    k0, k1 = window(i, w2)
    # Eq. (3d-attention): logits over the window, A[j, k] = scale * <q_i, k_j, k'_k>.
    logits = scale * np.einsum("d,jd,kd->jk", q[i], k[j0:j1], kp[k0:k1], optimize=True)
    # Eq. (softmax): one joint softmax over all (j, k) pairs of this query.
    m = logits.max()
    e = np.exp(logits - m)
    z = e.sum()
    p = e / z
    lse = m + np.log(z)
    # Eq. (attenval): o_i = sum_{j,k} P[j, k] (v_j o v'_k).
    o = np.einsum("jk,jd,kd->d", p, v[j0:j1], vp[k0:k1], optimize=True)
    return o, lse, p, (j0, j1), (k0, k1)


def forward(q, k, kp, v, vp, w1, w2, scale, queries=None):
    """Forward pass of one head; q, k, kp, v, vp are [N, D].

    `queries` restricts the work to the listed query indices (others stay 0 /
    NaN in the returned arrays). Returns (O [N, D], LSE [N]).
    """
    q, k, kp, v, vp = (np.asarray(a, dtype=np.float64) for a in (q, k, kp, v, vp))
    n, d = q.shape
    out = np.zeros((n, d))
    lse = np.full(n, np.nan)
    for i in range(n) if queries is None else queries:
        out[i], lse[i], _, _, _ = query_forward(q, k, kp, v, vp, i, w1, w2, scale)
    return out, lse


def backward(q, k, kp, v, vp, do, w1, w2, scale, queries=None):
    """Backward pass of one head (Section 7's gradient equations, read as above).

    Accumulates the contribution of every query in `queries` (default: all) to
    the five gradients and returns (dQ, dK, dK', dV, dV'), each [N, D]. A row
    of dK/dV is complete when `queries` covers i in [j, j + w1); a row of
    dK'/dV' when it covers i in [k, k + w2); a row of dQ when it holds i.
    The probabilities come from this module's own forward.
    """
    q, k, kp, v, vp, do = (np.asarray(a, dtype=np.float64) for a in (q, k, kp, v, vp, do))
    n, d = q.shape
    dq, dk, dkp, dv, dvp = (np.zeros((n, d)) for _ in range(5))
    for i in range(n) if queries is None else queries:
        _, _, p, (j0, j1), (k0, k1) = query_forward(q, k, kp, v, vp, i, w1, w2, scale)
        kj, kk, vj, vk = k[j0:j1], kp[k0:k1], v[j0:j1], vp[k0:k1]
        # dP_ijk = sum_d dO_id V_jd V'_kd
        dp = np.einsum("d,jd,kd->jk", do[i], vj, vk, optimize=True)
        # dS = dsoftmax(dP): the vector-Jacobian product of the joint softmax.
        ds = p * (dp - (p * dp).sum())
        # dQ_i = scale * sum_{jk} dS_ijk (K_j o K'_k)
        dq[i] += scale * np.einsum("jk,jd,kd->d", ds, kj, kk, optimize=True)
        # dK_j += scale * sum_k dS_ijk (Q_i o K'_k)
        dk[j0:j1] += scale * np.einsum("jk,d,kd->jd", ds, q[i], kk, optimize=True)
        # dK'_k += scale * sum_j dS_ijk (Q_i o K_j)
        dkp[k0:k1] += scale * np.einsum("jk,d,jd->kd", ds, q[i], kj, optimize=True)
        # dV_j += sum_k P_ijk (dO_i o V'_k)
        dv[j0:j1] += np.einsum("jk,d,kd->jd", p, do[i], vk, optimize=True)
        # dV'_k += sum_j P_ijk (dO_i o V_j)
        dvp[k0:k1] += np.einsum("jk,d,jd->kd", p, do[i], vj, optimize=True)
    return dq, dk, dkp, dv, dvp


def forward_batched(q, k, kp, v, vp, w1, w2, scale, heads=None, queries=None):
    """[B, N, H, D] inputs -> (O [B, N, H, D], LSE [B, H, N]); optional head/query subsets."""
    q, k, kp, v, vp = (np.asarray(a, dtype=np.float64) for a in (q, k, kp, v, vp))
    bsz, n, nh, d = q.shape
    out = np.zeros((bsz, n, nh, d))
    lse = np.full((bsz, nh, n), np.nan)
    for b in range(bsz):
        for h in range(nh):
            if heads is not None and (b, h) not in heads:
                continue
            o, l = forward(q[b, :, h], k[b, :, h], kp[b, :, h], v[b, :, h], vp[b, :, h],
                           w1, w2, scale, queries)
            out[b, :, h] = o
            lse[b, h] = l
    return out, lse


def backward_batched(q, k, kp, v, vp, do, w1, w2, scale, heads=None, queries=None):
    """[B, N, H, D] inputs -> five [B, N, H, D] gradients; optional head/query subsets."""
    arrs = [np.asarray(a, dtype=np.float64) for a in (q, k, kp, v, vp, do)]
    bsz, n, nh, d = arrs[0].shape
    grads = [np.zeros((bsz, n, nh, d)) for _ in range(5)]
    for b in range(bsz):
        for h in range(nh):
            if heads is not None and (b, h) not in heads:
                continue
            g = backward(*(a[b, :, h] for a in arrs), w1, w2, scale, queries)
            for dst, src in zip(grads, g):
                dst[b, :, h] = src
    return tuple(grads)


def brute_force_forward(q, k, kp, v, vp, w1, w2, scale):
    """Algorithm 1 of Section 4 executed literally on [B, N, H, D] inputs (tiny N only).

    The dense logits tensor [B, H, t, s, r] is built with one einsum, the
    windowed causal mask (s in (t-w1, t], r in (t-w2, t]) sets excluded entries
    to -inf, the softmax runs jointly over the last two axes and a second
    einsum forms the output. Returns (O [B, N, H, D], LSE [B, H, N], P).
    """
    q, k, kp, v, vp = (np.asarray(a, dtype=np.float64) for a in (q, k, kp, v, vp))
    n = q.shape[1]
    logits = scale * np.einsum("btnh,bsnh,brnh->bntsr", q, k, kp)
    t = np.arange(n)[:, None, None]
    s = np.arange(n)[None, :, None]
    r = np.arange(n)[None, None, :]
    mask = (s <= t) & (s > t - w1) & (r <= t) & (r > t - w2)
    logits = np.where(mask, logits, -np.inf)
    m = logits.max(axis=(-1, -2), keepdims=True)
    e = np.exp(logits - m)
    z = e.sum(axis=(-1, -2), keepdims=True)
    p = e / z
    out = np.einsum("bntsr,bsnh,brnh->btnh", p, v, vp)
    lse = (m + np.log(z))[..., 0, 0]
    return out, lse, p
