"""Plain CPU oracle for the determinant (rotation-invariant) form of 2-simplicial
attention, Section 5 of arXiv 2507.02754.

TEST INFRASTRUCTURE. Like simplicial_oracle, this module is the checker, not the
product: only the test suite, the smoke check and the benchmark's CPU-baseline
leg may import it. It shares no code with the HIP path and imports nothing from
the package.

* Section 5, Eq. (det): the signed determinant of three 3-vectors, a trilinear
  form that is unchanged when one rotation in SO(3) is applied to all three.
* Section 5, Eq. (logits): the vectors are cut into chunks of 3 components and
  A_ijk = scale * sum_l det([q_i^(l); k_j^(l); k'_k^(l)]).
  Reading: Eq. (logits) has no scale factor; `scale` is kept as an argument so
  that both logit forms share one interface, and scale = 1 is the paper's form
  (pinned by test_scale_one_is_the_papers_unscaled_form).
  Reading: the paper takes the head dimension as a multiple of 3; for other D
  the chunks are components 3l .. 3l + 2 for l < floor(D / 3) and the D mod 3
  trailing components enter no logit (their Q, K, K' gradients are zero).
* The softmax (Eq. (softmax)), the output (Eq. (attenval)) and the windows
  (Section 6) are those of the trilinear form (simplicial_oracle).
* Backward: A is multilinear in (q_i, k_j, k'_k), so the gradient of a logit
  with respect to one operand is the same contraction with that operand left
  out; dS = P * (dP - sum_{jk} P dP) as for the trilinear form.

The determinant is written as a contraction with the Levi-Civita symbol
eps_abc (the sign of the permutation (a, b, c) of (0, 1, 2), 0 if an index
repeats), which is its definition (the Leibniz formula).

Layout: a single head, arrays [N, D]; LSE is the natural-log log-sum-exp.
"""

import itertools

import numpy as np

__all__ = ["levi_civita", "chunks", "det_logits", "forward", "backward"]


def levi_civita():
    """eps[a, b, c] = sign of the permutation (a, b, c) of (0, 1, 2), 0 otherwise."""
    eps = np.zeros((3, 3, 3))
    for perm in itertools.permutations(range(3)):
        inversions = sum(1 for x in range(3) for y in range(x + 1, 3) if perm[x] > perm[y])
        eps[perm] = (-1.0) ** inversions
    return eps


EPS = levi_civita()


def chunks(x):
    """[..., D] -> [..., p, 3], p = D // 3: the 3-component chunks of Eq. (logits)."""
    p = x.shape[-1] // 3
    return x[..., : 3 * p].reshape(*x.shape[:-1], p, 3)


def unchunk(xc, d):
    """[..., p, 3] -> [..., D], zeros in the D mod 3 trailing components."""
    out = np.zeros((*xc.shape[:-2], d))
    out[..., : 3 * xc.shape[-2]] = xc.reshape(*xc.shape[:-2], -1)
    return out


def det_logits(qi, kj, kk, scale):
    """A[j, k] = scale * sum_l det([q_i^(l); k_j^(l); k'_k^(l)]) for one query
    (Eq. (logits)); qi [D], kj [nj, D], kk [nk, D]."""
    return scale * np.einsum("la,jlb,klc,abc->jk", chunks(qi), chunks(kj), chunks(kk), EPS,
                             optimize=True)


def _window(i, w):
    return max(0, i - w + 1), i + 1


def query_forward(q, k, kp, v, vp, i, w1, w2, scale):
    j0, j1 = _window(i, w1)
    k0, k1 = _window(i, w2)
    logits = det_logits(q[i], k[j0:j1], kp[k0:k1], scale)
    m = logits.max()
    e = np.exp(logits - m)
    z = e.sum()
    p = e / z
    o = np.einsum("jk,jd,kd->d", p, v[j0:j1], vp[k0:k1], optimize=True)
    return o, m + np.log(z), p, (j0, j1), (k0, k1)


def forward(q, k, kp, v, vp, w1, w2, scale, queries=None):
    """(O [N, D], LSE [N]) of one head with determinant logits."""
    q, k, kp, v, vp = (np.asarray(a, dtype=np.float64) for a in (q, k, kp, v, vp))
    n, d = q.shape
    out = np.zeros((n, d))
    lse = np.full(n, np.nan)
    for i in range(n) if queries is None else queries:
        out[i], lse[i], _, _, _ = query_forward(q, k, kp, v, vp, i, w1, w2, scale)
    return out, lse


def backward(q, k, kp, v, vp, do, w1, w2, scale, queries=None):
    """(dQ, dK, dK', dV, dV') of one head with determinant logits, accumulated
    over `queries` (default all; completeness of rows as in simplicial_oracle)."""
    q, k, kp, v, vp, do = (np.asarray(a, dtype=np.float64) for a in (q, k, kp, v, vp, do))
    n, d = q.shape
    dq, dk, dkp, dv, dvp = (np.zeros((n, d)) for _ in range(5))
    for i in range(n) if queries is None else queries:
        _, _, p, (j0, j1), (k0, k1) = query_forward(q, k, kp, v, vp, i, w1, w2, scale)
        qc, kjc, kkc = chunks(q[i]), chunks(k[j0:j1]), chunks(kp[k0:k1])
        vj, vk = v[j0:j1], vp[k0:k1]
        dp = np.einsum("d,jd,kd->jk", do[i], vj, vk, optimize=True)
        ds = p * (dp - (p * dp).sum())
        # dA/dq_i, dA/dk_j, dA/dk'_k: the contraction without that operand.
        dq[i] += scale * unchunk(np.einsum("jk,jlb,klc,abc->la", ds, kjc, kkc, EPS, optimize=True), d)
        dk[j0:j1] += scale * unchunk(np.einsum("jk,la,klc,abc->jlb", ds, qc, kkc, EPS, optimize=True), d)
        dkp[k0:k1] += scale * unchunk(np.einsum("jk,la,jlb,abc->klc", ds, qc, kjc, EPS, optimize=True), d)
        dv[j0:j1] += np.einsum("jk,d,kd->jd", p, do[i], vk, optimize=True)
        dvp[k0:k1] += np.einsum("jk,d,jd->kd", p, do[i], vj, optimize=True)
    return dq, dk, dkp, dv, dvp
