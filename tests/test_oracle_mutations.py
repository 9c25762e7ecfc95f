"""Planted mistakes in a copy of the oracle must be caught by its pins.

Each case rewrites one expression of oracle/simplicial_oracle.py in memory (a
dropped term, a wrong sign, an off-by-one window, a swapped operand, a softmax
over the wrong axes), loads the result as a throw-away module and runs a short
battery of the pins from test_oracle_pins.py against it. At least one pin must
fail for every mutation; the unmodified source must pass them all.
"""

import importlib.util
import os
import types

import numpy as np
import pytest
import torch

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC_PATH = os.path.join(ROOT, "oracle", "simplicial_oracle.py")

MUTATIONS = [
    ("window_off_by_one", "max(0, i - w + 1)", "max(0, i - w)"),
    ("logit_scale_dropped", 'logits = scale * np.einsum("d,jd,kd->jk"', 'logits = np.einsum("d,jd,kd->jk"'),
    ("lse_missing_max", "lse = m + np.log(z)", "lse = np.log(z)"),
    ("softmax_per_j_row", "z = e.sum()", "z = e.sum(axis=1, keepdims=True)"),
    ("output_uses_k_prime", 'p, v[j0:j1], vp[k0:k1], optimize=True)', 'p, v[j0:j1], kp[k0:k1], optimize=True)'),
    ("ds_sign", "ds = p * (dp - (p * dp).sum())", "ds = p * (dp + (p * dp).sum())"),
    ("ds_no_delta", "ds = p * (dp - (p * dp).sum())", "ds = p * dp"),
    ("dq_scale_dropped", "dq[i] += scale * ", "dq[i] += "),
    ("dk_scale_dropped", "dk[j0:j1] += scale * ", "dk[j0:j1] += "),
    ("dv_uses_ds", 'dv[j0:j1] += np.einsum("jk,d,kd->jd", p,', 'dv[j0:j1] += np.einsum("jk,d,kd->jd", ds,'),
    ("dvp_uses_q", '"jk,d,jd->kd", p, do[i], vj', '"jk,d,jd->kd", p, q[i], vj'),
    ("dkp_uses_dp", '"jk,d,jd->kd", ds, q[i], kj', '"jk,d,jd->kd", dp, q[i], kj'),
    ("brute_mask_inclusive", "(s > t - w1)", "(s >= t - w1)"),
]


def _load(src):
    mod = types.ModuleType("mutated_oracle")
    exec(compile(src, SRC_PATH, "exec"), mod.__dict__)
    return mod


def _sdpa(q, k, v, w, scale):
    n = q.shape[0]
    i = torch.arange(n)[:, None]
    j = torch.arange(n)[None, :]
    mask = (j <= i) & (j > i - w)
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a))[None, None]
    return torch.nn.functional.scaled_dot_product_attention(
        t(q), t(k), t(v), attn_mask=mask[None, None], scale=scale)[0, 0].numpy()


def _battery(orc):
    """Return the list of pins the module fails (exceptions count as failures)."""
    failed = []
    rng = np.random.default_rng(3)

    def check(name, fn):
        try:
            if not fn():
                failed.append(name)
        except Exception:  # a shape error from a mutation is a caught mistake too
            failed.append(name)

    b, n, h, d, w1, w2 = 1, 12, 1, 4, 5, 3
    q, k, kp, v, vp = (rng.standard_normal((b, n, h, d)) for _ in range(5))

    def brute():
        o_bf, l_bf, _ = orc.brute_force_forward(q, k, kp, v, vp, w1, w2, 0.5)
        o, l = orc.forward_batched(q, k, kp, v, vp, w1, w2, 0.5)
        return np.allclose(o, o_bf, atol=1e-12) and np.allclose(l, l_bf, atol=1e-12)

    def swa():
        ones = np.ones((n, d))
        o, _ = orc.forward(q[0, :, 0], k[0, :, 0], ones, v[0, :, 0], ones, w1, w2, 0.5)
        return np.allclose(o, _sdpa(q[0, :, 0], k[0, :, 0], v[0, :, 0], w1, 0.5), atol=1e-12)

    def q0():
        o, l = orc.forward(q[0, :, 0], k[0, :, 0], kp[0, :, 0], v[0, :, 0], vp[0, :, 0], w1, w2, 0.5)
        return (np.allclose(o[0], v[0, 0, 0] * vp[0, 0, 0], atol=1e-14)
                and abs(l[0] - 0.5 * np.sum(q[0, 0, 0] * k[0, 0, 0] * kp[0, 0, 0])) < 1e-13)

    def fd():
        arrs = [a[0, :, 0].copy() for a in (q, k, kp, v, vp)]
        do = rng.standard_normal((n, d))
        grads = orc.backward(*arrs, do, w1, w2, 0.5)
        eps = 1e-6
        for t in range(5):
            for (i, c) in [(n - 1, 1), (n // 2, 2), (3, 0)]:
                p_ = [a.copy() for a in arrs]
                m_ = [a.copy() for a in arrs]
                p_[t][i, c] += eps
                m_[t][i, c] -= eps
                lp = np.sum(orc.forward(*p_, w1, w2, 0.5)[0] * do)
                lm = np.sum(orc.forward(*m_, w1, w2, 0.5)[0] * do)
                if abs(grads[t][i, c] - (lp - lm) / (2 * eps)) > 1e-6:
                    return False
        return True

    check("brute_force", brute)
    check("swa_reduction", swa)
    check("query_zero", q0)
    check("finite_differences", fd)
    return failed


def test_unmodified_oracle_passes_battery():
    with open(SRC_PATH) as f:
        assert _battery(_load(f.read())) == []


@pytest.mark.parametrize("name,old,new", MUTATIONS, ids=[m[0] for m in MUTATIONS])
def test_planted_mistake_is_caught(name, old, new):
    with open(SRC_PATH) as f:
        src = f.read()
    assert src.count(old) == 1, f"mutation anchor for {name} not unique/present"
    failed = _battery(_load(src.replace(old, new)))
    assert failed, f"planted mistake {name} passed every pin"
