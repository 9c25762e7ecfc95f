"""Runs the CPU oracle over chunks of queries in worker processes.

Test infrastructure. The oracle itself is unchanged: each worker calls
`oracle.forward` / `oracle.backward` on a contiguous chunk of query indices of
one head and returns the rows the caller asked for. Forward rows are per query;
backward rows are sums of per-query contributions, so the partial sums of the
chunks add up to exactly what one call over all the queries returns (up to the
order of the fp64 additions).

Workers come from a "forkserver" context: they are started from a clean
interpreter, never forked from a process that has initialised the GPU, and they
only touch NumPy. Each worker is limited to one BLAS thread. The head arrays go
to the workers as memory-mapped .npy files.
"""

import os
import tempfile
import uuid
from concurrent.futures import ProcessPoolExecutor

import numpy as np

_POOL = None
_DIR = None


def workers():
    return max(1, min(16, os.cpu_count() or 1))


def _init():
    try:
        from threadpoolctl import threadpool_limits

        threadpool_limits(1)
    except ImportError:
        pass


def _pool():
    global _POOL
    if _POOL is None:
        import multiprocessing as mp

        _POOL = ProcessPoolExecutor(max_workers=workers(), mp_context=mp.get_context("forkserver"),
                                    initializer=_init)
    return _POOL


def shutdown():
    global _POOL
    if _POOL is not None:
        _POOL.shutdown()
        _POOL = None


def _save(arrs):
    global _DIR
    if _DIR is None:
        _DIR = tempfile.mkdtemp(prefix="oracle_pool_")
    paths = []
    for a in arrs:
        p = os.path.join(_DIR, uuid.uuid4().hex + ".npy")
        np.save(p, np.ascontiguousarray(a, dtype=np.float64))
        paths.append(p)
    return paths


def _drop(paths):
    for p in paths:
        try:
            os.remove(p)
        except OSError:
            pass


def _load(paths):
    return [np.load(p, mmap_mode="r") for p in paths]


def _oracle(module):
    import importlib

    return importlib.import_module(module)


def _fwd_task(paths, w1, w2, scale, queries, module="oracle"):
    orc = _oracle(module)

    arrs = _load(paths)
    o, lse = orc.forward(*arrs, w1, w2, scale, queries=queries)
    return queries, o[queries], lse[queries]


def _bwd_task(paths, w1, w2, scale, queries, rows, module="oracle"):
    orc = _oracle(module)

    arrs = _load(paths)
    grads = orc.backward(*arrs, w1, w2, scale, queries=queries)
    return [g[r] for g, r in zip(grads, rows)]


def _chunks(queries, n):
    queries = list(queries)
    size = max(1, -(-len(queries) // n))
    return [queries[i:i + size] for i in range(0, len(queries), size)]


def forward(q, k, kp, v, vp, w1, w2, scale, queries, module="oracle"):
    """Oracle O and LSE of one head ([N, D] arrays) at the listed queries:
    returns (o [len(queries), D], lse [len(queries)]) in the order given.
    `module`: "oracle" (trilinear logits) or "oracle.determinant_oracle"."""
    paths = _save([q, k, kp, v, vp])
    try:
        pos = {x: i for i, x in enumerate(queries)}
        o = np.zeros((len(queries), q.shape[1]))
        lse = np.zeros(len(queries))
        futs = [_pool().submit(_fwd_task, paths, w1, w2, scale, c, module)
                for c in _chunks(queries, 4 * workers())]
        for f in futs:
            qs, oc, lc = f.result()
            idx = [pos[x] for x in qs]
            o[idx] = oc
            lse[idx] = lc
        return o, lse
    finally:
        _drop(paths)


def backward(q, k, kp, v, vp, do, w1, w2, scale, queries, rows, module="oracle"):
    """The oracle's backward of one head restricted to the listed queries,
    evaluated at rows = (dQ rows, dK rows, dK' rows, dV rows, dV' rows); returns
    five arrays [len(rows[t]), D]. A dK / dV row r is complete when `queries`
    holds every i in [r, r + w1), a dK' / dV' row when it holds [r, r + w2)."""
    paths = _save([q, k, kp, v, vp, do])
    try:
        rows = [list(r) for r in rows]
        acc = [np.zeros((len(r), q.shape[1])) for r in rows]
        futs = [_pool().submit(_bwd_task, paths, w1, w2, scale, c, rows, module)
                for c in _chunks(sorted(set(queries)), 4 * workers())]
        for f in futs:
            for a, part in zip(acc, f.result()):
                a += part
        return acc
    finally:
        _drop(paths)
