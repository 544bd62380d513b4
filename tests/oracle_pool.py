"""Runs the fp64 oracle over many heads, or over row ranges of one long head, in
a pool of worker processes, so that the full-size parity tests compare every
head (and every row of a long head) in seconds.

The pool is started with "spawn": the test process holds a GPU context, which
a forked child must not inherit. Each worker uses one BLAS thread. Splitting a
head into row ranges changes no arithmetic of a row (each row of F is its own
softmax); only the order in which the per-range dk and dv sums are added
changes, at fp64 rounding level.
"""
from __future__ import annotations

import multiprocessing as mp
import os

import numpy as np

_POOL = None


def n_workers() -> int:
    return max(1, min(16, os.cpu_count() or 1))


def _init_worker():
    from threadpoolctl import threadpool_limits
    threadpool_limits(1)
    import oracle  # noqa: F401
    import scipy.special  # noqa: F401


def get_pool():
    global _POOL
    if _POOL is None:
        _POOL = mp.get_context("spawn").Pool(n_workers(), initializer=_init_worker)
    return _POOL


def close_pool() -> None:
    global _POOL
    if _POOL is not None:
        _POOL.close()
        _POOL.join()
        _POOL = None


def _fwd_job(args):
    q, k, v, lam, rows, kw = args
    import oracle
    f = oracle.forward(q, k, v, lam, want_matrices=False, row_block=256, rows=rows, **kw)
    return {n: f[n] for n in ("Y", "M", "self_mass", "exch_mass", "LE", "rows")}


def _bwd_job(args):
    q, k, v, lam, dout, rows, kw = args
    import oracle
    r = oracle.backward(q, k, v, lam, dout, row_block=256, rows=rows, **kw)
    return {n: r[n] for n in ("dq", "dk", "dv", "dS", "dlam", "rows")}


def row_ranges(T: int, parts: int) -> list:
    """Contiguous row ranges of roughly equal causal work (row i costs about i)."""
    parts = max(1, min(parts, T))
    w = np.arange(1, T + 1, dtype=np.float64)
    cum = np.cumsum(w) / w.sum()
    cuts = [0] + [int(np.searchsorted(cum, p / parts)) + 1 for p in range(1, parts)] + [T]
    cuts = sorted(set(min(max(c, 0), T) for c in cuts))
    return [np.arange(a, b) for a, b in zip(cuts[:-1], cuts[1:]) if b > a]


def forward_heads(qr, kr, vr, lam, heads, rows=None, **kw) -> list:
    """Oracle forward of each (b, h) head (optionally a row subset of each)."""
    jobs = [(qr[b, h], kr[b, h], vr[b, h], lam, rows, kw) for (b, h) in heads]
    return get_pool().map(_fwd_job, jobs, chunksize=1)


def backward_heads(qr, kr, vr, lam, dor, heads, rows=None, **kw) -> list:
    """Oracle backward of each (b, h) head (optionally a row subset of each)."""
    jobs = [(qr[b, h], kr[b, h], vr[b, h], lam, dor[b, h], rows, kw) for (b, h) in heads]
    return get_pool().map(_bwd_job, jobs, chunksize=1)


def forward_split(q, k, v, lam, parts=None, **kw) -> dict:
    """Oracle forward of one head with its rows spread over the pool."""
    ranges = row_ranges(q.shape[0], parts or 2 * n_workers())
    res = get_pool().map(_fwd_job, [(q, k, v, lam, rr, kw) for rr in ranges], chunksize=1)
    return {n: np.concatenate([r[n] for r in res]) for n in res[0]}


def backward_split(q, k, v, lam, dout, parts=None, **kw) -> dict:
    """Oracle backward of one whole head with its rows spread over the pool:
    dq and dS are concatenated, dk and dv (sums over rows) added."""
    ranges = row_ranges(q.shape[0], parts or 2 * n_workers())
    res = get_pool().map(_bwd_job, [(q, k, v, lam, dout, rr, kw) for rr in ranges], chunksize=1)
    out = {n: np.concatenate([r[n] for r in res]) for n in ("dq", "dS", "rows")}
    out["dk"] = np.sum([r["dk"] for r in res], axis=0)
    out["dv"] = np.sum([r["dv"] for r in res], axis=0)
    out["dlam"] = float(sum(r["dlam"] for r in res))
    return out
