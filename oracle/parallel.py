"""The oracle over many rows at once (test infrastructure, like the rest of
this package): independent row ranges of one oracle function run in threads
(ctypes releases the GIL during a call).  Every output element is still
computed by the same function from the same rows in the same loop order, so
the results are those of one call over all rows; tests/test_oracle_parallel.py
checks this bit for bit.  Used by the GPU parity tests at the large workloads
and by the all-cores leg of the benchmark's CPU baseline.
"""

from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

from . import assign as _assign
from . import center as _center
from . import cosine as _cosine
from . import maxpool as _maxpool

_POOL = None


def workers() -> int:
    """Threads for the oracle: the host's CPUs, at most 16."""
    return max(1, min(16, os.cpu_count() or 1))


def pool() -> ThreadPoolExecutor:
    global _POOL
    if _POOL is None:
        _POOL = ThreadPoolExecutor(workers())
    return _POOL


def _chunks(n: int, parts: int):
    step = max(1, -(-n // parts))
    return [(i, min(i + step, n)) for i in range(0, n, step)]


def oracle_p(anchors: np.ndarray, vis: np.ndarray) -> np.ndarray:
    """p of every sample (Sec. 4.3, equations for M, M-hat and p): the cosine
    rows of each sample split over the pool, then centring and max-pool."""
    B, Nt, _ = anchors.shape
    A64 = [np.ascontiguousarray(anchors[b], np.float64) for b in range(B)]
    V64 = [np.ascontiguousarray(vis[b], np.float64) for b in range(B)]
    parts = max(1, (2 * workers()) // B)
    jobs = [(b, i0, i1) for b in range(B) for (i0, i1) in _chunks(Nt, parts)]
    res = list(pool().map(lambda j: _cosine(A64[j[0]][j[1]:j[2]], V64[j[0]]), jobs))
    p = np.empty((B, vis.shape[1]), np.float64)
    for b in range(B):
        M = np.concatenate([r for j, r in zip(jobs, res) if j[0] == b], axis=0)
        p[b] = _maxpool(_center(M))
    return p


def oracle_assign(vis_b: np.ndarray, kept: np.ndarray, rows: np.ndarray):
    """oracle.assign over `rows` of one sample, the rows split over the pool.
    Returns (assign, best_cos, second_cos) in the order of rows."""
    v64 = np.ascontiguousarray(vis_b, np.float64)
    rows = np.ascontiguousarray(rows, np.int32)
    jobs = _chunks(len(rows), 4 * workers())
    res = list(pool().map(lambda j: _assign(v64, kept, rows[j[0]:j[1]]), jobs))
    if not res:
        e = np.empty(0)
        return np.empty(0, np.int32), e, e
    return tuple(np.concatenate([r[i] for r in res]) for i in range(3))
