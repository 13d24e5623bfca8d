"""Thread-parallel drivers of the oracle for the full-size GPU tests (test infrastructure).

The oracle's C functions are re-entrant and ctypes releases the GIL while one runs, so
independent pieces of one oracle computation run on host threads: the sketch of each worker
(the sketch is per worker), and the estimate of disjoint coordinate ranges (each estimate
depends only on its coordinate). The pieces are put together exactly as the single call
would produce them; nothing of the method is computed here."""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

import oracle

THREADS = max(1, min(16, os.cpu_count() or 1))


def sketch(v: np.ndarray, hp: dict, c: int) -> np.ndarray:
    """oracle.sketch(v, hp, c), one worker per thread."""
    P = v.shape[0]
    r = len(hp["a"])
    out = np.empty((P, r, c), dtype=np.float32)

    def one(q):
        out[q] = oracle.sketch(v[q:q + 1], hp, c)[0]

    with ThreadPoolExecutor(min(THREADS, P)) as ex:
        list(ex.map(one, range(P)))
    return out


def unsketch(merged: np.ndarray, hp: dict, d: int, chunk: int = 1 << 21) -> np.ndarray:
    """oracle.unsketch(merged, hp, d) over coordinate chunks in parallel."""
    if d <= chunk:
        return oracle.unsketch(merged, hp, d)
    out = np.empty(d, dtype=np.float32)
    starts = list(range(0, d, chunk))

    def one(lo):
        hi = min(d, lo + chunk)
        out[lo:hi] = oracle.unsketch_at(merged, hp, np.arange(lo, hi, dtype=np.int64))

    with ThreadPoolExecutor(THREADS) as ex:
        list(ex.map(one, starts))
    return out
