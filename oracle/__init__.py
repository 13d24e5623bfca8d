"""CPU oracle of the gs-SGD compression step -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of ``bench.py`` may
import this package. The GPU library never imports, links or calls it, and the two share
no code: the oracle is ``gs_oracle.c`` (plain C, fp64 sketch cells, full sorts), loaded
here through ctypes and wrapped for numpy arrays. See the header of ``gs_oracle.c`` for the
paper passages each function follows.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "gs_oracle.c")
_LIB_PATH = os.path.join(_HERE, "libgs_oracle.so")
_lib = None

CFLAGS = ["-O2", "-ffp-contract=off", "-fno-fast-math", "-std=c11", "-fPIC", "-shared"]


def build(verbose: bool = False) -> str:
    cmd = ["gcc", *CFLAGS, "-o", _LIB_PATH, _SRC]
    if verbose:
        print(" ".join(cmd))
    subprocess.run(cmd, check=True)
    return _LIB_PATH


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        build()
    lib = ctypes.CDLL(_LIB_PATH)
    i32, i64, u32, u64, f32, f64, vp = (ctypes.c_int32, ctypes.c_int64, ctypes.c_uint32, ctypes.c_uint64,
                                        ctypes.c_float, ctypes.c_double, ctypes.c_void_p)
    sig = {
        "ora_hash_raw": (u64, [u32, u32, i64]),
        "ora_bucket": (i64, [u32, u32, i64, i64]),
        "ora_sign": (ctypes.c_int, [u32, u32, i64]),
        "ora_buckets": (None, [u32, u32, i64, i64, vp, vp]),
        "ora_signs": (None, [u32, u32, i64, vp, vp]),
        "ora_hash_raws": (None, [u32, u32, i64, vp, vp]),
        "ora_accumulate": (None, [i64, f32, vp, vp, vp]),
        "ora_sketch": (ctypes.c_int, [i32, i64, i32, i64, vp, vp, vp, vp, vp, vp]),
        "ora_sketch_cells": (ctypes.c_int, [i32, i64, i32, i64, vp, vp, vp, vp, vp, i64, vp, vp, vp]),
        "ora_tree_sum": (f32, [i32, vp]),
        "ora_merge": (ctypes.c_int, [i32, i64, vp, vp]),
        "ora_unsketch": (ctypes.c_int, [i64, i32, i64, vp, vp, vp, vp, vp, vp]),
        "ora_unsketch_at": (ctypes.c_int, [i32, i64, vp, vp, vp, vp, vp, i64, vp, vp]),
        "ora_topk": (ctypes.c_int, [i64, i64, vp, vp, vp]),
        "ora_gather_reset": (ctypes.c_int, [i32, i64, i64, vp, i32, vp, vp, vp]),
        "ora_l2sq_estimate": (f64, [i32, i64, vp]),
        "ora_heavy_count": (i64, [i64, i64, vp, f64]),
        "ora_row_sq_sum": (f64, [i64, vp]),
        "ora_heavymix": (ctypes.c_int, [i64, i32, i64, i64, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp]),
        "ora_apply_update": (ctypes.c_int, [i64, i64, vp, vp, f32, vp]),
        "ora_sketch_state_update": (ctypes.c_int, [i64, i32, i64, i64, f32, i32, vp, vp, vp, vp, vp, vp, vp, vp,
                                                   vp, vp]),
        "ora_sketch_momentum_step": (ctypes.c_int, [i32, i64, i32, i64, i64, f32, i32, vp, vp, vp, vp, vp, vp, vp,
                                                    vp, vp, vp, vp]),
        "ora_step": (ctypes.c_int, [i32, i64, i32, i64, i64, f32, i32, vp, vp, vp, vp, vp, vp, vp, vp, vp,
                                    vp, vp, vp]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def _p(a: np.ndarray | None):
    return None if a is None else a.ctypes.data


def _u32(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.uint32)


def _f32(a) -> np.ndarray:
    a = np.ascontiguousarray(a)
    assert a.dtype == np.float32, a.dtype
    return a


def _hp(hp: dict):
    return _u32(hp["a"]), _u32(hp["b"]), _u32(hp["a2"]), _u32(hp["b2"])


def _check(rc: int, what: str):
    if rc != 0:
        raise RuntimeError(f"oracle {what} failed (status {rc})")


# --- hashes --------------------------------------------------------------------------

def hash_raw(a: int, b: int, idx) -> np.ndarray:
    idx = np.ascontiguousarray(idx, dtype=np.int64)
    out = np.empty(idx.size, dtype=np.int64)
    _load().ora_hash_raws(a, b, idx.size, _p(idx), _p(out))
    return out


def buckets(a: int, b: int, c: int, idx) -> np.ndarray:
    idx = np.ascontiguousarray(idx, dtype=np.int64)
    out = np.empty(idx.size, dtype=np.int64)
    _load().ora_buckets(a, b, c, idx.size, _p(idx), _p(out))
    return out


def signs(a2: int, b2: int, idx) -> np.ndarray:
    idx = np.ascontiguousarray(idx, dtype=np.int64)
    out = np.empty(idx.size, dtype=np.int32)
    _load().ora_signs(a2, b2, idx.size, _p(idx), _p(out))
    return out


# --- the five steps ------------------------------------------------------------------

def accumulate(g: np.ndarray, u: np.ndarray, v: np.ndarray, rho: float = 0.9) -> None:
    """In place: u <- rho*u + g, v <- v + u (fp32, elementwise)."""
    g, u_, v_ = _f32(g), u, v
    assert u_.flags.c_contiguous and v_.flags.c_contiguous and u_.dtype == v_.dtype == np.float32
    assert g.size == u_.size == v_.size
    _load().ora_accumulate(g.size, rho, _p(g), _p(u_), _p(v_))


def sketch(v: np.ndarray, hp: dict, c: int) -> np.ndarray:
    """Per-worker Count Sketch tables, shape [P][r][c], of v shaped [P][d]."""
    v = _f32(v)
    P, d = v.shape
    a, b, a2, b2 = _hp(hp)
    r = a.size
    out = np.empty((P, r, c), dtype=np.float32)
    _check(_load().ora_sketch(P, d, r, c, _p(a), _p(b), _p(a2), _p(b2), _p(v), _p(out)), "sketch")
    return out


def sketch_cells(v: np.ndarray, hp: dict, c: int, rows, cols) -> np.ndarray:
    """Sketch cells (rows[n], cols[n]) of every worker, shape [n][P]. Cells must be distinct."""
    v = _f32(v)
    P, d = v.shape
    a, b, a2, b2 = _hp(hp)
    rows = np.ascontiguousarray(rows, dtype=np.int32)
    cols = np.ascontiguousarray(cols, dtype=np.int64)
    out = np.empty((rows.size, P), dtype=np.float32)
    _check(_load().ora_sketch_cells(P, d, a.size, c, _p(a), _p(b), _p(a2), _p(b2), _p(v), rows.size, _p(rows),
                                    _p(cols), _p(out)), "sketch_cells")
    return out


def tree_sum(x) -> np.float32:
    x = np.ascontiguousarray(x, dtype=np.float32)
    return np.float32(_load().ora_tree_sum(x.size, _p(x)))


def merge(tables: np.ndarray) -> np.ndarray:
    """Tree-order sum over the leading (worker) axis."""
    tables = _f32(tables)
    P = tables.shape[0]
    out = np.empty(tables.shape[1:], dtype=np.float32)
    _check(_load().ora_merge(P, out.size, _p(tables), _p(out)), "merge")
    return out


def unsketch(merged: np.ndarray, hp: dict, d: int) -> np.ndarray:
    merged = _f32(merged)
    a, b, a2, b2 = _hp(hp)
    r, c = merged.shape
    out = np.empty(d, dtype=np.float32)
    _check(_load().ora_unsketch(d, r, c, _p(a), _p(b), _p(a2), _p(b2), _p(merged), _p(out)), "unsketch")
    return out


def unsketch_at(merged: np.ndarray, hp: dict, idx) -> np.ndarray:
    merged = _f32(merged)
    a, b, a2, b2 = _hp(hp)
    r, c = merged.shape
    idx = np.ascontiguousarray(idx, dtype=np.int64)
    out = np.empty(idx.size, dtype=np.float32)
    _check(_load().ora_unsketch_at(r, c, _p(a), _p(b), _p(a2), _p(b2), _p(merged), idx.size, _p(idx), _p(out)),
           "unsketch_at")
    return out


def topk(est: np.ndarray, k: int) -> tuple[np.ndarray, np.float32]:
    """(ascending int32 indices of the k largest |est|, ties to lower index; the k-th key)."""
    est = _f32(est)
    out = np.empty(k, dtype=np.int32)
    kth = ctypes.c_float(0.0)
    _check(_load().ora_topk(est.size, k, _p(est), _p(out), ctypes.addressof(kth)), "topk")
    return out, np.float32(kth.value)


def gather_reset(idx: np.ndarray, u: np.ndarray, v: np.ndarray, reset_momentum: bool = True) -> np.ndarray:
    """Exact tree-order sums of v over workers at idx; then zero v (and u) there. In place."""
    idx = np.ascontiguousarray(idx, dtype=np.int32)
    assert u.flags.c_contiguous and v.flags.c_contiguous
    P, d = v.shape
    out = np.empty(idx.size, dtype=np.float32)
    _check(_load().ora_gather_reset(P, d, idx.size, _p(idx), int(bool(reset_momentum)), _p(u), _p(v), _p(out)),
           "gather_reset")
    return out


def l2sq_estimate(merged: np.ndarray) -> float:
    merged = _f32(merged)
    r, c = merged.shape
    return float(_load().ora_l2sq_estimate(r, c, _p(merged)))


def heavy_count(est: np.ndarray, k: int, l2sq: float) -> int:
    est = _f32(est)
    return int(_load().ora_heavy_count(est.size, k, _p(est), l2sq))


def row_sq_sum(row) -> float:
    """Sum of squares of one sketch row in the pairwise-tree order (fp64)."""
    row = _f32(row)
    return float(_load().ora_row_sq_sum(row.size, _p(row)))


def heavymix(merged: np.ndarray, hp: dict, d: int, k: int, rnd: np.ndarray) -> dict:
    """HEAVYMIX as printed (Alg. 2): heavy set by est^2 >= l2sq/k plus a fill of the
    non-heavy coordinates with the largest draws rnd[i] >> 1 (ties to the lower index).

    Returns {"idx": ascending int32[k], "n_heavy": |H|, "l2sq": the l2-norm-squared
    estimate, "est": the estimates}."""
    merged = _f32(merged)
    a, b, a2, b2 = _hp(hp)
    r, c = merged.shape
    rnd = np.ascontiguousarray(rnd, dtype=np.uint32)
    assert rnd.size == d
    est = np.empty(d, dtype=np.float32)
    idx = np.empty(k, dtype=np.int32)
    nh = ctypes.c_int64(0)
    l2 = ctypes.c_double(0.0)
    _check(_load().ora_heavymix(d, r, c, k, _p(a), _p(b), _p(a2), _p(b2), _p(merged), _p(rnd), _p(est), _p(idx),
                                ctypes.addressof(nh), ctypes.addressof(l2)), "heavymix")
    return {"idx": idx, "n_heavy": int(nh.value), "l2sq": float(l2.value), "est": est}


def sketch_momentum_step(g, U, E, hp: dict, k: int, rho: float = 0.9, reset_momentum: bool = True,
                         want_est: bool = True) -> dict:
    """Momentum and error kept in the sketch (one step): U, E ([r][c] fp32) are updated in
    place. Returns {"merged", "idx" (ascending), "values" (the estimates at idx), "est"}."""
    g = _f32(g)
    P, d = g.shape
    a, b, a2, b2 = _hp(hp)
    r, c = U.shape
    assert U.dtype == np.float32 and E.dtype == np.float32 and U.flags.c_contiguous and E.flags.c_contiguous
    assert E.shape == (r, c) and a.size == r
    merged = np.empty((r, c), dtype=np.float32)
    est = np.empty(d, dtype=np.float32) if want_est else None
    idx = np.empty(k, dtype=np.int32)
    values = np.empty(k, dtype=np.float32)
    _check(_load().ora_sketch_momentum_step(P, d, r, c, k, rho, int(bool(reset_momentum)), _p(a), _p(b), _p(a2),
                                            _p(b2), _p(g), _p(U), _p(E), _p(merged), _p(est), _p(idx), _p(values)),
           "sketch_momentum_step")
    return {"merged": merged, "idx": idx, "values": values, "est": est}


def apply_update(w: np.ndarray, idx, values, lr: float) -> None:
    """w[idx] -= lr * values (fp32, each operation rounded), in place."""
    assert w.dtype == np.float32 and w.flags.c_contiguous
    idx = np.ascontiguousarray(idx, dtype=np.int32)
    values = _f32(values)
    _check(_load().ora_apply_update(w.size, idx.size, _p(idx), _p(values), lr, _p(w)), "apply_update")


def sketch_state_update(merged, U, E, hp: dict, d: int, k: int, rho: float = 0.9,
                        reset_momentum: bool = True) -> dict:
    """The sketch-space step after the merge, from a given merged sketch S ([r][c])."""
    merged = _f32(merged)
    a, b, a2, b2 = _hp(hp)
    r, c = merged.shape
    assert U.shape == E.shape == (r, c) and U.flags.c_contiguous and E.flags.c_contiguous
    idx = np.empty(k, dtype=np.int32)
    values = np.empty(k, dtype=np.float32)
    _check(_load().ora_sketch_state_update(d, r, c, k, rho, int(bool(reset_momentum)), _p(a), _p(b), _p(a2), _p(b2),
                                           _p(merged), _p(U), _p(E), None, _p(idx), _p(values)),
           "sketch_state_update")
    return {"idx": idx, "values": values}


def step(g, u, v, hp: dict, c: int, k: int, rho: float = 0.9, reset_momentum: bool = True,
         want_tables: bool = True, want_est: bool = True) -> dict:
    """One full step in C (accumulate, sketch, merge, estimate, Top_k, gather+reset).

    u and v are updated in place. Returns the intermediate results as numpy arrays.
    """
    g = _f32(g)
    P, d = g.shape
    a, b, a2, b2 = _hp(hp)
    r = a.size
    tables = np.empty((P, r, c), dtype=np.float32) if want_tables else None
    est = np.empty(d, dtype=np.float32) if want_est else None
    merged = np.empty((r, c), dtype=np.float32)
    idx = np.empty(k, dtype=np.int32)
    values = np.empty(k, dtype=np.float32)
    _check(_load().ora_step(P, d, r, c, k, rho, int(bool(reset_momentum)), _p(a), _p(b), _p(a2), _p(b2), _p(g),
                            _p(u), _p(v), _p(tables), _p(merged), _p(est), _p(idx), _p(values)), "step")
    return {"tables": tables, "merged": merged, "est": est, "idx": idx, "values": values}
