"""Seeded synthetic workloads shared by the oracle-side tests, the GPU tests and the benchmark.

This package draws random numbers and nothing else: it holds none of the compression
method's arithmetic. It provides

* the five workloads (flat gradient size d, worker count P, sketch shape r x c, top-k k,
  number of consecutive steps) with their input recipes, and
* ``hash_params`` -- the seeded (a, b) pairs of the bucket and sign hash families
  (``1 <= a < p``, ``0 <= b < p`` with ``p = 2**31 - 1``), and
* ``gradients`` -- the P workers' fp32 gradients of one step, as a [P][d] array, and
* ``fill_draws`` -- the uniform 32-bit random draws of HEAVYMIX's random fill for one step.

Generation is counter-based (SplitMix64, see ``synth.c``), so any step and worker can be
produced independently and reproducibly. Distributions stand in for the gradients of the
networks the paper trains (ResNet-20 and VGG-16 on CIFAR-10, Sec. IV) and for two larger
sizes (ResNet-50, a 2-layer LSTM language model); no dataset or trained model is used.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass, field

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "libsynth.so")
_lib = None

MERSENNE_P = (1 << 31) - 1
BASE_SEED = 2108060040

TAG_GRAD = ord("G")
TAG_HASH = ord("H")
TAG_SCALE = ord("S")
TAG_INDEX = ord("X")
TAG_ROWS = ord("R")
TAG_FILL = ord("F")

KIND_T3, KIND_LAPLACE, KIND_NORMAL = 0, 1, 2


def build(verbose: bool = False) -> str:
    """Compile libsynth.so with gcc (OpenMP, -O2, no fast-math)."""
    import subprocess

    src = os.path.join(_HERE, "synth.c")
    cmd = ["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c11", "-o", _LIB_PATH, src, "-lm"]
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
    u64, i64, vp = ctypes.c_uint64, ctypes.c_int64, ctypes.c_void_p
    lib.synth_mix.restype = u64
    lib.synth_mix.argtypes = [u64]
    lib.synth_key.restype = u64
    lib.synth_key.argtypes = [u64, u64, u64, u64]
    lib.synth_fill.restype = ctypes.c_int
    lib.synth_fill.argtypes = [ctypes.c_int, u64, i64, i64, vp, vp, vp]
    lib.synth_draw_at.restype = None
    lib.synth_draw_at.argtypes = [ctypes.c_int, u64, i64, vp, vp]
    lib.synth_words.restype = None
    lib.synth_words.argtypes = [u64, i64, i64, vp]
    _lib = lib
    return lib


def key(seed: int, tag: int, step: int = 0, worker: int = 0) -> int:
    return int(_load().synth_key(seed, tag, step, worker))


def words(k: int, n0: int, count: int) -> np.ndarray:
    out = np.empty(count, dtype=np.uint64)
    if count:
        _load().synth_words(k, n0, count, out.ctypes.data)
    return out


def uniforms(k: int, count: int) -> np.ndarray:
    w = words(k, 0, count)
    return ((w >> np.uint64(11)).astype(np.float64) + 0.5) * 2.0 ** -53


def fill(kind: int, k: int, seg_start: np.ndarray, seg_scale: np.ndarray, out: np.ndarray) -> None:
    seg_start = np.ascontiguousarray(seg_start, dtype=np.int64)
    seg_scale = np.ascontiguousarray(seg_scale, dtype=np.float64)
    assert out.dtype == np.float32 and out.flags.c_contiguous
    rc = _load().synth_fill(kind, k, out.size, seg_scale.size, seg_start.ctypes.data,
                            seg_scale.ctypes.data, out.ctypes.data)
    if rc != 0:
        raise ValueError("synth_fill: bad segment table")


def draw_at(kind: int, k: int, idx: np.ndarray) -> np.ndarray:
    idx = np.ascontiguousarray(idx, dtype=np.int64)
    out = np.empty(idx.size, dtype=np.float64)
    if idx.size:
        _load().synth_draw_at(kind, k, idx.size, idx.ctypes.data, out.ctypes.data)
    return out


def sample_without_replacement(k: int, n: int, m: int) -> np.ndarray:
    """m distinct values of [0, n) by a partial Fisher-Yates shuffle over the word stream k."""
    if m > n:
        raise ValueError("m > n")
    w = words(k, 0, m)
    swap: dict[int, int] = {}
    out = np.empty(m, dtype=np.int64)
    for t in range(m):
        j = t + int(w[t] % np.uint64(n - t))
        vt, vj = swap.get(t, t), swap.get(j, j)
        swap[j] = vt
        out[t] = vj
    return out


@dataclass(frozen=True)
class Workload:
    """One synthetic workload: sizes plus the recipe of its gradients."""

    name: str
    d: int
    P: int
    r: int
    c: int
    k: int
    steps: int
    recipe: str
    seed: int
    rho: float = 0.9
    note: str = field(default="", compare=False)


WORKLOADS = {
    w.name: w
    for w in [
        Workload("t3planted-d65536-P4", 65_536, 4, 5, 4_096, 655, 1, "t3planted", BASE_SEED + 1,
                 note="Student-t(3) x 1e-3 plus 64 planted +-0.1 coordinates shared by all workers"),
        Workload("laplace20-d270000-P4", 270_000, 4, 5, 27_000, 2_700, 10, "laplace20", BASE_SEED + 2,
                 note="ResNet-20-sized; Laplace with 20 log-uniform layer scales in [1e-4, 1e-2]"),
        Workload("t3scaled-d14.7M-P4", 14_700_000, 4, 5, 1_470_000, 14_700, 5, "t3scaled", BASE_SEED + 3,
                 note="VGG-16-sized; Student-t(3) x 1e-3 with a fixed 0.1% of coordinates x100"),
        Workload("laplace53-d25.6M-P8", 25_600_000, 8, 5, 256_000, 25_600, 5, "laplace53", BASE_SEED + 4,
                 note="ResNet-50-sized; Laplace with 53 log-uniform layer scales in [1e-5, 1e-2]"),
        Workload("rowsparse-d66M-P16", 66_000_000, 16, 7, 1_320_000, 66_000, 3, "rowsparse", BASE_SEED + 5,
                 note="LSTM-LM-sized; 2% of 22,000 embedding rows N(0,1e-2), dense half N(0,1e-4)"),
    ]
}
WORKLOAD_ORDER = list(WORKLOADS)


def hash_params(w: Workload | int, r: int | None = None) -> dict[str, np.ndarray]:
    """Bucket hash (a, b) and sign hash (a2, b2) per row, drawn from the 'H' stream.

    Row j uses words 4j .. 4j+3: a = 1 + w0 mod (p-1), b = w1 mod p, a2 = 1 + w2 mod (p-1),
    b2 = w3 mod p. Accepts a Workload, or a bare seed plus a row count.
    """
    seed = w.seed if isinstance(w, Workload) else int(w)
    rows = w.r if isinstance(w, Workload) else int(r)
    ws = words(key(seed, TAG_HASH), 0, 4 * rows).reshape(rows, 4)
    p = np.uint64(MERSENNE_P)
    return {
        "a": (np.uint64(1) + ws[:, 0] % (p - np.uint64(1))).astype(np.uint32),
        "b": (ws[:, 1] % p).astype(np.uint32),
        "a2": (np.uint64(1) + ws[:, 2] % (p - np.uint64(1))).astype(np.uint32),
        "b2": (ws[:, 3] % p).astype(np.uint32),
    }


def fill_draws(w: Workload | int, step: int, d: int | None = None) -> np.ndarray:
    """The random draws of HEAVYMIX's fill for one step: one uniform 32-bit word per
    coordinate (the high half of word i of the 'F' stream of that step). Accepts a
    Workload, or a bare seed plus d."""
    seed = w.seed if isinstance(w, Workload) else int(w)
    n = w.d if isinstance(w, Workload) else int(d)
    return (words(key(seed, TAG_FILL, step), 0, n) >> np.uint64(32)).astype(np.uint32)


def _log_uniform_scales(seed: int, nseg: int, lo_exp: float, hi_exp: float) -> np.ndarray:
    u = uniforms(key(seed, TAG_SCALE), nseg)
    return 10.0 ** (lo_exp + (hi_exp - lo_exp) * u)


def _equal_segments(d: int, nseg: int) -> np.ndarray:
    base = d // nseg
    starts = np.arange(nseg + 1, dtype=np.int64) * base
    starts[-1] = d
    return starts


def layer_segments(w: Workload) -> tuple[np.ndarray, np.ndarray]:
    """(segment starts, Laplace scales) of the two layered-Laplace workloads."""
    if w.recipe == "laplace20":
        return _equal_segments(w.d, 20), _log_uniform_scales(w.seed, 20, -4.0, -2.0)
    if w.recipe == "laplace53":
        return _equal_segments(w.d, 53), _log_uniform_scales(w.seed, 53, -5.0, -2.0)
    raise ValueError(w.recipe)


def planted(w: Workload) -> tuple[np.ndarray, np.ndarray]:
    """Indices and signs of the 64 planted coordinates of the t3planted workload."""
    idx = sample_without_replacement(key(w.seed, TAG_INDEX), w.d, 64)
    sg = words(key(w.seed, TAG_INDEX, 1), 0, 64)
    return idx, np.where((sg & np.uint64(1)) == 1, 1.0, -1.0)


def scaled_set(w: Workload) -> np.ndarray:
    """The fixed 0.1% of coordinates multiplied by 100 in the t3scaled workload."""
    return sample_without_replacement(key(w.seed, TAG_INDEX), w.d, w.d // 1000)


EMB_ROWS, EMB_COLS, EMB_ACTIVE = 22_000, 1_500, 440


def active_rows(w: Workload, step: int, worker: int) -> np.ndarray:
    return np.sort(sample_without_replacement(key(w.seed, TAG_ROWS, step, worker), EMB_ROWS, EMB_ACTIVE))


def gradients(w: Workload, step: int, out: np.ndarray | None = None, workers=None) -> np.ndarray:
    """fp32 gradients of every worker at one step, shape [P][d] (or [len(workers)][d])."""
    workers = list(range(w.P)) if workers is None else list(workers)
    if out is None:
        out = np.empty((len(workers), w.d), dtype=np.float32)
    for row, q in enumerate(workers):
        g = out[row]
        kq = key(w.seed, TAG_GRAD, step, q)
        if w.recipe == "t3planted":
            fill(KIND_T3, kq, np.array([0, w.d]), np.array([1e-3]), g)
            idx, sgn = planted(w)
            g[idx] = (1e-3 * draw_at(KIND_T3, kq, idx) + 0.1 * sgn).astype(np.float32)
        elif w.recipe in ("laplace20", "laplace53"):
            starts, scales = layer_segments(w)
            fill(KIND_LAPLACE, kq, starts, scales, g)
        elif w.recipe == "t3scaled":
            fill(KIND_T3, kq, np.array([0, w.d]), np.array([1e-3]), g)
            idx = scaled_set(w)
            g[idx] = (1e-1 * draw_at(KIND_T3, kq, idx)).astype(np.float32)
        elif w.recipe == "rowsparse":
            emb = EMB_ROWS * EMB_COLS
            assert w.d == 2 * emb
            sigma = np.zeros(EMB_ROWS + 1)
            sigma[active_rows(w, step, q)] = 1e-2
            sigma[EMB_ROWS] = 1e-4
            starts = np.append(np.arange(EMB_ROWS + 1, dtype=np.int64) * EMB_COLS, w.d)
            fill(KIND_NORMAL, kq, starts, sigma, g)
        else:
            raise ValueError(w.recipe)
    return out


def small_workload(name: str, d: int, P: int, r: int, c: int, k: int, recipe: str = "laplace20",
                   seed: int = BASE_SEED + 100, steps: int = 1) -> Workload:
    """A workload of arbitrary shape for edge-case tests (laplace20 scaling adapts to d)."""
    return Workload(name, d, P, r, c, k, steps, recipe, seed)
