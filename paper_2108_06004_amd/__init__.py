"""Python binding of the gs-SGD compression hot path (C ABI in include/gs.h).

Argument marshalling only: every computation runs in the HIP kernels of ``libgs.so``.
Tensors are torch CUDA (ROCm) tensors owned by the caller; the stream is torch's current
stream unless one is given. There is no CPU fallback: if ``libgs.so`` has not been built,
loading raises ``GsLibraryMissing``.

Names follow the C ABI: ``gs_create``, ``gs_accumulate``, ``gs_sketch``, ``gs_merge``,
``gs_unsketch_topk``, ``gs_gather_reset``, ``gs_step``, ``gs_destroy``. ``GsContext``
bundles them with shape checks.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libgs.so")

GS_OK, GS_ERR_INVALID_ARG, GS_ERR_OUT_OF_MEMORY, GS_ERR_DEVICE, GS_ERR_UNSUPPORTED = range(5)
GS_MAX_WORKERS = 64
GS_MAX_ROWS = 16
EXPORTED = ("gs_create", "gs_destroy", "gs_accumulate", "gs_sketch", "gs_merge", "gs_unsketch_topk",
            "gs_gather_reset", "gs_step", "gs_heavymix_topk", "gs_step_heavymix", "gs_step_sketch_momentum",
            "gs_apply_update", "gs_step_profiled", "gs_timing_start", "gs_timing_stop", "gs_unsketch_topk_static",
            "gs_describe", "gs_status_string", "gs_last_error")
GS_STATIC_MAX_D = 4194304  # largest d of gs_unsketch_topk_static (its fixed scratch array)
GS_NUM_STAGES = 5
STAGES = ("accumulate", "sketch", "merge", "select", "gather_reset")
# layouts of the per-worker state u, v (gs_config.state_layout)
GS_STATE_WORKER_MAJOR, GS_STATE_INTERLEAVED = 0, 1
STATE_LAYOUTS = {"worker_major": GS_STATE_WORKER_MAJOR, "interleaved": GS_STATE_INTERLEAVED}


def state_stride(P: int) -> int:
    """Row length of the interleaved state: P rounded up to a multiple of 4."""
    return (P + 3) // 4 * 4


class GsLibraryMissing(RuntimeError):
    pass


class GsError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{msg} (status {status})")
        self.status = status


class gs_config(ctypes.Structure):
    _fields_ = [
        ("d", ctypes.c_int64),
        ("P", ctypes.c_int32),
        ("r", ctypes.c_int32),
        ("c", ctypes.c_int64),
        ("k_max", ctypes.c_int64),
        ("rho", ctypes.c_float),
        ("reset_momentum", ctypes.c_int32),
        ("hash_a", ctypes.POINTER(ctypes.c_uint32)),
        ("hash_b", ctypes.POINTER(ctypes.c_uint32)),
        ("sign_a", ctypes.POINTER(ctypes.c_uint32)),
        ("sign_b", ctypes.POINTER(ctypes.c_uint32)),
        ("state_layout", ctypes.c_int32),
        ("options", ctypes.c_int32),
    ]


GS_OPT_ROW_COPY = 1
GS_SKETCH_GATHER, GS_SKETCH_ATOMIC = 0, 1  # gs_plan.sketch


class gs_plan(ctypes.Structure):
    _fields_ = [(name, ctypes.c_int32) for name in
                ("sketch", "tile_width", "tiles", "segments", "packed_lists", "prune",
                 "row_copy")]


_lib = None


def load_library():
    """Load libgs.so (built in-tree by ``__graft_entry__.build()``)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise GsLibraryMissing(f"{LIB_PATH} is not built; run __graft_entry__.build() first")
    lib = ctypes.CDLL(LIB_PATH)
    vp, i64, st = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int
    lib.gs_create.argtypes = [ctypes.POINTER(gs_config), ctypes.POINTER(vp)]
    lib.gs_destroy.argtypes = [vp]
    lib.gs_accumulate.argtypes = [vp, vp, vp, vp, vp]
    lib.gs_sketch.argtypes = [vp, vp, vp, vp]
    lib.gs_merge.argtypes = [vp, vp, vp, vp]
    lib.gs_unsketch_topk.argtypes = [vp, vp, vp, i64, vp, vp]
    lib.gs_gather_reset.argtypes = [vp, vp, vp, i64, vp, vp, vp]
    lib.gs_step.argtypes = [vp, vp, vp, vp, vp, i64, vp, vp, vp]
    lib.gs_step_profiled.argtypes = [vp, vp, vp, vp, vp, i64, vp, vp, vp, vp]
    lib.gs_heavymix_topk.argtypes = [vp, vp, vp, i64, vp, vp, vp, vp, vp]
    lib.gs_step_heavymix.argtypes = [vp, vp, vp, vp, vp, i64, vp, vp, vp, vp, vp]
    lib.gs_step_sketch_momentum.argtypes = [vp, vp, vp, vp, vp, i64, vp, vp, vp]
    lib.gs_apply_update.argtypes = [vp, vp, vp, vp, i64, ctypes.c_float, vp]
    lib.gs_timing_start.argtypes = [vp, ctypes.c_int32]
    lib.gs_timing_stop.argtypes = [vp, vp, vp]
    lib.gs_unsketch_topk_static.argtypes = [ctypes.POINTER(gs_config), vp, vp, i64, vp, vp]
    lib.gs_describe.argtypes = [vp, ctypes.POINTER(gs_plan)]
    for name in ("gs_create", "gs_destroy", "gs_accumulate", "gs_sketch", "gs_merge", "gs_unsketch_topk",
                 "gs_gather_reset", "gs_step", "gs_heavymix_topk", "gs_step_heavymix", "gs_step_sketch_momentum",
                 "gs_apply_update", "gs_step_profiled", "gs_timing_start", "gs_timing_stop",
                 "gs_unsketch_topk_static"):
        getattr(lib, name).restype = st
    lib.gs_status_string.argtypes = [st]
    lib.gs_status_string.restype = ctypes.c_char_p
    lib.gs_last_error.argtypes = [vp]
    lib.gs_last_error.restype = ctypes.c_char_p
    _lib = lib
    return lib


def _check(status: int, ctx=None, what: str = ""):
    if status != GS_OK:
        lib = load_library()
        detail = lib.gs_last_error(ctx).decode() if lib.gs_last_error(ctx) is not None else ""
        raise GsError(status, f"{what}: {lib.gs_status_string(status).decode()}: {detail}")


def gs_describe(ctx) -> dict:
    plan = gs_plan()
    _check(load_library().gs_describe(ctx, ctypes.byref(plan)), ctx, "gs_describe")
    return {name: getattr(plan, name) for name, _ in gs_plan._fields_}


def _ptr(t, dtype=None, numel=None, name="tensor"):
    """Device pointer of a contiguous CUDA tensor after shape/dtype checks (None -> NULL)."""
    if t is None:
        return None
    import torch

    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{name} must be a CUDA tensor")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if numel is not None and t.numel() != numel:
        raise ValueError(f"{name} must have {numel} elements, got {t.numel()}")
    return t.data_ptr()


def _stream(stream):
    import torch

    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def gs_create(d: int, P: int, r: int, c: int, k_max: int, hash_a, hash_b, sign_a, sign_b, rho: float = 0.9,
              reset_momentum: bool = True, state_layout: int = GS_STATE_WORKER_MAJOR, options: int = 0) -> int:
    """Create a context on the current device; returns the opaque handle (an int)."""
    lib = load_library()
    arrs = [np.ascontiguousarray(a, dtype=np.uint32) for a in (hash_a, hash_b, sign_a, sign_b)]
    if any(a.size != r for a in arrs):
        raise ValueError("hash parameter arrays must have r entries")
    u32p = ctypes.POINTER(ctypes.c_uint32)
    cfg = gs_config(d, P, r, c, k_max, rho, int(bool(reset_momentum)), *(a.ctypes.data_as(u32p) for a in arrs),
                    int(state_layout), int(options))
    out = ctypes.c_void_p()
    _check(lib.gs_create(ctypes.byref(cfg), ctypes.byref(out)), None, "gs_create")
    return out.value


def gs_unsketch_topk_static(d: int, r: int, c: int, hash_params: dict, merged, k: int, est, idx,
                            stream=None) -> None:
    """gs_unsketch_topk without a context and without allocating (the library's fixed
    scratch array; d <= GS_STATIC_MAX_D). merged: [r][c] fp32; est: [d] fp32 or None;
    idx: [k] int32. Errors are read from gs_last_error(NULL)."""
    import torch

    lib = load_library()
    arrs = [np.ascontiguousarray(hash_params[n], dtype=np.uint32) for n in ("a", "b", "a2", "b2")]
    if any(a.size != r for a in arrs):
        raise ValueError("hash parameter arrays must have r entries")
    u32p = ctypes.POINTER(ctypes.c_uint32)
    cfg = gs_config(d, 1, r, c, max(1, k), 0.0, 1, *(a.ctypes.data_as(u32p) for a in arrs), GS_STATE_WORKER_MAJOR,
                    0)
    _check(lib.gs_unsketch_topk_static(ctypes.byref(cfg), _stream(stream),
                                       _ptr(merged, torch.float32, r * c, "merged"), k,
                                       _ptr(est, torch.float32, d, "est"), _ptr(idx, torch.int32, k, "idx")),
           None, "gs_unsketch_topk_static")


def gs_destroy(ctx: int) -> None:
    _check(load_library().gs_destroy(ctx), None, "gs_destroy")


def gs_accumulate(ctx: int, g, u, v, stream=None) -> None:
    _check(load_library().gs_accumulate(ctx, _stream(stream), _ptr(g, name="g"), _ptr(u, name="u"),
                                        _ptr(v, name="v")), ctx, "gs_accumulate")


def gs_sketch(ctx: int, v, tables, stream=None) -> None:
    _check(load_library().gs_sketch(ctx, _stream(stream), _ptr(v, name="v"), _ptr(tables, name="tables")), ctx,
           "gs_sketch")


def gs_merge(ctx: int, tables, merged, stream=None) -> None:
    _check(load_library().gs_merge(ctx, _stream(stream), _ptr(tables, name="tables"), _ptr(merged, name="merged")),
           ctx, "gs_merge")


def gs_unsketch_topk(ctx: int, merged, k: int, est, idx, stream=None) -> None:
    _check(load_library().gs_unsketch_topk(ctx, _stream(stream), _ptr(merged, name="merged"), k,
                                           _ptr(est, name="est"), _ptr(idx, name="idx")), ctx, "gs_unsketch_topk")


def gs_gather_reset(ctx: int, idx, k: int, u, v, values, stream=None) -> None:
    _check(load_library().gs_gather_reset(ctx, _stream(stream), _ptr(idx, name="idx"), k, _ptr(u, name="u"),
                                          _ptr(v, name="v"), _ptr(values, name="values")), ctx, "gs_gather_reset")


def gs_step(ctx: int, g, u, v, k: int, merged, idx, values, stream=None) -> None:
    _check(load_library().gs_step(ctx, _stream(stream), _ptr(g, name="g"), _ptr(u, name="u"), _ptr(v, name="v"), k,
                                  _ptr(merged, name="merged"), _ptr(idx, name="idx"), _ptr(values, name="values")),
           ctx, "gs_step")


def gs_heavymix_topk(ctx: int, merged, k: int, rnd, est, idx, n_heavy, l2sq, stream=None) -> None:
    _check(load_library().gs_heavymix_topk(ctx, _stream(stream), _ptr(merged, name="merged"), k,
                                           _ptr(rnd, name="rnd"), _ptr(est, name="est"), _ptr(idx, name="idx"),
                                           _ptr(n_heavy, name="n_heavy"), _ptr(l2sq, name="l2sq")),
           ctx, "gs_heavymix_topk")


def gs_step_heavymix(ctx: int, g, u, v, k: int, rnd, merged, idx, values, n_heavy, stream=None) -> None:
    _check(load_library().gs_step_heavymix(ctx, _stream(stream), _ptr(g, name="g"), _ptr(u, name="u"),
                                           _ptr(v, name="v"), k, _ptr(rnd, name="rnd"), _ptr(merged, name="merged"),
                                           _ptr(idx, name="idx"), _ptr(values, name="values"),
                                           _ptr(n_heavy, name="n_heavy")), ctx, "gs_step_heavymix")


def gs_step_sketch_momentum(ctx: int, g, U, E, k: int, merged, idx, values, stream=None) -> None:
    _check(load_library().gs_step_sketch_momentum(ctx, _stream(stream), _ptr(g, name="g"), _ptr(U, name="U"),
                                                  _ptr(E, name="E"), k, _ptr(merged, name="merged"),
                                                  _ptr(idx, name="idx"), _ptr(values, name="values")),
           ctx, "gs_step_sketch_momentum")


def gs_apply_update(ctx: int, idx, values, k: int, lr: float, w, stream=None) -> None:
    _check(load_library().gs_apply_update(ctx, _stream(stream), _ptr(idx, name="idx"), _ptr(values, name="values"),
                                          k, lr, _ptr(w, name="w")), ctx, "gs_apply_update")


def gs_step_profiled(ctx: int, g, u, v, k: int, merged, idx, values, stream=None) -> dict:
    """gs_step with per-stage HIP-event timing (blocks until done); returns stage -> ms."""
    ms = (ctypes.c_float * GS_NUM_STAGES)()
    _check(load_library().gs_step_profiled(ctx, _stream(stream), _ptr(g, name="g"), _ptr(u, name="u"),
                                           _ptr(v, name="v"), k, _ptr(merged, name="merged"), _ptr(idx, name="idx"),
                                           _ptr(values, name="values"), ms), ctx, "gs_step_profiled")
    return dict(zip(STAGES, [float(x) for x in ms]))


class GsContext:
    """A context plus shape/dtype checks on every call."""

    def __init__(self, d: int, P: int, r: int, c: int, k_max: int, hash_params: dict, rho: float = 0.9,
                 reset_momentum: bool = True, state_layout: str = "worker_major", row_copy: bool = False):
        """row_copy: reserve the interleaved row copy in an interleaved-state context too
        (GS_OPT_ROW_COPY; needed there by step_sketch_momentum and by v views that are not
        16-byte aligned)."""
        if state_layout not in STATE_LAYOUTS:
            raise ValueError(f"state_layout must be one of {sorted(STATE_LAYOUTS)}")
        self.d, self.P, self.r, self.c, self.k_max = d, P, r, c, k_max
        self.state_layout = state_layout
        self.handle = gs_create(d, P, r, c, k_max, hash_params["a"], hash_params["b"], hash_params["a2"],
                                hash_params["b2"], rho, reset_momentum, STATE_LAYOUTS[state_layout],
                                GS_OPT_ROW_COPY if row_copy else 0)

    def describe(self) -> dict:
        """gs_describe: the form this context computes in (sketch form, tiles, write-out buckets, ...)."""
        return gs_describe(self.handle)

    @property
    def state_shape(self) -> tuple:
        """Shape of u and v: (P, d) worker-major, or (d, P rounded up to 4) interleaved."""
        if self.state_layout == "interleaved":
            return (self.d, state_stride(self.P))
        return (self.P, self.d)

    def state_numel(self) -> int:
        a, b = self.state_shape
        return a * b

    def to_state(self, x):
        """A [P][d] tensor (worker rows) rearranged into this context's state layout (a new
        tensor; interleaved padding is zero)."""
        import torch

        if self.state_layout == "worker_major":
            return x.reshape(self.P, self.d).contiguous().clone()
        out = torch.zeros(self.state_shape, dtype=x.dtype, device=x.device)
        out[:, :self.P] = x.reshape(self.P, self.d).t()
        return out

    def from_state(self, t):
        """The [P][d] view of a state tensor in this context's layout (a copy for interleaved)."""
        if self.state_layout == "worker_major":
            return t.reshape(self.P, self.d)
        return t.reshape(self.state_shape)[:, :self.P].t().contiguous()

    def close(self):
        if self.handle:
            gs_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def _f32(self, t, n, name):
        import torch

        _ptr(t, torch.float32, n, name)
        return t

    def accumulate(self, g, u, v, stream=None):
        ns = self.state_numel()
        gs_accumulate(self.handle, self._f32(g, self.P * self.d, "g"), self._f32(u, ns, "u"), self._f32(v, ns, "v"),
                      stream)

    def sketch(self, v, tables, stream=None):
        gs_sketch(self.handle, self._f32(v, self.state_numel(), "v"),
                  self._f32(tables, self.P * self.r * self.c, "tables"), stream)

    def merge(self, tables, merged, stream=None):
        gs_merge(self.handle, self._f32(tables, self.P * self.r * self.c, "tables"),
                 self._f32(merged, self.r * self.c, "merged"), stream)

    def unsketch_topk(self, merged, k, idx, est=None, stream=None):
        import torch

        _ptr(idx, torch.int32, k, "idx")
        if est is not None:
            self._f32(est, self.d, "est")
        gs_unsketch_topk(self.handle, self._f32(merged, self.r * self.c, "merged"), k, est, idx, stream)

    def gather_reset(self, idx, k, u, v, values, stream=None):
        import torch

        _ptr(idx, torch.int32, k, "idx")
        ns = self.state_numel()
        gs_gather_reset(self.handle, idx, k, self._f32(u, ns, "u"), self._f32(v, ns, "v"),
                        self._f32(values, k, "values"), stream)

    def step(self, g, u, v, k, merged, idx, values, stream=None):
        import torch

        n, ns = self.P * self.d, self.state_numel()
        _ptr(idx, torch.int32, k, "idx")
        gs_step(self.handle, self._f32(g, n, "g"), self._f32(u, ns, "u"), self._f32(v, ns, "v"), k,
                self._f32(merged, self.r * self.c, "merged"), idx, self._f32(values, k, "values"), stream)

    def heavymix_topk(self, merged, k, rnd, idx, est=None, n_heavy=None, l2sq=None, stream=None):
        """HEAVYMIX as printed. rnd: uint32 [d] draws (torch has no uint32 arithmetic, so an
        int32 tensor holding the same bits is accepted too). n_heavy: int64 [1], l2sq:
        float64 [1] (optional outputs)."""
        import torch

        _ptr(idx, torch.int32, k, "idx")
        if rnd.dtype not in (torch.int32, torch.uint32):
            raise TypeError("rnd must hold 32-bit draws (int32 or uint32)")
        _ptr(rnd, None, self.d, "rnd")
        if est is not None:
            self._f32(est, self.d, "est")
        if n_heavy is not None:
            _ptr(n_heavy, torch.int64, 1, "n_heavy")
        if l2sq is not None:
            _ptr(l2sq, torch.float64, 1, "l2sq")
        gs_heavymix_topk(self.handle, self._f32(merged, self.r * self.c, "merged"), k, rnd, est, idx, n_heavy, l2sq,
                         stream)

    def step_heavymix(self, g, u, v, k, rnd, merged, idx, values, n_heavy=None, stream=None):
        import torch

        n, ns = self.P * self.d, self.state_numel()
        _ptr(idx, torch.int32, k, "idx")
        if rnd.dtype not in (torch.int32, torch.uint32):
            raise TypeError("rnd must hold 32-bit draws (int32 or uint32)")
        _ptr(rnd, None, self.d, "rnd")
        if n_heavy is not None:
            _ptr(n_heavy, torch.int64, 1, "n_heavy")
        gs_step_heavymix(self.handle, self._f32(g, n, "g"), self._f32(u, ns, "u"), self._f32(v, ns, "v"), k, rnd,
                         self._f32(merged, self.r * self.c, "merged"), idx, self._f32(values, k, "values"), n_heavy,
                         stream)

    def step_sketch_momentum(self, g, U, E, k, merged, idx, values, stream=None):
        """Momentum and error kept in the sketch: U, E are [r][c] fp32 state tensors."""
        import torch

        rc = self.r * self.c
        _ptr(idx, torch.int32, k, "idx")
        gs_step_sketch_momentum(self.handle, self._f32(g, self.P * self.d, "g"), self._f32(U, rc, "U"),
                                self._f32(E, rc, "E"), k, self._f32(merged, rc, "merged"), idx,
                                self._f32(values, k, "values"), stream)

    def apply_update(self, idx, values, k, lr, w, stream=None):
        """w[idx] -= lr * values (fp32, no fused multiply-add); w: [d] fp32 parameters."""
        import torch

        _ptr(idx, torch.int32, None, "idx")
        if idx.numel() < k or values.numel() < k:
            raise ValueError("idx and values need at least k elements")
        _ptr(values, torch.float32, None, "values")
        gs_apply_update(self.handle, idx, values, k, lr, self._f32(w, self.d, "w"), stream)

    def timing_start(self, max_steps: int) -> None:
        """Record stage events inside the next max_steps fused steps (no synchronization)."""
        _check(load_library().gs_timing_start(self.handle, max_steps), self.handle, "gs_timing_start")

    def timing_stop(self) -> tuple[dict, int]:
        """(stage -> mean ms over the timed steps, number of timed steps); synchronizes."""
        ms = (ctypes.c_float * GS_NUM_STAGES)()
        n = ctypes.c_int32(0)
        _check(load_library().gs_timing_stop(self.handle, ms, ctypes.byref(n)), self.handle, "gs_timing_stop")
        return dict(zip(STAGES, [float(x) for x in ms])), int(n.value)

    def step_profiled(self, g, u, v, k, merged, idx, values, stream=None) -> dict:
        import torch

        n, ns = self.P * self.d, self.state_numel()
        _ptr(idx, torch.int32, k, "idx")
        return gs_step_profiled(self.handle, self._f32(g, n, "g"), self._f32(u, ns, "u"), self._f32(v, ns, "v"), k,
                                self._f32(merged, self.r * self.c, "merged"), idx, self._f32(values, k, "values"),
                                stream)
