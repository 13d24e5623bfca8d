"""Training integration: the loop body of Alg. 1 on one GPU with P simulated workers.

Each call to ``GlobalSketchSGD.step`` takes the P workers' flat gradients of one iteration
([P][d], computed by the caller, e.g. on P micro-batches) and the flat parameters ``w``
([d]); it runs one compression step of the library (accumulate, sketch, merge, selection,
exact values and reset -- or one of the variants below) and applies the update
``w <- w - (lr / P) * G~`` through ``gs_apply_update``. The values are sums over the P
workers (Alg. 1 sums the sketches), so the learning rate of a mean gradient is divided by P
here.

The density (k / d) and learning rate follow a warm-up schedule by epoch, as in the paper's
experiments (Sec. IV: the first epochs use densities 0.25, 0.0725, 0.015, 0.004 and smaller
learning rates before the target density).

``GlobalSketchOptimizer`` is the same step as a ``torch.optim.Optimizer`` over a module's
parameters: it moves the parameters into one flat fp32 buffer (each parameter's ``data``
becomes a view of it), collects the P simulated workers' gradients into the [P][d] buffer
(``collect(q)`` after worker q's backward pass), and its ``step()`` runs the library's
fused step and ``gs_apply_update`` on that flat buffer.

Variants: ``selection="heavymix"`` uses HEAVYMIX as printed (Alg. 2) with fresh uniform
32-bit fill draws every step from a seeded torch generator; ``state="sketch"`` keeps
momentum and error in the merged sketch (``gs_step_sketch_momentum``). The sketch-space
state applies sketch estimates rather than exact values, so it needs gradients with heavy
hitters that the sketch can recover (k well below c): on a dense quadratic with 8
coordinates per cell it diverges, where the vector-space state still descends.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import torch

from . import GsContext


@dataclass
class DensitySchedule:
    """Per-epoch (density, lr) pairs for the warm-up, then (final_density, lr) onwards."""

    final_density: float
    lr: float
    warmup: list = field(default_factory=list)  # [(density, lr), ...] for epochs 0, 1, ...

    def at(self, epoch: int) -> tuple[float, float]:
        if 0 <= epoch < len(self.warmup):
            d, lr = self.warmup[epoch]
            return float(d), float(lr)
        return float(self.final_density), float(self.lr)

    def k_at(self, epoch: int, d: int) -> int:
        density, _ = self.at(epoch)
        return min(d, max(1, int(math.ceil(density * d))))

    def k_max(self, d: int) -> int:
        epochs = range(len(self.warmup) + 1)
        return max(self.k_at(e, d) for e in epochs)


class GlobalSketchSGD:
    """gs-SGD updates of a flat fp32 parameter vector on one GPU (P simulated workers)."""

    def __init__(self, d: int, P: int, r: int, c: int, hash_params: dict, schedule: DensitySchedule,
                 rho: float = 0.9, reset_momentum: bool = True, selection: str = "topk", state: str = "vector",
                 seed: int = 0, device="cuda:0"):
        import torch

        if selection not in ("topk", "heavymix") or state not in ("vector", "sketch"):
            raise ValueError("selection must be 'topk' or 'heavymix'; state 'vector' or 'sketch'")
        if state == "sketch" and selection != "topk":
            raise ValueError("the sketch-space state uses the deterministic top-k selection")
        self.d, self.P, self.r, self.c = d, P, r, c
        self.schedule, self.selection, self.state = schedule, selection, state
        self.k_max = schedule.k_max(d)
        self.ctx = GsContext(d, P, r, c, self.k_max, hash_params, rho=rho, reset_momentum=reset_momentum)
        f32 = dict(dtype=torch.float32, device=device)
        if state == "vector":
            self.u = torch.zeros((P, d), **f32)
            self.v = torch.zeros((P, d), **f32)
        else:
            self.U = torch.zeros((r, c), **f32)
            self.E = torch.zeros((r, c), **f32)
        self.merged = torch.empty((r, c), **f32)
        self.idx = torch.empty(self.k_max, dtype=torch.int32, device=device)
        self.values = torch.empty(self.k_max, **f32)
        if selection == "heavymix":
            self.gen = torch.Generator(device=device)
            self.gen.manual_seed(seed)
            self.rnd = torch.empty(d, dtype=torch.int32, device=device)
            self.n_heavy = torch.empty(1, dtype=torch.int64, device=device)

    def step(self, grads, w, epoch: int = 0) -> dict:
        """One iteration: compress the P gradients ([P][d]) and update w ([d]) in place.
        Returns k and the learning rate used (the selection stays in self.idx[:k])."""
        import torch

        k = self.schedule.k_at(epoch, self.d)
        _, lr = self.schedule.at(epoch)
        idx, vals = self.idx[:k], self.values[:k]
        if self.state == "sketch":
            self.ctx.step_sketch_momentum(grads, self.U, self.E, k, self.merged, idx, vals)
        elif self.selection == "heavymix":
            self.rnd.random_(-(1 << 31), 1 << 31, generator=self.gen)
            self.ctx.step_heavymix(grads, self.u, self.v, k, self.rnd, self.merged, idx, vals, n_heavy=self.n_heavy)
        else:
            self.ctx.step(grads, self.u, self.v, k, self.merged, idx, vals)
        self.ctx.apply_update(idx, vals, k, lr / self.P, w)
        return {"k": k, "lr": lr}

    def close(self):
        self.ctx.close()


class GlobalSketchOptimizer(torch.optim.Optimizer):
    """gs-SGD as a torch optimizer over fp32 CUDA parameters, with P simulated workers.

    Usage per iteration (Alg. 1 loop body): for each worker q, run its forward and backward
    pass on its own micro-batch and call ``collect(q)`` (copies the parameters' gradients into
    row q of the [P][d] gradient buffer and clears them); then ``step()``: the fused
    compression step of the library over the P rows (momentum and error accumulation,
    sketch, tree merge, top-k or HEAVYMIX selection, exact values and reset) and the update
    w <- w - (lr / P) * G~ on the selected coordinates (the values sum the P workers).
    ``set_epoch(e)`` picks the schedule's (density, lr) for the warm-up (Sec. IV).

    The parameters are moved into one flat buffer (``flat``) at construction; each
    parameter's ``data`` is then a view of it, so gs_apply_update writes them in place.
    """

    def __init__(self, params, num_workers: int, r: int, c: int, hash_params: dict, schedule: DensitySchedule,
                 rho: float = 0.9, reset_momentum: bool = True, selection: str = "topk", seed: int = 0,
                 state_layout: str = "interleaved"):
        params = [p for p in params]
        if not params:
            raise ValueError("no parameters")
        for p in params:
            if p.dtype != torch.float32 or not p.is_cuda:
                raise TypeError("GlobalSketchOptimizer needs fp32 CUDA parameters")
        if selection not in ("topk", "heavymix"):
            raise ValueError("selection must be 'topk' or 'heavymix'")
        super().__init__(params, {"lr": schedule.at(0)[1]})
        dev = params[0].device
        self.P = int(num_workers)
        self.d = sum(p.numel() for p in params)
        self.schedule, self.selection, self.epoch = schedule, selection, 0
        self.k_max = schedule.k_max(self.d)
        # one flat buffer holding every parameter; each parameter's data becomes a view of it
        self.flat = torch.empty(self.d, dtype=torch.float32, device=dev)
        self._views = []
        off = 0
        for p in params:
            n = p.numel()
            self.flat[off:off + n].copy_(p.data.reshape(-1))
            p.data = self.flat[off:off + n].view_as(p)
            self._views.append((p, off, n))
            off += n
        self.ctx = GsContext(self.d, self.P, r, c, self.k_max, hash_params, rho=rho, reset_momentum=reset_momentum,
                             state_layout=state_layout)
        f32 = dict(dtype=torch.float32, device=dev)
        self.grads = torch.zeros((self.P, self.d), **f32)
        self.u = torch.zeros(self.ctx.state_shape, **f32)
        self.v = torch.zeros_like(self.u)
        self.merged = torch.empty((r, c), **f32)
        self.idx = torch.empty(self.k_max, dtype=torch.int32, device=dev)
        self.values = torch.empty(self.k_max, **f32)
        self.last_k = 0
        if selection == "heavymix":
            self.gen = torch.Generator(device=dev)
            self.gen.manual_seed(seed)
            self.rnd = torch.empty(self.d, dtype=torch.int32, device=dev)
            self.n_heavy = torch.empty(1, dtype=torch.int64, device=dev)

    def set_epoch(self, epoch: int) -> None:
        self.epoch = int(epoch)

    @torch.no_grad()
    def collect(self, worker: int) -> None:
        """Copy the parameters' current gradients into row `worker` of the gradient buffer
        (zeros for a parameter without one) and clear them for the next worker's pass."""
        if not 0 <= worker < self.P:
            raise ValueError(f"worker must be in [0, {self.P})")
        row = self.grads[worker]
        for p, off, n in self._views:
            if p.grad is None:
                row[off:off + n].zero_()
            else:
                row[off:off + n].copy_(p.grad.reshape(-1))
                p.grad = None

    @torch.no_grad()
    def step(self, closure=None):
        loss = None
        if closure is not None:
            with torch.enable_grad():
                loss = closure()
        k = self.schedule.k_at(self.epoch, self.d)
        _, lr = self.schedule.at(self.epoch)
        for group in self.param_groups:
            group["lr"] = lr
        idx, vals = self.idx[:k], self.values[:k]
        if self.selection == "heavymix":
            self.rnd.random_(-(1 << 31), 1 << 31, generator=self.gen)
            self.ctx.step_heavymix(self.grads, self.u, self.v, k, self.rnd, self.merged, idx, vals,
                                   n_heavy=self.n_heavy)
        else:
            self.ctx.step(self.grads, self.u, self.v, k, self.merged, idx, vals)
        self.ctx.apply_update(idx, vals, k, lr / self.P, self.flat)
        self.last_k = k
        return loss

    def close(self):
        self.ctx.close()
