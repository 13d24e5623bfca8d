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
