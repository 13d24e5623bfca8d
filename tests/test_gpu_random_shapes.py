"""Seeded random shapes through every entry point and the fused step against the oracle
(the comparison rules of test_gpu_parity.chain_check), two steps each with the state carried
over: sizes from one coordinate up to 2^18, P from 1 to 20 (beyond the unrolled kernels),
r from 1 to 16 (even r), c from 1 to twice d, k from 1 to d, both state layouts, the momentum
reset on and off. Plans vary with the shape: list segments per tile, packed and unpacked
lists, the interleaved row copy, the pruned selection with its fallback."""
import os

import numpy as np
import pytest

import synth
from test_gpu_parity import Dev, chain_check

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")

# GS_RANDOM_SHAPES=n runs the first n shapes of the same seeded sequence (default 32)
N_SHAPES = int(os.environ.get("GS_RANDOM_SHAPES", "32"))


def shape(n):
    rng = np.random.default_rng(9000 + n)
    d = int(np.exp(rng.uniform(0.0, np.log(1 << 18))))
    d = max(1, d)
    P = int(rng.integers(1, 21))
    r = int(rng.integers(1, 17))
    c = max(1, int(np.exp(rng.uniform(0.0, np.log(2 * d + 1)))))
    k = max(1, min(d, int(np.exp(rng.uniform(0.0, np.log(d + 1))))))
    layout = "interleaved" if rng.integers(2) else "worker_major"
    reset = bool(rng.integers(2))
    rho = float(np.float32(rng.uniform(0.0, 0.99)))
    return d, P, r, c, k, layout, reset, rho


@pytest.mark.parametrize("n", range(N_SHAPES))
def test_random_shape_two_steps(n):
    d, P, r, c, k, layout, reset, rho = shape(n)
    hp = synth.hash_params(synth.BASE_SEED + 7919 * n + 3, r)
    rng = np.random.default_rng(n)
    dv = Dev(d, P, r, c, k, hp, rho, reset_momentum=reset, layout=layout)
    u = (rng.standard_normal((P, d)) * 1e-2).astype(np.float32)
    v = (rng.standard_normal((P, d)) * 1e-2).astype(np.float32)
    for t in range(2):
        g = rng.laplace(0.0, 1e-2, (P, d)).astype(np.float32)
        u, v = chain_check(dv, g, u, v, k, rho, reset_momentum=reset,
                           label=f"random {n}: d={d} P={P} r={r} c={c} k={k} {layout} reset={reset} t={t}")
    dv.close()
