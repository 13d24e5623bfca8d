"""GPU-vs-oracle parity on shapes whose sketch has rows with a swizzled LDS tile (needs an
MI355X). The pull places cell t of a tile at t ^ ((t >> s) & 31) when the step that at least
3/4 of consecutive coordinates take between scaled positions is a multiple of 2^s, s >= 2
(otherwise a run's cells would share a few LDS banks); the hash seeds below give such rows,
with s = 5 or more and with s = 2. The chain of checks is test_gpu_parity.chain_check's:
tables within 1e-5 relative + 1e-7 absolute of the oracle, everything else bit for bit, two
steps with the state carried over. The premise (a swizzled row) is checked on the host first
from the library's published rule: theta_j minimises the expected distance
(1 - f) |theta alpha|_c + f |theta (alpha - beta)|_c over theta coprime to c, f = a / p,
alpha = a mod c, beta = p mod c."""
import math

import numpy as np
import pytest

import synth
from test_gpu_parity import Dev, chain_check

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")

MERSENNE = (1 << 31) - 1


def swizzled_rows(hp, r, c):
    """{row: s} for the rows the library swizzles (common step a multiple of 2^s, s >= 2)."""
    rows = {}
    for j in range(r):
        a = int(hp["a"][j])
        alpha, beta, f = a % c, MERSENNE % c, a / MERSENNE
        if max(f, 1 - f) < 0.75:
            continue
        th = np.arange(1, min(c, 1 << 22), dtype=np.int64)
        s1, s2 = (th * alpha) % c, (th * ((alpha + c - beta) % c)) % c
        cost = (1 - f) * np.minimum(s1, c - s1) + f * np.minimum(s2, c - s2)
        theta = next(int(th[o]) for o in np.argsort(cost, kind="stable") if math.gcd(int(th[o]), c) == 1)
        step = alpha if f <= 0.5 else (alpha + c - beta) % c
        t = theta * step % c
        dist = min(t, c - t)
        if dist and (dist & 3) == 0:
            rows[j] = (dist & -dist).bit_length() - 1
    return rows


CASES = [
    # d, P, r, c, k, hash seed, layout (swizzled rows: row -> s)
    (300_007, 8, 5, 256_000, 500, 1014, "interleaved"),       # {0: 2, 4: 5}; two lanes per entry
    (300_007, 8, 5, 256_000, 500, 2001, "worker_major"),      # {1: 2}
    (200_003, 4, 4, 65_536, 300, 1022, "worker_major"),       # {2: 6}; one lane per entry
    (2_000_003, 4, 4, 65_536, 2_000, 2001, "interleaved"),    # {1: 2}; list segments (fp64 partials)
    (100_003, 16, 3, 100_000, 200, 1022, "interleaved"),      # {2: 5}; four lanes per entry
]


@pytest.mark.parametrize("d,P,r,c,k,seed,layout", CASES)
def test_swizzled_tile_rows(d, P, r, c, k, seed, layout):
    hp = synth.hash_params(seed, r)
    assert swizzled_rows(hp, r, c), "the shape must have a swizzled row"
    rng = np.random.default_rng(seed + d)
    dv = Dev(d, P, r, c, k, hp, 0.9, layout=layout)
    u = (rng.standard_normal((P, d)) * 1e-2).astype(np.float32)
    v = (rng.standard_normal((P, d)) * 1e-2).astype(np.float32)
    for t in range(2):
        g = rng.laplace(0.0, 1e-2, (P, d)).astype(np.float32)
        u, v = chain_check(dv, g, u, v, k, 0.9, label=f"swizzle d={d} P={P} r={r} c={c} seed={seed} {layout} t={t}")
    dv.close()
