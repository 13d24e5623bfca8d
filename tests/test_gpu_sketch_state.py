"""GPU-vs-oracle parity of gs_step_sketch_momentum: momentum and error accumulation kept in
the merged sketch (needs an MI355X).

Bars: the merged gradient sketch within 1e-5 rel + 1e-7 abs of the oracle's; given that
merged sketch (identical input), the updated U and E, the selection and its values are
bit-exact against the oracle. Multi-step runs re-sync the state from the oracle.
"""
import numpy as np
import pytest

import oracle
import synth

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
gs = pytest.importorskip("paper_2108_06004_amd")

DEV = "cuda:0"
REL, ABS = 1e-5, 1e-7


def _flush(msg):
    print(msg, flush=True)


def to_dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


def assert_tol(gpu, ref, what):
    g64, r64 = np.asarray(gpu, np.float64), np.asarray(ref, np.float64)
    bad = np.abs(g64 - r64) > REL * np.abs(r64) + ABS
    assert not bad.any(), f"{what}: {int(bad.sum())} of {bad.size} outside 1e-5 rel + 1e-7 abs"


def state_step(ctx, g, U0, E0, hp, k, rho, reset, label, check_sketch=True):
    """One GPU step from host state (U0, E0); returns the oracle's state after the step on
    the GPU's merged sketch (equal to the GPU's, checked)."""
    r, c = U0.shape
    d = g.shape[1]
    U_d, E_d = to_dev(U0), to_dev(E0)
    merged = torch.empty((r, c), dtype=torch.float32, device=DEV)
    idx = torch.empty(k, dtype=torch.int32, device=DEV)
    vals = torch.empty(k, dtype=torch.float32, device=DEV)
    _flush(f"[{label}] GPU step")
    ctx.step_sketch_momentum(to_dev(g), U_d, E_d, k, merged, idx, vals)
    mg = host(merged)
    if check_sketch:
        _flush(f"[{label}] oracle sketch")
        assert_tol(mg, oracle.merge(oracle.sketch(g, hp, c)), f"{label}: merged gradient sketch")
    _flush(f"[{label}] oracle state update")
    U1, E1 = U0.copy(), E0.copy()
    ref = oracle.sketch_state_update(mg, U1, E1, hp, d, k, rho=rho, reset_momentum=reset)
    assert np.array_equal(host(idx), ref["idx"]), f"{label}: selection"
    assert np.array_equal(host(vals), ref["values"]), f"{label}: values"
    assert np.array_equal(host(U_d), U1), f"{label}: U after the step"
    assert np.array_equal(host(E_d), E1), f"{label}: E after the step"
    return U1, E1


@pytest.mark.parametrize("name,steps", [("t3planted-d65536-P4", 1), ("laplace20-d270000-P4", 4),
                                        ("laplace53-d25.6M-P8", 2)])
def test_sketch_state_workloads(name, steps):
    w = synth.WORKLOADS[name]
    hp = synth.hash_params(w)
    ctx = gs.GsContext(w.d, w.P, w.r, w.c, w.k, hp, rho=w.rho)
    U = np.zeros((w.r, w.c), np.float32)
    E = np.zeros((w.r, w.c), np.float32)
    for t in range(steps):
        U, E = state_step(ctx, synth.gradients(w, t), U, E, hp, w.k, w.rho, True, f"{name} step {t}",
                          check_sketch=(t == 0 or w.d < 1_000_000))
    ctx.close()


def test_sketch_state_planted_coordinates_selected():
    # the 64 planted coordinates (+-0.4 summed over workers) dominate the sketch estimates
    w = synth.WORKLOADS["t3planted-d65536-P4"]
    hp = synth.hash_params(w)
    ctx = gs.GsContext(w.d, w.P, w.r, w.c, w.k, hp, rho=w.rho)
    U = torch.zeros((w.r, w.c), dtype=torch.float32, device=DEV)
    E = torch.zeros_like(U)
    merged = torch.empty_like(U)
    idx = torch.empty(w.k, dtype=torch.int32, device=DEV)
    vals = torch.empty(w.k, dtype=torch.float32, device=DEV)
    ctx.step_sketch_momentum(to_dev(synth.gradients(w, 0)), U, E, w.k, merged, idx, vals)
    pidx, psgn = synth.planted(w)
    sel = host(idx)
    assert np.isin(pidx, sel).all()
    pos = np.searchsorted(sel, pidx)
    assert np.all(np.abs(host(vals)[pos] - 0.4 * psgn) < 0.05)
    ctx.close()


EDGE = [
    # d, P, r, c, k, reset
    (1, 1, 1, 1, 1, True),
    (37, 3, 4, 5, 37, True),         # k = d, even r, d not a multiple of 4 (generic interleave)
    (4099, 6, 3, 1, 50, True),       # one column: every selected pair shares the cell
    (10_007, 7, 7, 211, 500, False),  # momentum kept
    (3001, 17, 5, 97, 60, True),     # P beyond the unrolled instances
    (65_536, 2, 16, 4096, 655, True),  # maximum r
    (200_003, 1, 5, 20_011, 300, True),  # one worker: its gradient vector is gathered directly
]


@pytest.mark.parametrize("d,P,r,c,k,reset", EDGE)
def test_sketch_state_edge(d, P, r, c, k, reset):
    hp = synth.hash_params(synth.BASE_SEED + 41 * d + P, r)
    rng = np.random.default_rng(d + 3 * P + r)
    ctx = gs.GsContext(d, P, r, c, k, hp, rho=0.9, reset_momentum=reset)
    U = rng.standard_normal((r, c)).astype(np.float32)
    E = rng.standard_normal((r, c)).astype(np.float32)
    for t in range(2):
        g = rng.laplace(0, 1e-2, (P, d)).astype(np.float32)
        U, E = state_step(ctx, g, U, E, hp, k, 0.9, reset, f"edge d={d} P={P} r={r} c={c} k={k} t={t}")
    ctx.close()


def test_sketch_state_rejects_invalid_arguments():
    w = synth.WORKLOADS["t3planted-d65536-P4"]
    hp = synth.hash_params(w)
    ctx = gs.GsContext(w.d, w.P, w.r, w.c, w.k, hp)
    U = torch.zeros((w.r, w.c), dtype=torch.float32, device=DEV)
    g = torch.zeros((w.P, w.d), dtype=torch.float32, device=DEV)
    idx = torch.empty(w.k, dtype=torch.int32, device=DEV)
    vals = torch.empty(w.k, dtype=torch.float32, device=DEV)
    with pytest.raises(gs.GsError) as e:
        gs.gs_step_sketch_momentum(ctx.handle, g, U, None, w.k, U, idx, vals)
    assert e.value.status == gs.GS_ERR_INVALID_ARG
    with pytest.raises(gs.GsError) as e:
        gs.gs_step_sketch_momentum(ctx.handle, g, U, U.clone(), w.k + 1, U.clone(), idx, vals)
    assert e.value.status == gs.GS_ERR_INVALID_ARG
    ctx.close()


def test_sketch_state_atomic_sketch_path(monkeypatch):
    monkeypatch.setenv("GS_SKETCH_PATH", "atomic")
    d, P, r, c, k = 20_000, 4, 5, 700, 150
    hp = synth.hash_params(synth.BASE_SEED + 77, r)
    rng = np.random.default_rng(77)
    ctx = gs.GsContext(d, P, r, c, k, hp, rho=0.9)
    U = np.zeros((r, c), np.float32)
    E = np.zeros((r, c), np.float32)
    for t in range(3):
        g = rng.standard_normal((P, d)).astype(np.float32)
        U, E = state_step(ctx, g, U, E, hp, k, 0.9, True, f"atomic sketch state t={t}")
    ctx.close()


def test_sketch_state_one_worker_interleaved_context():
    # with one worker the gradient [1][d] is a plain vector the pull gathers, so an
    # interleaved-state context runs the sketch-space step without the row copy
    d, P, r, c, k = 100_003, 1, 5, 10_007, 200
    hp = synth.hash_params(synth.BASE_SEED + 61, r)
    rng = np.random.default_rng(61)
    ctx = gs.GsContext(d, P, r, c, k, hp, rho=0.9, state_layout="interleaved")
    U = np.zeros((r, c), np.float32)
    E = np.zeros((r, c), np.float32)
    for t in range(2):
        g = rng.laplace(0, 1e-2, (P, d)).astype(np.float32)
        U, E = state_step(ctx, g, U, E, hp, k, 0.9, True, f"one worker interleaved t={t}")
    ctx.close()
