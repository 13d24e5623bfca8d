"""GPU-vs-oracle parity of HEAVYMIX as printed (Alg. 2): gs_heavymix_topk and the fused
gs_step_heavymix (needs an MI355X).

Bars: given an identical merged sketch and identical draws, the estimates, the
l2-norm-squared estimate, |H| and the selected index set are bit-exact (the heavy test
and the fill are integer decisions both sides take in the same precision, in the same
summation order). The fused step's values and u, v after the reset are bit-exact against
the oracle applied to its own selection; its merged sketch is within 1e-5 rel + 1e-7 abs.
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


def rnd_dev(rnd):
    return to_dev(np.ascontiguousarray(rnd, dtype=np.uint32).view(np.int32))


def host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


def assert_tol(gpu, ref, what):
    g64, r64 = np.asarray(gpu, np.float64), np.asarray(ref, np.float64)
    bad = np.abs(g64 - r64) > REL * np.abs(r64) + ABS
    assert not bad.any(), f"{what}: {int(bad.sum())} of {bad.size} outside 1e-5 rel + 1e-7 abs"


def gpu_heavymix(ctx, merged_d, d, k, rnd_d):
    est = torch.empty(d, dtype=torch.float32, device=DEV)
    idx = torch.empty(k, dtype=torch.int32, device=DEV)
    nh = torch.empty(1, dtype=torch.int64, device=DEV)
    l2 = torch.empty(1, dtype=torch.float64, device=DEV)
    ctx.heavymix_topk(merged_d, k, rnd_d, idx, est=est, n_heavy=nh, l2sq=l2)
    return host(idx), host(est), int(host(nh)[0]), float(host(l2)[0])


def check_identical_sketch(ctx, merged_h, hp, d, k, rnd, label):
    """GPU HEAVYMIX on a merged sketch vs the oracle on the same sketch and draws."""
    _flush(f"[{label}] heavymix k={k}")
    idx, est, nh, l2 = gpu_heavymix(ctx, to_dev(merged_h), d, k, rnd_dev(rnd))
    ref = oracle.heavymix(merged_h, hp, d, k, rnd)
    assert np.array_equal(est, ref["est"]), f"{label}: estimates not exact"
    assert l2 == ref["l2sq"], f"{label}: l2sq {l2!r} vs oracle {ref['l2sq']!r}"
    assert nh == ref["n_heavy"], f"{label}: |H| {nh} vs oracle {ref['n_heavy']}"
    assert np.array_equal(idx, ref["idx"]), f"{label}: selection differs ({np.setxor1d(idx, ref['idx']).size} indices)"
    # without an estimate vector the pruned pass runs (heavy-cell bitmap, sampled fill bound,
    # unpruned fallback when its candidates fall short of k): the same selection and |H|
    idx_p = torch.empty(k, dtype=torch.int32, device=DEV)
    nh_p = torch.empty(1, dtype=torch.int64, device=DEV)
    ctx.heavymix_topk(to_dev(merged_h), k, rnd_dev(rnd), idx_p, n_heavy=nh_p)
    assert np.array_equal(host(idx_p), ref["idx"]), f"{label}: pruned HEAVYMIX selection differs"
    assert int(host(nh_p)[0]) == ref["n_heavy"], f"{label}: pruned |H|"
    # the other selection path on the same context still works after a HEAVYMIX call
    idx_t = torch.empty(k, dtype=torch.int32, device=DEV)
    ctx.unsketch_topk(to_dev(merged_h), k, idx_t)
    assert np.array_equal(host(idx_t), oracle.topk(ref["est"], k)[0]), f"{label}: top-k after HEAVYMIX"
    return ref


# ---------------------------------------------------------------------------------------
# Workloads: the fused step from zero state, then the selection on its own merged sketch.

@pytest.mark.parametrize("name", ["t3planted-d65536-P4", "laplace20-d270000-P4", "t3scaled-d14.7M-P4",
                                  "laplace53-d25.6M-P8"])
def test_heavymix_fused_step_and_identical_sketch(name):
    w = synth.WORKLOADS[name]
    hp = synth.hash_params(w)
    ctx = gs.GsContext(w.d, w.P, w.r, w.c, w.k, hp, rho=w.rho)
    g = synth.gradients(w, 0)
    rnd = synth.fill_draws(w, 0)
    u_d = torch.zeros((w.P, w.d), dtype=torch.float32, device=DEV)
    v_d = torch.zeros_like(u_d)
    merged = torch.empty((w.r, w.c), dtype=torch.float32, device=DEV)
    idx = torch.empty(w.k, dtype=torch.int32, device=DEV)
    vals = torch.empty(w.k, dtype=torch.float32, device=DEV)
    nh = torch.empty(1, dtype=torch.int64, device=DEV)
    _flush(f"[{name}] fused HEAVYMIX step")
    ctx.step_heavymix(to_dev(g), u_d, v_d, w.k, rnd_dev(rnd), merged, idx, vals, n_heavy=nh)
    mg, jf, valf, nhf = host(merged), host(idx), host(vals), int(host(nh)[0])
    ref = check_identical_sketch(ctx, mg, hp, w.d, w.k, rnd, name)
    assert np.array_equal(jf, ref["idx"]) and nhf == ref["n_heavy"], f"{name}: fused selection"
    # values and reset: exact against the oracle's state after accumulation from zero (u = v = g)
    u1, v1 = np.zeros_like(g), np.zeros_like(g)
    oracle.accumulate(g, u1, v1, w.rho)
    vals_o = oracle.gather_reset(jf, u1, v1, True)
    assert np.array_equal(valf, vals_o), f"{name}: fused values"
    assert np.array_equal(host(u_d), u1) and np.array_equal(host(v_d), v1), f"{name}: fused u/v after reset"
    # the merged sketch against the oracle's sketch of the same state, and end to end
    _flush(f"[{name}] oracle sketch")
    v0 = np.zeros_like(g)
    u0 = np.zeros_like(g)
    oracle.accumulate(g, u0, v0, w.rho)
    om = oracle.merge(oracle.sketch(v0, hp, w.c))
    assert_tol(mg, om, f"{name}: merged sketch")
    if np.array_equal(mg, om):
        e2e = oracle.heavymix(om, hp, w.d, w.k, rnd)
        assert np.array_equal(jf, e2e["idx"]), f"{name}: end-to-end selection"
        _flush(f"[{name}] merged sketch bit-identical to the oracle's; end-to-end selection identical "
               f"(|H| = {nhf}, k = {w.k})")
    else:
        _flush(f"[{name}] merged sketch within tolerance, not bit-identical; |H| = {nhf}")
    ctx.close()


def test_heavymix_rowsparse_properties():
    # 66M coordinates: the estimates at 200,000 sampled coordinates, l2sq exactly, and the
    # selection characterised by properties that hold at any size.
    w = synth.WORKLOADS["rowsparse-d66M-P16"]
    hp = synth.hash_params(w)
    ctx = gs.GsContext(w.d, w.P, w.r, w.c, w.k, hp, rho=w.rho)
    g_d = to_dev(synth.gradients(w, 0))
    u_d = torch.zeros_like(g_d)
    v_d = torch.zeros_like(g_d)
    merged = torch.empty((w.r, w.c), dtype=torch.float32, device=DEV)
    idx = torch.empty(w.k, dtype=torch.int32, device=DEV)
    vals = torch.empty(w.k, dtype=torch.float32, device=DEV)
    rnd = synth.fill_draws(w, 0)
    _flush("[rowsparse] fused HEAVYMIX step")
    ctx.step_heavymix(g_d, u_d, v_d, w.k, rnd_dev(rnd), merged, idx, vals)
    mg, jf = host(merged), host(idx)
    del g_d, u_d, v_d
    sel, est, nh, l2 = gpu_heavymix(ctx, merged, w.d, w.k, rnd_dev(rnd))
    assert np.array_equal(sel, jf), "rowsparse: fused selection vs gs_heavymix_topk"
    smp = np.unique(np.concatenate([np.random.default_rng(5).integers(0, w.d, 200_000), sel]))
    assert np.array_equal(est[smp], oracle.unsketch_at(mg, hp, smp)), "rowsparse: estimates"
    assert l2 == oracle.l2sq_estimate(mg), "rowsparse: l2sq"
    heavy = est.astype(np.float64) ** 2 >= l2 / w.k
    assert nh == int(heavy.sum()), "rowsparse: |H|"
    assert sel.size == w.k and np.all(np.diff(sel) > 0), "rowsparse: idx"
    in_sel = np.zeros(w.d, bool)
    in_sel[sel] = True
    if nh >= w.k:
        assert np.all(heavy[sel]), "rowsparse: a non-heavy coordinate selected with |H| >= k"
    else:
        assert np.all(in_sel[heavy]), "rowsparse: a heavy coordinate left out"
        fill = sel[~heavy[sel]]
        assert fill.size == w.k - nh
        key = rnd >> np.uint32(1)
        t = key[fill].min()
        light = ~heavy
        assert np.all(in_sel[light & (key > t)]), "rowsparse: a larger draw left out of the fill"
        ties = np.flatnonzero(light & (key == t))
        n_take = int(np.count_nonzero(in_sel[ties]))
        assert np.array_equal(ties[:n_take], np.flatnonzero(in_sel & light & (key == t))), "rowsparse: fill ties"
    _flush(f"[rowsparse] |H| = {nh}, k = {w.k}")
    ctx.close()


# ---------------------------------------------------------------------------------------
# Edge shapes on synthetic merged sketches (no sketch step needed).

EDGE = [
    # d, r, c, k, kind
    (1, 1, 1, 1, "normal"),
    (37, 4, 5, 37, "normal"),           # k = d, even r
    (4099, 3, 64, 100, "spiky"),        # ragged d
    (20_000, 3, 50, 5_000, "normal"),   # narrow sketch: |H| > k
    (3001, 5, 97, 60, "spiky"),
    (1000, 5, 5_000_000, 10, "spiky"),  # c > 2048^2: three passes of the row-sum tree
    (65_536, 16, 3000, 655, "spiky"),   # maximum r, even
    (50_000, 5, 1000, 333, "zero"),     # l2sq = 0: every coordinate heavy
    (50_000, 5, 1000, 333, "equal"),    # all draws equal: the fill is the lowest indices
    (20_000, 5, 300, 20_000, "normal"),  # k = d > the sample: the pruned fill bound admits fewer
    (50_000, 3, 400, 45_000, "spiky"),   # than k coordinates, so the unpruned pass takes over
]


@pytest.mark.parametrize("d,r,c,k,kind", EDGE)
def test_heavymix_edge(d, r, c, k, kind):
    hp = synth.hash_params(synth.BASE_SEED + 29 * d + r, r)
    rng = np.random.default_rng(d + r + c)
    if kind == "zero":
        merged = np.zeros((r, c), np.float32)
    else:
        merged = rng.standard_normal((r, c)).astype(np.float32)
        if kind == "spiky":
            m = max(1, c // 50)
            merged[:, rng.integers(0, c, m)] *= 40.0
    rnd = synth.fill_draws(d + 7, 0, d)
    if kind == "equal":
        rnd[:] = 0xFFFFFFFF
    ctx = gs.GsContext(d, 2, r, c, k, hp)
    label = f"edge d={d} r={r} c={c} k={k} {kind}"
    ref = check_identical_sketch(ctx, merged, hp, d, k, rnd, label)
    if kind == "zero":
        assert ref["n_heavy"] == d and np.array_equal(ref["idx"], np.arange(k))
    # a second, smaller k on the same context (the selection state is per call)
    if k > 1:
        check_identical_sketch(ctx, merged, hp, d, max(1, k // 3), rnd, label + " (smaller k)")
    ctx.close()


def test_heavymix_rejects_invalid_arguments():
    w = synth.WORKLOADS["t3planted-d65536-P4"]
    hp = synth.hash_params(w)
    ctx = gs.GsContext(w.d, w.P, w.r, w.c, w.k, hp)
    merged = torch.zeros((w.r, w.c), dtype=torch.float32, device=DEV)
    idx = torch.empty(w.k, dtype=torch.int32, device=DEV)
    rnd = rnd_dev(synth.fill_draws(w, 0))
    with pytest.raises(gs.GsError) as e:
        gs.gs_heavymix_topk(ctx.handle, merged, w.k, None, None, idx, None, None)
    assert e.value.status == gs.GS_ERR_INVALID_ARG
    with pytest.raises(gs.GsError) as e:
        gs.gs_heavymix_topk(ctx.handle, merged, w.k + 1, rnd, None, idx, None, None)
    assert e.value.status == gs.GS_ERR_INVALID_ARG
    ctx.close()
