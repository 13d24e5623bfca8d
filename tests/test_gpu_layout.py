"""GPU-vs-oracle parity with the worker-interleaved state layout (u, v as [d][PP], PP = P
rounded up to a multiple of 4): every entry point that takes u or v, the fused steps, the
fp64-atomic sketch path, misaligned state views and the row padding (needs an MI355X).

Bars as for the worker-major layout: u and v after accumulation and after the reset, the
gathered values and every selection given identical inputs are bit-exact; tables and merged
sketches are within 1e-5 relative + 1e-7 absolute of the oracle. The oracle works on [P][d]
arrays; the tests rearrange the state on the way in and out.
"""
import numpy as np
import pytest

import oracle
import synth
from test_gpu_parity import DEV, Dev, assert_tol, chain_check, host, to_dev

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
gs = pytest.importorskip("paper_2108_06004_amd")

IL = "interleaved"


def _flush(msg):
    print(msg, flush=True)


@pytest.mark.parametrize("name", ["t3planted-d65536-P4", "laplace20-d270000-P4"])
def test_interleaved_small_workload_all_steps(name):
    w = synth.WORKLOADS[name]
    hp = synth.hash_params(w)
    dv = Dev(w.d, w.P, w.r, w.c, w.k, hp, w.rho, layout=IL)
    u = np.zeros((w.P, w.d), np.float32)
    v = np.zeros((w.P, w.d), np.float32)
    for t in range(w.steps):
        u, v = chain_check(dv, synth.gradients(w, t), u, v, w.k, w.rho, label=f"{name} interleaved step {t}")
    dv.close()


EDGE = [
    # d, P, r, c, k
    (1, 1, 1, 1, 1),
    (37, 3, 4, 5, 37),           # P = 3: rows padded to 4, ragged d
    (4099, 6, 3, 64, 100),       # P = 6: rows padded to 8 (generic accumulation)
    (10_007, 7, 7, 211, 500),
    (5_003, 12, 5, 300, 50),     # P = 12: three 16-byte groups per row (one idle lane per wave)
    (6_007, 11, 3, 257, 33),     # P = 11: rows padded to 12 (generic accumulation, masked pull lanes)
    (4_097, 16, 3, 128, 40),     # P = 16: four groups, ragged tail of the 16-coordinate chunks
    (5, 8, 3, 7, 2),             # P = 8: d below one 32-coordinate chunk (only the ragged one)
    (100_003, 8, 5, 5_003, 300), # P = 8: groups of four chunks, single chunks, then the ragged one
    (63, 4, 5, 17, 9),           # P = 4: d below one 64-coordinate chunk
    (3001, 17, 5, 97, 60),       # P beyond the unrolled pulls (rows of 20)
    (65_536, 4, 16, 4096, 655),  # P = 4: one group per coordinate, maximum r
]


@pytest.mark.parametrize("d,P,r,c,k", EDGE)
def test_interleaved_edge_shapes(d, P, r, c, k):
    hp = synth.hash_params(synth.BASE_SEED + 23 * d + P, r)
    rng = np.random.default_rng(d * 37 + P)
    dv = Dev(d, P, r, c, k, hp, 0.9, layout=IL)
    u = rng.standard_normal((P, d)).astype(np.float32)
    v = rng.standard_normal((P, d)).astype(np.float32)
    for t in range(2):
        g = rng.laplace(0, 1e-2, (P, d)).astype(np.float32)
        u, v = chain_check(dv, g, u, v, k, 0.9, label=f"interleaved d={d} P={P} r={r} c={c} k={k} t={t}")
    dv.close()


@pytest.mark.parametrize("d,P,r,c,k", [(10_007, 3, 5, 211, 300), (65_536, 8, 4, 4096, 655)])
def test_interleaved_atomic_sketch_path(monkeypatch, d, P, r, c, k):
    monkeypatch.setenv("GS_SKETCH_PATH", "atomic")
    hp = synth.hash_params(synth.BASE_SEED + 29 * d + P, r)
    rng = np.random.default_rng(d + 3 * P)
    dv = Dev(d, P, r, c, k, hp, 0.9, layout=IL)
    u = rng.standard_normal((P, d)).astype(np.float32)
    v = rng.standard_normal((P, d)).astype(np.float32)
    g = rng.laplace(0, 1e-2, (P, d)).astype(np.float32)
    chain_check(dv, g, u, v, k, 0.9, label=f"interleaved atomic d={d} P={P}")
    dv.close()


@pytest.mark.parametrize("P", [3, 8])
def test_interleaved_padding_untouched_and_misaligned_views(P):
    # padding entries hold a sentinel that must survive and never reach a result; then the
    # same step on state views that start one float into their buffers (not 16-byte
    # aligned: generic accumulation, and the pull reads an aligned copy)
    d, r, c, k = 20_011, 5, 400, 150
    hp = synth.hash_params(synth.BASE_SEED + 31 + P, r)
    rng = np.random.default_rng(40 + P)
    g = rng.laplace(0, 1e-2, (P, d)).astype(np.float32)
    u0 = rng.standard_normal((P, d)).astype(np.float32)
    v0 = rng.standard_normal((P, d)).astype(np.float32)
    ref = oracle.step(g, u0.copy(), v0.copy(), hp, c, k, rho=0.9, want_tables=False)
    kth = float(oracle.topk(ref["est"], k)[1])
    # a v view that is not 16-byte aligned needs the context's row copy (GS_OPT_ROW_COPY)
    plain = Dev(d, P, r, c, k, hp, 0.9, layout=IL)
    PP = gs.state_stride(P)
    mis = [torch.zeros((d * PP + 1,), dtype=torch.float32, device=DEV)[1:].view(d, PP) for _ in range(2)]
    with pytest.raises(gs.GsError) as e:
        plain.ctx.step(to_dev(g), mis[0], mis[1], k, plain.merged, plain.idx, plain.values)
    assert e.value.status == gs.GS_ERR_INVALID_ARG
    with pytest.raises(gs.GsError) as e:  # the sketch-space step needs the copy too
        U = torch.zeros((r, c), dtype=torch.float32, device=DEV)
        plain.ctx.step_sketch_momentum(to_dev(g), U, U.clone(), k, plain.merged, plain.idx, plain.values)
    assert e.value.status == gs.GS_ERR_UNSUPPORTED
    plain.close()
    dv = Dev(d, P, r, c, k, hp, 0.9, layout=IL, row_copy=True)
    for offset in (0, 1):
        _flush(f"[padding P={P} offset={offset}]")
        bufs = [torch.full((d * PP + offset,), 12345.0, dtype=torch.float32, device=DEV) for _ in range(2)]
        u_d, v_d = (b[offset:].view(d, PP) for b in bufs)
        u_d[:, :P] = to_dev(u0).t()
        v_d[:, :P] = to_dev(v0).t()
        dv.ctx.step(to_dev(g), u_d, v_d, k, dv.merged, dv.idx, dv.values)
        jf = host(dv.idx)
        uh, vh = host(u_d), host(v_d)
        if PP > P:
            assert np.all(uh[:, P:] == 12345.0) and np.all(vh[:, P:] == 12345.0), "padding was written"
        # selection: the oracle's except within the tie band; values and state exact for it
        sd = np.setxor1d(jf, ref["idx"])
        assert sd.size == 0 or np.all(np.abs(np.abs(ref["est"][sd].astype(np.float64)) - kth) <= 1e-6 * kth)
        uc, vc = u0.copy(), v0.copy()
        oracle.accumulate(g, uc, vc, 0.9)
        assert np.array_equal(host(dv.values), oracle.gather_reset(jf, uc, vc, True)), "values"
        assert np.array_equal(uh[:, :P].T, uc) and np.array_equal(vh[:, :P].T, vc), "state after the step"
        assert_tol(host(dv.merged), ref["merged"], f"padding P={P} offset={offset}: merged sketch")
    dv.close()


@pytest.mark.parametrize("name", ["t3planted-d65536-P4", "laplace53-d25.6M-P8"])
def test_interleaved_heavymix_step_matches_worker_major(name):
    # HEAVYMIX as printed: the interleaved step gives the worker-major step's outputs bit for
    # bit (the pull sums the same rows in the same order), and its values and reset are exact
    # against the oracle applied to the selection
    w = synth.WORKLOADS[name]
    hp = synth.hash_params(w)
    g = synth.gradients(w, 0)
    rnd = torch.from_numpy(synth.fill_draws(w, 0).view(np.int32)).to(DEV)
    outs = {}
    for layout in ("worker_major", IL):
        _flush(f"[{name}] HEAVYMIX step, {layout}")
        dv = Dev(w.d, w.P, w.r, w.c, w.k, hp, w.rho, layout=layout)
        z = np.zeros((w.P, w.d), np.float32)
        u_d, v_d = dv.state(z), dv.state(z)
        nh = torch.empty(1, dtype=torch.int64, device=DEV)
        dv.ctx.step_heavymix(to_dev(g), u_d, v_d, w.k, rnd, dv.merged, dv.idx, dv.values, n_heavy=nh)
        outs[layout] = (host(dv.merged), host(dv.idx), host(dv.values), int(host(nh)[0]), dv.unstate(u_d),
                        dv.unstate(v_d))
        dv.close()
    a, b = outs["worker_major"], outs[IL]
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1]) and a[3] == b[3], f"{name}: selection"
    u1, v1 = np.zeros_like(g), np.zeros_like(g)
    oracle.accumulate(g, u1, v1, w.rho)
    assert np.array_equal(b[2], oracle.gather_reset(b[1], u1, v1, True)), f"{name}: values"
    assert np.array_equal(b[4], u1) and np.array_equal(b[5], v1), f"{name}: state after the reset"
