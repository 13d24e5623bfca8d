"""The training integration on the GPU: the weight update against the oracle, and
convergence of a noisy quadratic with the paper's warm-up schedule (needs an MI355X)."""
import numpy as np
import pytest

import oracle
import synth

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
gs = pytest.importorskip("paper_2108_06004_amd")
from paper_2108_06004_amd.train import DensitySchedule, GlobalSketchSGD  # noqa: E402

DEV = "cuda:0"


def host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


def test_apply_update_matches_oracle():
    d, k = 100_003, 5_000
    hp = synth.hash_params(synth.BASE_SEED + 91, 3)
    ctx = gs.GsContext(d, 2, 3, 1000, k, hp)
    rng = np.random.default_rng(91)
    w = rng.standard_normal(d).astype(np.float32)
    idx = np.sort(rng.choice(d, k, replace=False)).astype(np.int32)
    vals = rng.standard_normal(k).astype(np.float32)
    w_d = torch.from_numpy(w.copy()).to(DEV)
    ctx.apply_update(torch.from_numpy(idx).to(DEV), torch.from_numpy(vals).to(DEV), k, 0.037, w_d)
    oracle.apply_update(w, idx, vals, 0.037)
    assert np.array_equal(host(w_d), w)
    ctx.close()


def run_quadratic(opt, wstar, P, d, steps, noise, epoch_len, rng):
    w = torch.zeros(d, dtype=torch.float32, device=DEV)
    loss0 = 0.5 * float(torch.sum((w - wstar) ** 2))
    for t in range(steps):
        g = ((w - wstar).unsqueeze(0) +
             torch.from_numpy((noise * rng.standard_normal((P, d))).astype(np.float32)).to(DEV)).contiguous()
        w_before = host(w).copy()
        info = opt.step(g, w, epoch=t // epoch_len)
        k = info["k"]
        # the update touched exactly the selection, by fl(w - fl(lr/P * value))
        want = w_before.copy()
        oracle.apply_update(want, host(opt.idx)[:k], host(opt.values)[:k], info["lr"] / P)
        assert np.array_equal(host(w), want), t
    return 0.5 * float(torch.sum((w - wstar) ** 2)) / loss0


@pytest.mark.parametrize("selection,state", [("topk", "vector"), ("heavymix", "vector"), ("topk", "sketch")])
def test_sparse_optimum_converges(selection, state):
    # f(w) = |w - w*|^2 / 2 with 200 nonzero coordinates in w* (the gradients have heavy
    # hitters, which the sketch recovers), noise N(0, 0.01^2) per worker, density 0.4%
    d, P, r, c = 65_536, 4, 5, 8192
    hp = synth.hash_params(synth.BASE_SEED + 90, r)
    rng = np.random.default_rng(92)
    wstar = np.zeros(d, np.float32)
    wstar[rng.choice(d, 200, replace=False)] = 3 * rng.standard_normal(200).astype(np.float32)
    opt = GlobalSketchSGD(d, P, r, c, hp, DensitySchedule(0.004, 0.1), rho=0.5, selection=selection, state=state,
                          seed=6)
    rel = run_quadratic(opt, torch.from_numpy(wstar).to(DEV), P, d, 40, 0.01, 1000, rng)
    print(f"{selection}/{state}: loss {rel:.4f} of the initial", flush=True)
    assert rel < 0.01
    opt.close()


@pytest.mark.parametrize("selection", ["topk", "heavymix"])
def test_noisy_quadratic_converges_with_warmup(selection):
    # a dense optimum (no heavy hitters): only the vector-space state, whose values are exact,
    # descends here; the sketch-space state applies sketch estimates and needs heavy hitters
    # f(w) = |w - w*|^2 / 2, each worker's gradient (w - w*) plus N(0, 0.1^2) noise; warm-up
    # densities 0.25, 0.0725, 0.015, 0.004 for 10 steps each, then 0.001 (Sec. IV)
    d, P, r, c = 65_536, 4, 5, 8192
    hp = synth.hash_params(synth.BASE_SEED + 90, r)
    sched = DensitySchedule(0.001, 0.1, [(0.25, 0.1), (0.0725, 0.03), (0.015, 0.01), (0.004, 0.01)])
    opt = GlobalSketchSGD(d, P, r, c, hp, sched, rho=0.5, selection=selection, seed=5)
    rng = np.random.default_rng(90)
    wstar = torch.from_numpy(rng.standard_normal(d).astype(np.float32)).to(DEV)
    rel = run_quadratic(opt, wstar, P, d, 40, 0.1, 10, rng)
    print(f"{selection}/vector with warm-up: loss {rel:.3f} of the initial", flush=True)
    assert rel < 0.3
    opt.close()


def test_apply_update_rejects_invalid_arguments():
    hp = synth.hash_params(synth.BASE_SEED + 93, 3)
    ctx = gs.GsContext(1000, 2, 3, 100, 10, hp)
    idx = torch.arange(10, dtype=torch.int32, device=DEV)
    vals = torch.ones(10, dtype=torch.float32, device=DEV)
    w = torch.zeros(1000, dtype=torch.float32, device=DEV)
    for k, lr in ((11, 0.1), (0, 0.1), (10, float("nan")), (10, float("inf"))):
        with pytest.raises(gs.GsError) as e:
            gs.gs_apply_update(ctx.handle, idx, vals, k, lr, w)
        assert e.value.status == gs.GS_ERR_INVALID_ARG
    assert not host(w).any()
    ctx.close()


def test_optimizer_hook_on_a_module_matches_the_oracle_every_step():
    # a small MLP regressing a fixed random teacher (synthetic data, no dataset), P = 4
    # simulated workers on their own micro-batches, the warm-up schedule; at every step the
    # parameters after the update equal oracle.apply_update on the flat parameters before
    # it with the step's selection and values, bit for bit, and the step itself equals the
    # oracle's step from the same state (selection within the tie band, values and state
    # bit for bit)
    from paper_2108_06004_amd.train import GlobalSketchOptimizer

    torch.manual_seed(11)
    P, r, c, batch = 4, 5, 2048, 32
    model = torch.nn.Sequential(torch.nn.Linear(64, 256), torch.nn.Tanh(), torch.nn.Linear(256, 32)).to(DEV)
    teacher = torch.nn.Sequential(torch.nn.Linear(64, 32)).to(DEV)
    hp = synth.hash_params(synth.BASE_SEED + 94, r)
    sched = DensitySchedule(0.01, 0.05, [(0.25, 0.05), (0.05, 0.05)])
    opt = GlobalSketchOptimizer(model.parameters(), P, r, c, hp, sched, rho=0.9)
    d = opt.d
    assert d == sum(p.numel() for p in model.parameters()) == 64 * 256 + 256 + 256 * 32 + 32
    gen = torch.Generator(device=DEV)
    gen.manual_seed(3)
    losses = []
    for t in range(12):
        opt.set_epoch(t // 4)
        total = 0.0
        for q in range(P):
            x = torch.randn(batch, 64, device=DEV, generator=gen)
            with torch.no_grad():
                y = teacher(x)
            loss = ((model(x) - y) ** 2).mean()
            loss.backward()
            opt.collect(q)
            total += float(loss)
        losses.append(total / P)
        g = host(opt.grads).copy()
        u0, v0 = opt.ctx.from_state(opt.u).cpu().numpy(), opt.ctx.from_state(opt.v).cpu().numpy()
        w0 = host(opt.flat).copy()
        opt.step()
        k = opt.last_k
        lr = sched.at(t // 4)[1]
        idx, vals = host(opt.idx)[:k].copy(), host(opt.values)[:k].copy()
        want = w0.copy()
        oracle.apply_update(want, idx, vals, lr / P)
        assert np.array_equal(host(opt.flat), want), f"step {t}: update not bit-exact"
        assert torch.equal(torch.cat([p.detach().reshape(-1) for p in model.parameters()]), opt.flat)
        # the compression step from the same state
        uo, vo = u0.copy(), v0.copy()
        ref = oracle.step(g, uo, vo, hp, c, k, rho=0.9)
        kth = np.sort(np.abs(ref["est"]).astype(np.float64))[::-1][k - 1]
        sd = np.setxor1d(idx, ref["idx"])
        assert np.all(np.abs(np.abs(ref["est"][sd].astype(np.float64)) - kth) <= 1e-6 * kth), f"step {t}: selection"
        common, gi, oi = np.intersect1d(idx, ref["idx"], return_indices=True)
        assert np.array_equal(vals[gi], ref["values"][oi]), f"step {t}: values"
        if sd.size == 0:
            assert np.array_equal(opt.ctx.from_state(opt.u).cpu().numpy(), uo), f"step {t}: u"
            assert np.array_equal(opt.ctx.from_state(opt.v).cpu().numpy(), vo), f"step {t}: v"
    print(f"optimizer hook: loss {losses[0]:.4f} -> {losses[-1]:.4f}", flush=True)
    assert losses[-1] < losses[0]
    opt.close()
