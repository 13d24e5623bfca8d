"""The fused steps captured in a HIP graph (torch.cuda.CUDAGraph) and replayed: no per-step call
allocates, synchronizes or clears memory with a memset node, so every replay must equal the
same step run eagerly. Replays are interleaved with unrelated eager work and host
synchronizations, and each is checked. Covered: gs_step (both state layouts),
gs_step_heavymix, gs_step_sketch_momentum and gs_unsketch_topk_static."""
import numpy as np
import pytest
import torch

import paper_2108_06004_amd as gs
import synth

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")
STEPS = 3


def make_run(w, entry, layout):
    """A fresh context, its buffers, and (load inputs of step t, run one step, outputs)."""
    hp = synth.hash_params(w)
    ctx = gs.GsContext(w.d, w.P, w.r, w.c, w.k, hp, rho=w.rho, state_layout=layout)
    f32 = dict(dtype=torch.float32, device=DEV)
    b = dict(g=torch.empty((w.P, w.d), **f32), merged=torch.empty((w.r, w.c), **f32),
             idx=torch.empty(w.k, dtype=torch.int32, device=DEV), vals=torch.empty(w.k, **f32))
    if entry == "sketch_momentum":
        b["U"] = torch.zeros((w.r, w.c), **f32)
        b["E"] = torch.zeros((w.r, w.c), **f32)
    else:
        b["u"] = torch.zeros(ctx.state_shape, **f32)
        b["v"] = torch.zeros(ctx.state_shape, **f32)
    if entry == "heavymix":
        b["rnd"] = torch.empty(w.d, dtype=torch.int32, device=DEV)
        b["nh"] = torch.zeros(1, dtype=torch.int64, device=DEV)
    grads = [torch.from_numpy(synth.gradients(w, t % w.steps)) for t in range(STEPS)]
    draws = [torch.from_numpy(synth.fill_draws(w, t).view(np.int32)) for t in range(STEPS)]

    def load(t):
        b["g"].copy_(grads[t])
        if entry == "heavymix":
            b["rnd"].copy_(draws[t])

    def run():
        if entry == "step":
            ctx.step(b["g"], b["u"], b["v"], w.k, b["merged"], b["idx"], b["vals"])
        elif entry == "heavymix":
            ctx.step_heavymix(b["g"], b["u"], b["v"], w.k, b["rnd"], b["merged"], b["idx"], b["vals"], n_heavy=b["nh"])
        else:
            ctx.step_sketch_momentum(b["g"], b["U"], b["E"], w.k, b["merged"], b["idx"], b["vals"])

    def outputs():
        return {k: x for k, x in b.items() if k not in ("g", "rnd")}

    return ctx, load, run, outputs


@pytest.mark.parametrize("entry,layout", [("step", "interleaved"), ("step", "worker_major"),
                                          ("heavymix", "interleaved"), ("sketch_momentum", "worker_major")])
@pytest.mark.parametrize("name", ["t3planted-d65536-P4", "laplace20-d270000-P4"])
def test_graph_replays_equal_eager_steps(name, entry, layout):
    w = synth.WORKLOADS[name]

    # eager reference: three steps, each output recorded
    ctx, load, run, outputs = make_run(w, entry, layout)
    ref = []
    for t in range(STEPS):
        load(t)
        run()
        torch.cuda.synchronize()
        ref.append({k: x.clone() for k, x in outputs().items()})
    ctx.close()

    # the same steps as replays of one captured step (fresh context and state)
    ctx, load, run, outputs = make_run(w, entry, layout)
    load(0)
    torch.cuda.synchronize()
    before = {k: x.clone() for k, x in outputs().items()}
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        run()
    torch.cuda.synchronize()
    # capture records without running: the state is untouched
    for k in ("u", "v", "U", "E"):
        if k in before:
            assert torch.equal(outputs()[k], before[k]), f"capture ran the step ({k} changed)"
    noise = torch.empty(1 << 20, dtype=torch.float32, device=DEV)
    for t in range(STEPS):
        load(t)
        noise.normal_()
        noise.mul_(3.0).add_(1.0)  # unrelated eager work between replays
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        got = outputs()
        for k in ref[t]:
            assert torch.equal(got[k], ref[t][k]), f"{entry}/{layout} replay {t}: {k} differs from the eager step"
    del graph
    ctx.close()
    assert np.isfinite(noise.sum().item())


def test_graph_replays_of_the_static_selection():
    # gs_unsketch_topk_static (no context, no allocation) captured once, after its first call
    # on the device looked up the scratch array, and replayed on new sketches: every replay
    # equals the eager call on the same sketch
    d, r, c, k = 270_000, 5, 27_000, 2_700
    hp = synth.hash_params(synth.BASE_SEED + 55, r)
    rng = np.random.default_rng(55)
    tables = [torch.from_numpy((np.round(rng.laplace(0.0, 1.0, (r, c)) * 64.0) / 64.0).astype(np.float32))
              for _ in range(STEPS)]
    m = torch.empty((r, c), dtype=torch.float32, device=DEV)
    est = torch.empty(d, dtype=torch.float32, device=DEV)
    idx = torch.empty(k, dtype=torch.int32, device=DEV)
    ref = []
    for t in range(STEPS):
        m.copy_(tables[t])
        gs.gs_unsketch_topk_static(d, r, c, hp, m, k, est, idx)
        torch.cuda.synchronize()
        ref.append((est.clone(), idx.clone()))
    m.copy_(tables[0])
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        gs.gs_unsketch_topk_static(d, r, c, hp, m, k, est, idx)
    torch.cuda.synchronize()
    noise = torch.empty(1 << 20, dtype=torch.float32, device=DEV)
    for t in range(STEPS):
        m.copy_(tables[t])
        noise.normal_()
        gs.gs_unsketch_topk_static(1000, 3, 97, synth.hash_params(synth.BASE_SEED + 56, 3), m[:3, :97].contiguous(),
                                   10, None, torch.empty(10, dtype=torch.int32, device=DEV))  # other eager use
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(est, ref[t][0]) and torch.equal(idx, ref[t][1]), f"static selection replay {t}"
    del graph
    assert np.isfinite(noise.sum().item())
