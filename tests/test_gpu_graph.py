"""The fused step captured in a HIP graph (torch.cuda.CUDAGraph) and replayed: no call of the
step allocates, synchronizes or clears memory with a memset node, so every replay must equal
the same step run eagerly. Replays are interleaved with unrelated eager work and host
synchronizations, and each is checked."""
import numpy as np
import pytest
import torch

import paper_2108_06004_amd as gs
import synth

pytestmark = pytest.mark.gpu
DEV = torch.device("cuda:0")


@pytest.mark.parametrize("layout", ["interleaved", "worker_major"])
@pytest.mark.parametrize("name", ["t3planted-d65536-P4", "laplace20-d270000-P4"])
def test_graph_replays_equal_eager_steps(name, layout):
    w = synth.WORKLOADS[name]
    hp = synth.hash_params(w)
    steps = 3
    gh = [synth.gradients(w, t % w.steps) for t in range(steps)]

    def fresh():
        ctx = gs.GsContext(w.d, w.P, w.r, w.c, w.k, hp, rho=w.rho, state_layout=layout)
        u = torch.zeros(ctx.state_shape, dtype=torch.float32, device=DEV)
        v = torch.zeros_like(u)
        bufs = dict(g=torch.empty((w.P, w.d), dtype=torch.float32, device=DEV),
                    merged=torch.empty((w.r, w.c), dtype=torch.float32, device=DEV),
                    idx=torch.empty(w.k, dtype=torch.int32, device=DEV),
                    vals=torch.empty(w.k, dtype=torch.float32, device=DEV))
        return ctx, u, v, bufs

    # eager reference: three steps, each output recorded
    ctx, u, v, b = fresh()
    ref = []
    for t in range(steps):
        b["g"].copy_(torch.from_numpy(gh[t]))
        ctx.step(b["g"], u, v, w.k, b["merged"], b["idx"], b["vals"])
        torch.cuda.synchronize()
        ref.append({k: x.clone() for k, x in dict(u=u, v=v, merged=b["merged"], idx=b["idx"], vals=b["vals"]).items()})
    ctx.close()

    # the same steps as replays of one captured step (fresh context and state)
    ctx, u, v, b = fresh()
    b["g"].copy_(torch.from_numpy(gh[0]))
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        ctx.step(b["g"], u, v, w.k, b["merged"], b["idx"], b["vals"])
    torch.cuda.synchronize()
    # capture records without running: the state is still zero
    assert not torch.any(u) and not torch.any(v), "capture ran the step"
    noise = torch.empty(1 << 20, dtype=torch.float32, device=DEV)
    for t in range(steps):
        b["g"].copy_(torch.from_numpy(gh[t]))
        noise.normal_()
        noise.mul_(3.0).add_(1.0)  # unrelated eager work between replays
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        got = dict(u=u, v=v, merged=b["merged"], idx=b["idx"], vals=b["vals"])
        for k in ref[t]:
            assert torch.equal(got[k], ref[t][k]), f"replay {t}: {k} differs from the eager step"
    del graph
    ctx.close()
    assert np.isfinite(noise.sum().item())
