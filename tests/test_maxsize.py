"""The largest coordinate count the bucket hash admits, d = 2^31 - 2, through every entry point.

At this size P*d (worker-major state), 4*d (interleaved rows) and r*d (the tile lists) all
exceed 2^32, so every flat index on the path is past 32 bits. The input is zero except 16
planted coordinates (the last three among them) holding small dyadic values, so every sum
on the path is exact and every comparison is bit for bit.

The expected results need no pass over d. A table cell is nonzero only when a planted
coordinate lands in it, so the only coordinates whose estimate can be nonzero are those
sharing such a cell in some row. The bucket hash is affine modulo p (Sec. III-A), so the
coordinates of one cell are the preimages of its p/c raw hash values: i = a^-1 (y - b) mod
p. The oracle estimates exactly that set; every other estimate is 0.
"""
import numpy as np
import pytest

import oracle
import synth

MERSENNE = 2**31 - 1
D_MAX = MERSENNE - 1
P, R, C, K_SEL = 2, 3, 1 << 20, 12
RHO = 0.9
PLANTED = np.array([D_MAX - 1, D_MAX - 2, D_MAX - 65, 2**31 - 1000, 3 * 2**29, 2**30, 2**30 - 1, 2**29 + 3,
                    10**9, 7 * 10**8, 123_456_789, 3 * 65_536 + 5, 4097, 63, 1, 0], dtype=np.int64)
SEED = synth.BASE_SEED + 31


def sharing(hp: dict, c: int, d: int, idx: np.ndarray) -> np.ndarray:
    """Ascending coordinates below d that share a bucket with a coordinate of idx in some row
    (idx included)."""
    out = [np.asarray(idx, dtype=np.int64)]
    for j in range(len(hp["a"])):
        a, b = int(hp["a"][j]), int(hp["b"][j])
        a_inv = pow(a, -1, MERSENNE)
        for col in np.unique(oracle.buckets(a, b, c, idx)):
            y = np.arange(int(col), MERSENNE, c, dtype=np.int64)  # raw hash values in this bucket
            i = (a_inv * ((y - b) % MERSENNE)) % MERSENNE         # < 2^62: exact in int64
            out.append(i[i < d])
    return np.unique(np.concatenate(out))


def planted_values() -> np.ndarray:
    """[P][16] fp32: worker q, planted coordinate m holds (-1)^m (16 - m)(q + 1) / 16, so the
    coordinates at the top of the range are the largest and are selected."""
    m = np.arange(PLANTED.size)
    q = np.arange(P)[:, None]
    return (np.where(m % 2 == 0, 1.0, -1.0) * (PLANTED.size - m) * (q + 1) / 16.0).astype(np.float32)


def expected(hp: dict) -> dict:
    """Every result of one step from zero state, from the oracle at the coordinates that can
    be nonzero."""
    gp = planted_values()
    tables = np.zeros((P, R, C), np.float32)
    for j in range(R):
        col = oracle.buckets(int(hp["a"][j]), int(hp["b"][j]), C, PLANTED)
        sg = oracle.signs(int(hp["a2"][j]), int(hp["b2"][j]), PLANTED)
        assert np.unique(col).size == PLANTED.size, "planted coordinates must not share a bucket"
        tables[:, j, col] = gp * sg  # each nonzero cell holds one signed value
    merged = oracle.merge(tables)
    cand = sharing(hp, C, D_MAX, PLANTED)
    est = oracle.unsketch_at(merged, hp, cand)
    pos, kth = oracle.topk(est, K_SEL)
    assert kth != 0, "the k-th estimate must be nonzero (zero estimates lie outside the candidate set)"
    at = np.searchsorted(cand, PLANTED)
    g = np.zeros((P, cand.size), np.float32)
    g[:, at] = gp
    u, v = np.zeros_like(g), np.zeros_like(g)
    oracle.accumulate(g, u, v, RHO)
    u_acc, v_acc = u.copy(), v.copy()
    values = oracle.gather_reset(pos, u, v)
    return dict(gp=gp, tables=tables, merged=merged, cand=cand, est=est, idx=cand[pos].astype(np.int32), values=values,
                u_acc=u_acc, v_acc=v_acc, u_end=u, v_end=v)


def test_sharing_matches_brute_force():
    # the preimage listing against every coordinate's bucket, on a size where all fit
    d, c = 2_000_003, 16_384
    hp = synth.hash_params(SEED + 1, 4)
    idx = np.array([0, 5, 1234, 999_999, d - 1], dtype=np.int64)
    everything = np.arange(d, dtype=np.int64)
    hit = np.zeros(d, bool)
    for j in range(4):
        a, b = int(hp["a"][j]), int(hp["b"][j])
        hit |= np.isin(oracle.buckets(a, b, c, everything), oracle.buckets(a, b, c, idx))
    assert np.array_equal(sharing(hp, c, d, idx), everything[hit])


def test_maximum_d_expectation_is_consistent():
    # host side of the GPU test: planted buckets distinct, the selection determined by
    # nonzero estimates, the planted estimates exact
    exp = expected(synth.hash_params(SEED, R))
    at = np.searchsorted(exp["cand"], PLANTED)
    planted_sums = np.array([oracle.tree_sum(exp["gp"][:, m]) for m in range(PLANTED.size)], np.float32)
    assert np.array_equal(exp["est"][at], planted_sums)
    assert np.count_nonzero(exp["est"]) >= K_SEL
    assert exp["cand"].size > PLANTED.size
    assert exp["idx"].dtype == np.int32 and exp["idx"][-1] == D_MAX - 1


@pytest.mark.gpu
@pytest.mark.parametrize("layout", ["worker_major", "interleaved"])
def test_maximum_d_every_entry_point(layout):
    torch = pytest.importorskip("torch")
    gs = pytest.importorskip("paper_2108_06004_amd")
    dev = "cuda:0"

    def say(msg):
        print(f"[max d {layout}] {msg}", flush=True)

    hp = synth.hash_params(SEED, R)
    exp = expected(hp)
    cand_t = torch.from_numpy(exp["cand"]).to(dev)
    f32 = dict(dtype=torch.float32, device=dev)

    def state_at(t):
        """[P][len(cand)] host copy of a state tensor at the candidate coordinates."""
        x = t[:, cand_t] if layout == "worker_major" else t[cand_t, :P].t()
        return x.cpu().numpy()

    def nnz(t):
        """Nonzero count in chunks of 2^28 elements (a whole-tensor count needs a temporary of
        8 bytes per element)."""
        flat = t.view(-1)
        return sum(int(torch.count_nonzero(flat[o:o + (1 << 28)]).item()) for o in range(0, flat.numel(), 1 << 28))

    def check_state(u, v, u_ref, v_ref, what):
        torch.cuda.synchronize()
        assert np.array_equal(state_at(u), u_ref), f"{what}: u at the candidate coordinates"
        assert np.array_equal(state_at(v), v_ref), f"{what}: v at the candidate coordinates"
        # every other coordinate (and the interleaved padding) holds exactly zero
        assert nnz(u) == np.count_nonzero(u_ref), f"{what}: u nonzero elsewhere"
        assert nnz(v) == np.count_nonzero(v_ref), f"{what}: v nonzero elsewhere"

    torch.cuda.empty_cache()
    say("gs_create (list build over r*d = 6.4e9 entries)")
    ctx = gs.GsContext(D_MAX, P, R, C, K_SEL, hp, rho=RHO, state_layout=layout)
    g = torch.zeros((P, D_MAX), **f32)
    g[:, torch.from_numpy(PLANTED).to(dev)] = torch.from_numpy(exp["gp"]).to(dev)
    u = torch.zeros(ctx.state_shape, **f32)
    v = torch.zeros(ctx.state_shape, **f32)

    say("accumulate")
    ctx.accumulate(g, u, v)
    check_state(u, v, exp["u_acc"], exp["v_acc"], "accumulate")

    say("sketch")
    tables = torch.empty((P, R, C), **f32)
    ctx.sketch(v, tables)
    torch.cuda.synchronize()
    assert np.array_equal(tables.cpu().numpy(), exp["tables"]), "worker tables"

    say("merge")
    merged = torch.empty((R, C), **f32)
    ctx.merge(tables, merged)
    torch.cuda.synchronize()
    assert np.array_equal(merged.cpu().numpy(), exp["merged"]), "merged sketch"
    del tables

    say("unsketch_topk with the estimate vector (every coordinate estimated)")
    est = torch.empty(D_MAX, **f32)
    idx = torch.empty(K_SEL, dtype=torch.int32, device=dev)
    ctx.unsketch_topk(torch.from_numpy(exp["merged"]).to(dev), K_SEL, idx, est=est)
    torch.cuda.synchronize()
    assert np.array_equal(idx.cpu().numpy(), exp["idx"]), "top-k from the full estimate"
    assert np.array_equal(est[cand_t].cpu().numpy(), exp["est"]), "estimates at the candidate coordinates"
    assert nnz(est) == np.count_nonzero(exp["est"]), "nonzero estimates elsewhere"
    del est

    say("gather_reset")
    values = torch.empty(K_SEL, **f32)
    ctx.gather_reset(torch.from_numpy(exp["idx"]).to(dev), K_SEL, u, v, values)
    torch.cuda.synchronize()
    assert np.array_equal(values.cpu().numpy(), exp["values"]), "gathered values"
    check_state(u, v, exp["u_end"], exp["v_end"], "gather_reset")

    say("fused step from zero state (pruned selection)")
    u.zero_()
    v.zero_()
    merged.fill_(7.0)
    idx.fill_(-1)
    values.fill_(7.0)
    ctx.step(g, u, v, K_SEL, merged, idx, values)
    torch.cuda.synchronize()
    assert np.array_equal(merged.cpu().numpy(), exp["merged"]), "fused step: merged sketch"
    assert np.array_equal(idx.cpu().numpy(), exp["idx"]), "fused step: top-k"
    assert np.array_equal(values.cpu().numpy(), exp["values"]), "fused step: gathered values"
    check_state(u, v, exp["u_end"], exp["v_end"], "fused step")
    say("done")
    ctx.close()
    del g, u, v
    torch.cuda.empty_cache()
