"""Pins of the CPU oracle against what the paper and the mathematics fix (no GPU).

Each test ties one oracle function to something other than itself: hand-worked examples
(``tests/golden``), closed forms, invariants of the Count Sketch (linearity, S = C x),
exact recovery cases, and brute force on tiny inputs. A plausible mistake in any oracle
function (wrong modulus, dropped sign, transposed operand, wrong merge order, fused
multiply-add, wrong median or tie rule) fails at least one of them.
"""
import itertools
import os

import numpy as np
import pytest

import oracle
import synth

P31 = (1 << 31) - 1


def _read_golden(path):
    rows = []
    with open(path) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                rows.append(line.split())
    return rows


def _hp(rng, r):
    return {
        "a": rng.integers(1, P31, r, dtype=np.int64).astype(np.uint32),
        "b": rng.integers(0, P31, r, dtype=np.int64).astype(np.uint32),
        "a2": rng.integers(1, P31, r, dtype=np.int64).astype(np.uint32),
        "b2": rng.integers(0, P31, r, dtype=np.int64).astype(np.uint32),
    }


# ---------------------------------------------------------------------------------------
# Hash families (Count Sketch, Sec. III-A)

def test_hash_worked_examples(golden_dir):
    for a, b, c, i, raw, bucket, sign in _read_golden(os.path.join(golden_dir, "hash_worked_examples.txt")):
        a, b, c, i = int(a), int(b), int(c), int(i)
        assert oracle.hash_raw(a, b, [i])[0] == int(raw)
        assert oracle.buckets(a, b, c, [i])[0] == int(bucket)
        assert oracle.signs(a, b, [i])[0] == int(sign)


def test_hash_is_an_affine_progression_mod_p():
    # raw(i+1) - raw(i) = a (mod p) for every i: catches a wrong modulus or a dropped b.
    rng = np.random.default_rng(1)
    for _ in range(20):
        a, b = int(rng.integers(1, P31)), int(rng.integers(0, P31))
        i = np.concatenate([rng.integers(0, P31 - 1, 500), [0, P31 - 2]])
        r0 = oracle.hash_raw(a, b, i).astype(object)
        r1 = oracle.hash_raw(a, b, i + 1).astype(object)
        assert all((int(y) - int(x) - a) % P31 == 0 for x, y in zip(r0, r1))
        assert all(0 <= int(x) < P31 for x in r0)
        assert oracle.hash_raw(a, b, [0])[0] == b


def test_bucket_range_and_uniformity():
    rng = np.random.default_rng(2)
    a, b = int(rng.integers(1, P31)), int(rng.integers(0, P31))
    c = 97
    h = oracle.buckets(a, b, c, np.arange(200_000))
    assert h.min() >= 0 and h.max() < c
    counts = np.bincount(h, minlength=c)
    chi2 = ((counts - 200_000 / c) ** 2 / (200_000 / c)).sum()
    assert chi2 < 200  # 96 degrees of freedom; a broken hash gives thousands
    s = oracle.signs(a, b, np.arange(200_000))
    assert set(np.unique(s)) == {-1, 1}
    assert abs(s.mean()) < 0.01


# ---------------------------------------------------------------------------------------
# Accumulation (momentum + error feedback)

def test_accumulate_zero_state_gives_g_exactly():
    g = np.random.default_rng(3).standard_normal((3, 1000)).astype(np.float32)
    u = np.zeros_like(g)
    v = np.zeros_like(g)
    oracle.accumulate(g, u, v, 0.9)
    assert np.array_equal(u, g) and np.array_equal(v, g)


def test_accumulate_constant_gradient_geometric_series():
    # u_t = g (1 - rho^t) / (1 - rho), v_t = sum_{s<=t} u_s, within fp32 rounding.
    rho = np.float32(0.9)
    g = np.full((1, 64), 0.25, dtype=np.float32)
    u = np.zeros_like(g)
    v = np.zeros_like(g)
    for t in range(1, 31):
        oracle.accumulate(g, u, v, float(rho))
        ut = 0.25 * (1 - float(rho) ** t) / (1 - float(rho))
        vt = sum(0.25 * (1 - float(rho) ** s) / (1 - float(rho)) for s in range(1, t + 1))
        assert np.allclose(u, ut, rtol=1e-5) and np.allclose(v, vt, rtol=1e-5)


def test_accumulate_rho_zero_sums_gradients_exactly():
    rng = np.random.default_rng(4)
    gs = [rng.integers(-50, 50, (2, 100)).astype(np.float32) for _ in range(5)]
    u = np.zeros((2, 100), np.float32)
    v = np.zeros((2, 100), np.float32)
    for g in gs:
        oracle.accumulate(g, u, v, 0.0)
    assert np.array_equal(v, np.sum(gs, axis=0)) and np.array_equal(u, gs[-1])


def test_accumulate_rounds_each_operation_to_fp32():
    # IEEE binary32 evaluation of fl(fl(rho*u) + g) then fl(v + u); a fused multiply-add
    # (a single rounding of rho*u + g) differs on a sizeable fraction of random inputs.
    rng = np.random.default_rng(5)
    u0 = rng.standard_normal(100_000).astype(np.float32)
    g = rng.standard_normal(100_000).astype(np.float32)
    v0 = rng.standard_normal(100_000).astype(np.float32)
    u, v = u0.copy(), v0.copy()
    oracle.accumulate(g, u, v, 0.9)
    rho = np.float32(0.9)
    u_ref = (rho * u0) + g
    assert np.array_equal(u, u_ref)
    assert np.array_equal(v, v0 + u_ref)
    fused = (np.float64(rho) * u0.astype(np.float64) + g.astype(np.float64)).astype(np.float32)
    assert np.count_nonzero(fused != u_ref) > 100  # the test can tell the two apart


# ---------------------------------------------------------------------------------------
# Count Sketch insertion

def _explicit_C(hp, c, d):
    """The sketching matrix C (r*c x d) with one signed 1 per row block and column."""
    r = len(hp["a"])
    C = np.zeros((r * c, d))
    i = np.arange(d)
    for j in range(r):
        h = oracle.buckets(int(hp["a"][j]), int(hp["b"][j]), c, i)
        s = oracle.signs(int(hp["a2"][j]), int(hp["b2"][j]), i)
        C[j * c + h, i] = s
    return C


def test_sketch_equals_matrix_product():
    # S(x) = C x (Sec. III-A): the scatter must agree with a dense matrix product.
    rng = np.random.default_rng(6)
    d, c, r, P = 300, 17, 4, 3
    hp = _hp(rng, r)
    v = rng.standard_normal((P, d)).astype(np.float32)
    C = _explicit_C(hp, c, d)
    S = oracle.sketch(v, hp, c)
    for q in range(P):
        ref = (C @ v[q].astype(np.float64)).astype(np.float32).reshape(r, c)
        assert np.array_equal(S[q], ref)


def test_sketch_linearity_bit_exact_on_integers():
    rng = np.random.default_rng(7)
    d, c, r = 5000, 61, 5
    hp = _hp(rng, r)
    a = rng.integers(-1000, 1000, (1, d)).astype(np.float32)
    b = rng.integers(-1000, 1000, (1, d)).astype(np.float32)
    assert np.array_equal(oracle.sketch(a, hp, c) + oracle.sketch(b, hp, c), oracle.sketch(a + b, hp, c))


def test_sketch_single_spike():
    rng = np.random.default_rng(8)
    d, c, r = 1000, 50, 5
    hp = _hp(rng, r)
    i, alpha = 637, np.float32(3.25)
    x = np.zeros((1, d), np.float32)
    x[0, i] = alpha
    S = oracle.sketch(x, hp, c)[0]
    for j in range(r):
        h = oracle.buckets(int(hp["a"][j]), int(hp["b"][j]), c, [i])[0]
        s = oracle.signs(int(hp["a2"][j]), int(hp["b2"][j]), [i])[0]
        expect = np.zeros(c, np.float32)
        expect[h] = s * alpha
        assert np.array_equal(S[j], expect)


def test_sketch_row_sums_and_l1_bound():
    rng = np.random.default_rng(9)
    d, c, r = 20_000, 301, 3
    hp = _hp(rng, r)
    x = rng.standard_normal((1, d)).astype(np.float32)
    S = oracle.sketch(x, hp, c)[0].astype(np.float64)
    i = np.arange(d)
    for j in range(r):
        s = oracle.signs(int(hp["a2"][j]), int(hp["b2"][j]), i)
        assert abs(S[j].sum() - (s * x[0].astype(np.float64)).sum()) < 1e-4
        assert np.abs(S[j]).sum() <= np.abs(x).sum() * (1 + 1e-6)


def test_sketch_cells_match_full_sketch():
    rng = np.random.default_rng(10)
    d, c, r, P = 4000, 97, 3, 2
    hp = _hp(rng, r)
    v = rng.standard_normal((P, d)).astype(np.float32)
    S = oracle.sketch(v, hp, c)
    rows = np.array([0, 0, 1, 2, 2])
    cols = np.array([0, 96, 40, 3, 5])
    cells = oracle.sketch_cells(v, hp, c, rows, cols)
    assert np.array_equal(cells, S[:, rows, cols].T)


# ---------------------------------------------------------------------------------------
# Merge in the binomial-tree order of Alg. 1

def test_merge_tree_order_worked_pairs(golden_dir):
    for row in _read_golden(os.path.join(golden_dir, "merge_tree_pairs.txt")):
        P = int(row[0])
        meet = set() if row[1] == "-" else {tuple(int(t) for t in p.split(",")) for p in row[1:]}
        for m, n in itertools.combinations(range(1, P), 2):
            x = np.zeros((P, 1, 2), np.float32)
            x[0] = 2.0 ** 24
            x[m] = 1.0
            x[n] = 1.0
            expect = np.float32(2.0 ** 24 + 2) if (m, n) in meet else np.float32(2.0 ** 24)
            merged = oracle.merge(x)
            assert merged[0, 0] == expect, (P, m, n)
            assert oracle.tree_sum(x[:, 0, 0]) == expect, (P, m, n)


def test_merge_p4_non_associative_example():
    # (1 + 2^24) + (1 - 2^24) = 1 under the tree; left to right gives 0, right to left 2.
    x = np.array([1.0, 2.0 ** 24, 1.0, -(2.0 ** 24)], np.float32).reshape(4, 1, 1)
    assert oracle.merge(x)[0, 0] == 1.0


def test_merge_integer_inputs_equal_plain_sum_and_identity():
    rng = np.random.default_rng(11)
    for P in range(1, 18):
        x = rng.integers(-10_000, 10_000, (P, 3, 50)).astype(np.float32)
        assert np.array_equal(oracle.merge(x), x.sum(axis=0, dtype=np.float64).astype(np.float32))
    x = rng.standard_normal((1, 4, 9)).astype(np.float32)
    assert np.array_equal(oracle.merge(x), x[0])


# ---------------------------------------------------------------------------------------
# Estimate (HEAVYMIX query, Alg. 2)

def _collision_free_support(hp, c, d, m, rng):
    """m coordinates no two of which share a bucket in any row."""
    r = len(hp["a"])
    used = [set() for _ in range(r)]
    chosen = []
    for i in rng.permutation(d):
        hs = [int(oracle.buckets(int(hp["a"][j]), int(hp["b"][j]), c, [i])[0]) for j in range(r)]
        if all(h not in used[j] for j, h in enumerate(hs)):
            chosen.append(int(i))
            for j, h in enumerate(hs):
                used[j].add(h)
            if len(chosen) == m:
                return np.array(chosen)
    raise AssertionError("not enough collision-free coordinates")


def test_unsketch_exact_recovery_of_collision_free_sparse_vector():
    rng = np.random.default_rng(12)
    d, c, r = 5000, 400, 5
    hp = _hp(rng, r)
    K = _collision_free_support(hp, c, d, 60, rng)
    x = np.zeros((1, d), np.float32)
    x[0, K] = rng.standard_normal(K.size).astype(np.float32) * 10
    est = oracle.unsketch(oracle.sketch(x, hp, c)[0], hp, d)
    assert np.array_equal(est[K], x[0, K])


def test_unsketch_majority_collision_free():
    # If a strict majority of i's buckets hold i alone, the median returns x_i exactly.
    rng = np.random.default_rng(13)
    d, c, r = 3000, 2000, 5
    hp = _hp(rng, r)
    x = np.zeros((1, d), np.float32)
    sup = rng.choice(d, 200, replace=False)
    x[0, sup] = rng.standard_normal(200).astype(np.float32)
    est = oracle.unsketch(oracle.sketch(x, hp, c)[0], hp, d)
    H = np.stack([oracle.buckets(int(hp["a"][j]), int(hp["b"][j]), c, sup) for j in range(r)])
    checked = 0
    for t, i in enumerate(sup):
        alone = sum(int(np.count_nonzero(H[j] == H[j, t]) == 1) for j in range(r))
        if alone >= 3:
            assert est[i] == x[0, i]
            checked += 1
    assert checked > 100


def test_unsketch_r1_is_single_signed_lookup():
    rng = np.random.default_rng(14)
    d, c = 2000, 100
    hp = _hp(rng, 1)
    S = rng.standard_normal((1, c)).astype(np.float32)
    i = np.arange(d)
    h = oracle.buckets(int(hp["a"][0]), int(hp["b"][0]), c, i)
    s = oracle.signs(int(hp["a2"][0]), int(hp["b2"][0]), i)
    assert np.array_equal(oracle.unsketch(S, hp, d), (s * S[0, h]).astype(np.float32))


def test_unsketch_median_matches_numpy_for_odd_and_even_r():
    rng = np.random.default_rng(15)
    d, c = 3000, 37
    for r in (1, 2, 3, 4, 5, 6, 7):
        hp = _hp(rng, r)
        S = rng.standard_normal((r, c)).astype(np.float32)
        i = np.arange(d)
        vals = np.stack([oracle.signs(int(hp["a2"][j]), int(hp["b2"][j]), i)
                         * S[j, oracle.buckets(int(hp["a"][j]), int(hp["b"][j]), c, i)] for j in range(r)])
        srt = np.sort(vals.astype(np.float32), axis=0)
        ref = srt[r // 2] if r % 2 else (srt[r // 2 - 1] + srt[r // 2]) * np.float32(0.5)
        assert np.array_equal(oracle.unsketch(S, hp, d), ref)
        sel = rng.integers(0, d, 50)
        assert np.array_equal(oracle.unsketch_at(S, hp, sel), ref[sel])


def test_count_sketch_error_statistic():
    # Count Sketch approximates every coordinate within about ||x||_2 / sqrt(c) (Sec. III-A):
    # errors beyond 3 ||x||_2 / sqrt(c) are rare.
    rng = np.random.default_rng(16)
    d, c, r = 50_000, 2000, 5
    hp = _hp(rng, r)
    x = rng.laplace(0, 1, (1, d)).astype(np.float32)
    est = oracle.unsketch(oracle.sketch(x, hp, c)[0], hp, d)
    bound = 3 * np.linalg.norm(x) / np.sqrt(c)
    assert np.mean(np.abs(est - x[0]) > bound) < 0.01


# ---------------------------------------------------------------------------------------
# Top_k (Alg. 2 selection: the largest elements by magnitude)

def test_topk_brute_force_tiny():
    rng = np.random.default_rng(17)
    for d in (1, 2, 7, 64, 513, 4096):
        est = rng.standard_normal(d).astype(np.float32)
        est[rng.integers(0, d, d // 3)] = 0.5  # plenty of exact ties
        est[rng.integers(0, d, d // 5)] = -0.5
        for k in sorted({1, max(1, d // 10), max(1, d // 2), d}):
            order = sorted(range(d), key=lambda i: (-abs(float(est[i])), i))
            idx, kth = oracle.topk(est, k)
            assert list(idx) == sorted(order[:k]), (d, k)
            assert kth == abs(est[order[k - 1]])


def test_topk_all_zero_and_k_equals_d():
    est = np.zeros(1000, np.float32)
    assert np.array_equal(oracle.topk(est, 17)[0], np.arange(17))
    est = np.random.default_rng(18).standard_normal(100).astype(np.float32)
    assert np.array_equal(oracle.topk(est, 100)[0], np.arange(100))


def test_topk_recovers_heavy_hitters_with_wide_sketch():
    # With c >> d every coordinate is majority-collision-free, so the sketch top-k equals the
    # brute-force top-k of the summed error vectors.
    rng = np.random.default_rng(19)
    d, c, r, P, k = 256, 65536, 5, 3, 20
    hp = _hp(rng, r)
    v = rng.standard_normal((P, d)).astype(np.float32)
    merged = oracle.merge(oracle.sketch(v, hp, c))
    idx, _ = oracle.topk(oracle.unsketch(merged, hp, d), k)
    total = v.astype(np.float64).sum(axis=0)
    assert set(idx) == set(np.argsort(-np.abs(total), kind="stable")[:k])


# ---------------------------------------------------------------------------------------
# Exact values and reset (Alg. 2, second round)

def test_gather_reset_tree_sums_and_masks():
    rng = np.random.default_rng(20)
    P, d = 6, 500
    u = rng.standard_normal((P, d)).astype(np.float32)
    v = rng.standard_normal((P, d)).astype(np.float32)
    idx = np.sort(rng.choice(d, 40, replace=False)).astype(np.int32)
    u0, v0 = u.copy(), v.copy()
    vals = oracle.gather_reset(idx, u, v, True)
    for t, i in enumerate(idx):
        col = v0[:, i]
        expect = ((col[0] + col[1]) + (col[2] + col[3])) + (col[4] + col[5])  # P=6 tree
        assert vals[t] == np.float32(expect)
    mask = np.zeros(d, bool)
    mask[idx] = True
    assert np.all(u[:, mask] == 0) and np.all(v[:, mask] == 0)
    assert np.array_equal(u[:, ~mask], u0[:, ~mask]) and np.array_equal(v[:, ~mask], v0[:, ~mask])
    u2, v2 = u0.copy(), v0.copy()
    oracle.gather_reset(idx, u2, v2, False)
    assert np.array_equal(u2, u0) and np.all(v2[:, mask] == 0)


# ---------------------------------------------------------------------------------------
# Whole step

def test_tiny_step_worked_by_hand(golden_dir):
    f = {row[0]: row[1:] for row in _read_golden(os.path.join(golden_dir, "tiny_step_worked.txt"))}
    d, P, r, c, k = (int(f[n][0]) for n in ("d", "P", "r", "c", "k"))
    rho = float(f["rho"][0])
    hp = {n: np.array([int(t) for t in f[n]], np.uint32) for n in ("a", "b", "a2", "b2")}
    arr = lambda n: np.array([float(t) for t in f[n]], np.float32)
    g = np.stack([arr("g0"), arr("g1")])
    u = np.zeros_like(g)
    v = np.zeros_like(g)
    res = oracle.step(g, u, v, hp, c, k, rho=rho)
    assert np.array_equal(res["tables"][0].ravel(), arr("tables0"))
    assert np.array_equal(res["tables"][1].ravel(), arr("tables1"))
    assert np.array_equal(res["merged"].ravel(), arr("merged"))
    assert np.array_equal(res["est"], arr("est"))
    assert np.array_equal(res["idx"], arr("idx").astype(np.int32))
    assert np.array_equal(res["values"], arr("values"))
    assert np.array_equal(v[0], arr("v0_after")) and np.array_equal(v[1], arr("v1_after"))
    assert np.array_equal(u, v)
    oracle.accumulate(g, u, v, rho)
    assert np.array_equal(u[0], arr("u0_step2")) and np.array_equal(u[1], arr("u1_step2"))
    assert np.array_equal(v[0], arr("v0_step2")) and np.array_equal(v[1], arr("v1_step2"))


def test_step_composes_the_five_functions():
    rng = np.random.default_rng(21)
    P, d, r, c, k = 3, 3000, 5, 200, 30
    hp = _hp(rng, r)
    g = rng.standard_normal((P, d)).astype(np.float32)
    u = rng.standard_normal((P, d)).astype(np.float32)
    v = rng.standard_normal((P, d)).astype(np.float32)
    u1, v1 = u.copy(), v.copy()
    res = oracle.step(g, u, v, hp, c, k)
    oracle.accumulate(g, u1, v1)
    tables = oracle.sketch(v1, hp, c)
    merged = oracle.merge(tables)
    est = oracle.unsketch(merged, hp, d)
    idx, _ = oracle.topk(est, k)
    vals = oracle.gather_reset(idx, u1, v1)
    for a, b in ((res["tables"], tables), (res["merged"], merged), (res["est"], est), (res["idx"], idx),
                 (res["values"], vals), (u, u1), (v, v1)):
        assert np.array_equal(a, b)


def test_planted_workload_selects_every_planted_coordinate():
    # 64 coordinates planted at +-0.1 on all 4 workers (sum +-0.4) against Student-t noise
    # of scale 1e-3 are heavy hitters; the Count Sketch guarantee (Sec. III-A) puts them in
    # Top_k, with exact values near +-0.4.
    w = synth.WORKLOADS["t3planted-d65536-P4"]
    hp = synth.hash_params(w)
    g = synth.gradients(w, 0)
    u = np.zeros_like(g)
    v = np.zeros_like(g)
    res = oracle.step(g, u, v, hp, w.c, w.k)
    pidx, psgn = synth.planted(w)
    assert np.isin(pidx, res["idx"]).all()
    pos = np.searchsorted(res["idx"], pidx)
    assert np.all(np.abs(res["values"][pos] - 0.4 * psgn) < 0.05)


# ---------------------------------------------------------------------------------------
# HEAVYMIX as printed (Alg. 2): l2sq estimate, heavy set H, random fill from NH

def test_l2sq_row_order_worked_by_hand(golden_dir):
    for name, expected, *vals in _read_golden(os.path.join(golden_dir, "l2sq_row_order.txt")):
        row = np.array([float(x) for x in vals], dtype=np.float32)
        assert oracle.row_sq_sum(row) == float(int(expected)), name
        # r = 1: the l2sq estimate is the row's sum
        assert oracle.l2sq_estimate(row[None, :]) == float(int(expected)), name


def test_l2sq_integer_tables_exact_median_of_row_sums():
    # integer cells: every partial sum is an integer below 2^53, so any order is exact and
    # the estimate is the median of the exact row sums (mean of the middle two for even r)
    rng = np.random.default_rng(31)
    for r in (1, 4, 5, 7):
        m = rng.integers(-3000, 3001, size=(r, 1234)).astype(np.float32)
        rows = sorted(int(np.sum(m[j].astype(np.int64) ** 2)) for j in range(r))
        want = float(rows[r // 2]) if r % 2 else (rows[r // 2 - 1] + rows[r // 2]) / 2
        assert oracle.l2sq_estimate(m) == want


def test_l2sq_estimates_the_norm():
    rng = np.random.default_rng(22)
    d, c, r = 20_000, 2000, 5
    hp = _hp(rng, r)
    x = rng.standard_normal((1, d)).astype(np.float32)
    merged = oracle.sketch(x, hp, c)[0]
    l2 = oracle.l2sq_estimate(merged)
    true = float(np.sum(x.astype(np.float64) ** 2))
    assert 0.8 * true < l2 < 1.2 * true  # each row's squared-cell sum estimates ||x||^2
    est = oracle.unsketch(merged, hp, d)
    k = 100
    assert oracle.heavy_count(est, k, l2) == int(np.sum(est.astype(np.float64) ** 2 >= l2 / k))


def _hand_example():
    """d = 16, r = 3, a collision-free sketch of x = {3: 1, 9: -1, 12: 0.625}, so every
    estimate equals x exactly (Sec. III-A) and each row's sum of squares is
    1 + 1 + 0.390625 = 2.390625 exactly."""
    d, c, r = 16, 4096, 3
    rng = np.random.default_rng(7)
    for _ in range(100):
        hp = _hp(rng, r)
        if all(len(set(oracle.buckets(int(hp["a"][j]), int(hp["b"][j]), c, range(d)))) == d for j in range(r)):
            break
    else:
        raise AssertionError("no collision-free hash found")
    x = np.zeros((1, d), np.float32)
    x[0, 3], x[0, 9], x[0, 12] = 1.0, -1.0, 0.625
    merged = oracle.sketch(x, hp, c)[0]
    rnd = np.arange(d, dtype=np.uint32)  # small draws ...
    rnd[[3, 7, 9, 11]] = 0xFFFFFFFF        # ... except these (>> 1: all 0x7FFFFFFF)
    rnd[5] = 0xFFFFFFFE                    # (>> 1: also 0x7FFFFFFF, a tie)
    rnd[12] = 0x80000000
    return hp, merged, rnd, d


def test_heavymix_worked_example():
    hp, merged, rnd, d = _hand_example()
    # k = 4: theta = 2.390625 / 4 = 0.59765625. H = {3, 9} (1 >= theta; 0.625^2 = 0.390625 is
    # not, although 0.625 >= theta, so the test is on the square). l = 2 from NH: the largest
    # draws >> 1 are 0x7FFFFFFF at 5, 7 and 11; ties go to the lower index: 5 and 7.
    res = oracle.heavymix(merged, hp, d, 4, rnd)
    assert res["l2sq"] == 2.390625
    assert res["n_heavy"] == 2
    assert res["idx"].tolist() == [3, 5, 7, 9]
    # k = 2: theta = 1.1953125 > 1, so H is empty and the fill takes all 2 from NH = every
    # coordinate: the largest draws are at 3, 5, 7, 9, 11; the two lowest indices win.
    res = oracle.heavymix(merged, hp, d, 2, rnd)
    assert res["n_heavy"] == 0 and res["idx"].tolist() == [3, 5]
    # k = 16 = d: every coordinate is selected
    res = oracle.heavymix(merged, hp, d, 16, rnd)
    assert res["idx"].tolist() == list(range(16))


def test_heavymix_k_equal_spikes_are_exactly_heavy():
    # k equal spikes of a collision-free vector: l2sq = k s^2, theta = s^2, every spike is
    # heavy (s^2 >= s^2) and nothing else is, so |H| = k and the fill is empty.
    rng = np.random.default_rng(41)
    d, c, r, k = 3000, 6000, 5, 40
    hp = _hp(rng, r)
    K = _collision_free_support(hp, c, d, k, rng)
    x = np.zeros((1, d), np.float32)
    x[0, K] = np.where(rng.random(k) < 0.5, -0.75, 0.75).astype(np.float32)
    merged = oracle.sketch(x, hp, c)[0]
    assert np.array_equal(oracle.unsketch(merged, hp, d), x[0])  # every estimate exact
    rnd = synth.fill_draws(5, 0, d)
    res = oracle.heavymix(merged, hp, d, k, rnd)
    assert res["n_heavy"] == k
    assert res["idx"].tolist() == sorted(K.tolist())


def test_heavymix_all_zero_sketch_selects_lowest_indices():
    # l2sq = 0, theta = 0, every est^2 = 0 >= 0: all coordinates heavy; Top_k = the k largest
    # |est| with ties to the lower index = {0 .. k-1}.
    rng = np.random.default_rng(3)
    d, c, r, k = 500, 64, 5, 37
    hp = _hp(rng, r)
    res = oracle.heavymix(np.zeros((r, c), np.float32), hp, d, k, synth.fill_draws(9, 0, d))
    assert res["n_heavy"] == d and res["l2sq"] == 0.0
    assert res["idx"].tolist() == list(range(k))


def test_heavymix_with_large_heavy_set_is_topk_by_magnitude():
    # whenever |H| >= k the selection is the k largest |est| (every member of H outranks
    # NH). A narrow sketch (c < k) makes theta = l2sq / k small enough for |H| > k.
    rng = np.random.default_rng(44)
    d, c, r = 4000, 50, 5
    hp = _hp(rng, r)
    merged = rng.standard_normal((r, c)).astype(np.float32)
    est = oracle.unsketch(merged, hp, d)
    l2 = oracle.l2sq_estimate(merged)
    seen = set()
    for k in range(20, 4001, 45):
        nh = oracle.heavy_count(est, k, l2)
        res = oracle.heavymix(merged, hp, d, k, synth.fill_draws(11, k, d))
        assert res["n_heavy"] == nh
        seen.add(nh >= k)
        if nh >= k:
            assert np.array_equal(res["idx"], oracle.topk(est, k)[0]), k
    assert seen == {True, False}


def test_heavymix_fill_is_uniform_over_the_non_heavy_set():
    # H is always taken whole; each member of NH is picked with probability l / |NH|
    rng = np.random.default_rng(51)
    d, c, r, k = 400, 2000, 5, 60
    hp = _hp(rng, r)
    x = (rng.standard_normal((1, d)) * np.where(np.arange(d) % 37 == 0, 30.0, 1.0)).astype(np.float32)
    merged = oracle.sketch(x, hp, c)[0]
    base = oracle.heavymix(merged, hp, d, k, synth.fill_draws(0, 0, d))
    nh = base["n_heavy"]
    assert 0 < nh < k
    est = base["est"]
    heavy = set(np.flatnonzero(est.astype(np.float64) ** 2 >= base["l2sq"] / k).tolist())
    assert len(heavy) == nh
    trials = 600
    counts = np.zeros(d)
    for t in range(trials):
        res = oracle.heavymix(merged, hp, d, k, synth.fill_draws(1000 + t, 0, d))
        idx = res["idx"]
        assert idx.size == k and np.all(np.diff(idx) > 0)
        assert heavy <= set(idx.tolist())
        counts[idx] += 1
    light = np.array(sorted(set(range(d)) - heavy))
    p = (k - nh) / light.size
    expect = trials * p
    chi2 = float(np.sum((counts[light] - expect) ** 2 / (expect * (1 - p))))
    dof = light.size - 1
    assert abs(chi2 - dof) < 6 * np.sqrt(2 * dof), (chi2, dof)


# ---------------------------------------------------------------------------------------
# Momentum and error kept in the sketch (the sketch is linear: Sec. II, sketching paragraph)

def _collision_free_hash(d, c, r, seed):
    rng = np.random.default_rng(seed)
    for _ in range(200):
        hp = _hp(rng, r)
        if all(len(set(oracle.buckets(int(hp["a"][j]), int(hp["b"][j]), c, range(d)))) == d for j in range(r)):
            return hp
    raise AssertionError("no collision-free hash found")


def test_sketch_momentum_equals_vector_space_when_collision_free_and_exact():
    # With no two coordinates sharing a cell and every operation exact (small integer
    # gradients, rho = 0.5), the sketch of the summed vector-space state is the sketch-space
    # state: the same selections and values on every step, and the reset at Top_k in vector
    # space is the subtraction plus momentum mask in sketch space.
    d, P, r, c, k = 300, 3, 3, 1 << 20, 17
    hp = _collision_free_hash(d, c, r, 61)
    rng = np.random.default_rng(62)
    u = np.zeros((P, d), np.float32)
    v = np.zeros((P, d), np.float32)
    U = np.zeros((r, c), np.float32)
    E = np.zeros((r, c), np.float32)
    for t in range(5):
        g = rng.integers(-8, 9, size=(P, d)).astype(np.float32)
        vec = oracle.step(g, u, v, hp, c, k, rho=0.5, want_tables=False, want_est=False)
        sk = oracle.sketch_momentum_step(g, U, E, hp, k, rho=0.5)
        assert np.array_equal(sk["idx"], vec["idx"]), t
        assert np.array_equal(sk["values"], vec["values"]), t
        # the state itself: E and U are the sketches of sum_q v and sum_q u
        assert np.array_equal(E, oracle.sketch(v.sum(axis=0, keepdims=True), hp, c)[0]), t
        assert np.array_equal(U, oracle.sketch(u.sum(axis=0, keepdims=True), hp, c)[0]), t


def test_sketch_momentum_k_equals_d_clears_the_state():
    d, P, r, c = 64, 2, 3, 1 << 16
    hp = _collision_free_hash(d, c, r, 63)
    g = np.random.default_rng(64).standard_normal((P, d)).astype(np.float32)
    U = np.zeros((r, c), np.float32)
    E = np.zeros((r, c), np.float32)
    res = oracle.sketch_momentum_step(g, U, E, hp, d, rho=0.9)
    assert res["idx"].tolist() == list(range(d))
    assert not E.any() and not U.any()


def test_sketch_momentum_without_reset_keeps_momentum_and_composes():
    rng = np.random.default_rng(65)
    d, P, r, c, k = 3000, 4, 5, 400, 30
    hp = _hp(rng, r)
    U0 = rng.standard_normal((r, c)).astype(np.float32)
    E0 = rng.standard_normal((r, c)).astype(np.float32)
    g = rng.standard_normal((P, d)).astype(np.float32)
    U, E = U0.copy(), E0.copy()
    res = oracle.sketch_momentum_step(g, U, E, hp, k, rho=0.9, reset_momentum=False)
    S = oracle.merge(oracle.sketch(g, hp, c))
    assert np.array_equal(res["merged"], S)
    want_U = (np.float32(0.9) * U0).astype(np.float32) + S
    assert np.array_equal(U, want_U)
    E1 = E0 + want_U
    est = oracle.unsketch(E1, hp, d)
    idx, _ = oracle.topk(est, k)
    assert np.array_equal(res["idx"], idx) and np.array_equal(res["values"], est[idx])
    # untouched cells keep E1; the others moved by the selection's sketch
    touched = np.zeros((r, c), bool)
    for j in range(r):
        touched[j, oracle.buckets(int(hp["a"][j]), int(hp["b"][j]), c, idx)] = True
    assert np.array_equal(E[~touched], E1[~touched])
    assert not np.array_equal(E[touched], E1[touched])


def test_sketch_momentum_subtracts_the_selection_sketch_worked_example():
    # One cell (r = c = 1), two coordinates with sign +1, g = (1, 2), rho = 0, k = 2 = d:
    # U = S = 1 + 2 = 3, E = 3; both estimates are 3; the selection's sketch is 3 + 3 = 6,
    # so E becomes 3 - 6 = -3 (a cell shared by selected coordinates is over-corrected, not
    # zeroed), and U is masked to 0.
    rng = np.random.default_rng(66)
    for _ in range(1000):
        hp = _hp(rng, 1)
        if oracle.signs(int(hp["a2"][0]), int(hp["b2"][0]), [0, 1]).tolist() == [1, 1]:
            break
    else:
        raise AssertionError("no all-positive sign hash found")
    U = np.zeros((1, 1), np.float32)
    E = np.zeros((1, 1), np.float32)
    res = oracle.sketch_momentum_step(np.array([[1.0, 2.0]], np.float32), U, E, hp, 2, rho=0.0)
    assert res["merged"][0, 0] == 3.0 and res["values"].tolist() == [3.0, 3.0]
    assert E[0, 0] == -3.0 and U[0, 0] == 0.0


# ---------------------------------------------------------------------------------------
# Weight update (Alg. 1, last step)

def test_apply_update_closed_forms():
    d = 1000
    idx = np.array([3, 17, 999], np.int32)
    vals = np.array([0.5, -2.0, 3.25], np.float32)
    w = np.zeros(d, np.float32)
    oracle.apply_update(w, idx, vals, 1.0)  # eta = 1 from zero: w = -G~ exactly
    want = np.zeros(d, np.float32)
    want[idx] = -vals
    assert np.array_equal(w, want)
    w2 = np.full(d, 1.0, np.float32)
    oracle.apply_update(w2, idx, vals, 0.25)  # dyadic: exact
    want2 = np.full(d, 1.0, np.float32)
    want2[idx] = [1.0 - 0.125, 1.5, 1.0 - 0.8125]
    assert np.array_equal(w2, want2)


def test_apply_update_rounds_the_product_then_the_difference():
    # fl(w - fl(eta * x)) differs from a fused multiply-subtract on some inputs
    rng = np.random.default_rng(71)
    d = 100_000
    w = rng.standard_normal(d).astype(np.float32)
    x = rng.standard_normal(d).astype(np.float32)
    idx = np.arange(d, dtype=np.int32)
    w1 = w.copy()
    oracle.apply_update(w1, idx, x, 0.1)
    two_step = (w - (np.float32(0.1) * x).astype(np.float32)).astype(np.float32)
    assert np.array_equal(w1, two_step)
    fused = (w.astype(np.float64) - np.float64(np.float32(0.1)) * x.astype(np.float64)).astype(np.float32)
    assert np.count_nonzero(fused != w1) > 100
