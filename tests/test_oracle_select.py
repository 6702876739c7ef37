"""Pins for the selection oracle: brute force, closed forms, the paper's budgets, invariants."""
import itertools
import json
import os

import numpy as np
import pytest

from oracle import select as osel
from oracle.errors import DcutArgError, DcutDataError, DERR_CONF

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _conf(rng, B, D, kind):
    if kind == "beta":
        a = rng.uniform(1, 8, size=B)
        return np.power(rng.random((B, D)), 1 / a[:, None]).astype(np.float32)
    if kind == "coarse":      # many exact ties in s
        return rng.choice(np.array([0.0, 0.25, 0.5, 1.0], np.float32), size=(B, D))
    if kind == "tiny":        # scores below the 2^-40 resolution
        return rng.choice(np.array([1e-7, 1e-3, 0.9, 1.0], np.float32), size=(B, D))
    raise ValueError(kind)


def _brute(conf, budgets, costs):
    """Enumerate every allocation (n_0..n_{B-1}); best integer benefit per budget."""
    B, D = conf.shape
    s = np.cumprod(np.concatenate([np.ones((B, 1), np.float32), conf], axis=1), axis=1, dtype=np.float32)
    u = np.trunc(s.astype(np.float64) * 2.0 ** 40).astype(np.uint64)
    cum = np.cumsum(u, axis=1, dtype=np.uint64)            # cum[i][n] = sum_{k<=n} u
    grids = np.meshgrid(*[np.arange(D + 1)] * B, indexing="ij")
    tot_k = sum(g + 1 for g in grids).ravel()
    ben = sum(cum[i][grids[i]] for i in range(B)).ravel()
    best = {}
    for K in set(budgets):
        best[K] = int(ben[tot_k == K].max())
    objs = [best[K] * 2.0 ** -40 / c for K, c in zip(budgets, costs)]
    r = int(np.argmax(objs))  # numpy argmax: first occurrence of the max
    return s, best, r


@pytest.mark.parametrize("B", [1, 2, 3, 4])
@pytest.mark.parametrize("kind", ["beta", "coarse", "tiny"])
def test_bruteforce_optimal_and_canonical(B, kind):
    rng = np.random.default_rng(100 * B + len(kind))
    D = 15
    for trial in range(3):
        conf = _conf(rng, B, D, kind)
        draft = rng.integers(0, 1000, size=(B, D + 1)).astype(np.int32)
        ctx = rng.integers(0, 50, size=B).astype(np.int32)
        R = int(rng.integers(1, 6))
        budgets = sorted(rng.integers(B, B * (D + 1) + 1, size=R).tolist())
        costs = rng.uniform(0.5, 3.0, size=R).tolist()
        out = osel.select(conf, draft, ctx, budgets, costs)
        s, best, r = _brute(conf, budgets, costs)
        # (i) exact optimal integer benefit per candidate budget
        assert [int(b) for b in out["benefit"]] == [best[K] for K in budgets]
        # (iii) same ratio choice from the brute-force objectives
        assert int(out["choice"][1]) == r and int(out["choice"][0]) == budgets[r]
        # (ii) the kept allocation attains the optimum and is the tie-rule canonical one:
        keep = out["keep_len"]
        u = np.trunc(s.astype(np.float64) * 2.0 ** 40).astype(np.uint64)
        got = sum(int(u[i, :keep[i]].sum()) for i in range(B))
        assert got == best[budgets[r]] and int(keep.sum()) == budgets[r]
        kept = [(float(s[i, k]), -k, -i) for i in range(B) for k in range(keep[i])]
        dropped = [(float(s[i, k]), -k, -i) for i in range(B) for k in range(keep[i], D + 1)]
        if kept and dropped:
            assert min(kept) > max(dropped)


def test_bruteforce_five_requests():
    rng = np.random.default_rng(5)
    B, D = 5, 15
    conf = _conf(rng, B, D, "beta")
    budgets = [5, 17, 33, 40, 64, 80]
    costs = [1.0, 1.3, 1.9, 2.1, 2.6, 3.4]
    out = osel.select(conf, np.zeros((B, D + 1), np.int32), np.zeros(B, np.int32), budgets, costs)
    _, best, r = _brute(conf, budgets, costs)
    assert [int(b) for b in out["benefit"]] == [best[K] for K in budgets]
    assert int(out["choice"][1]) == r


def test_tie_rule_worked_example():
    g = json.load(open(os.path.join(GOLD, "tie_rule_example.json")))
    conf = np.array(g["conf"], np.float32)
    for K, want in g["keep_len_by_K"].items():
        out = osel.select(conf, np.zeros((2, 3), np.int32), np.zeros(2, np.int32), [int(K)], [1.0])
        assert out["keep_len"].tolist() == want


@pytest.mark.parametrize("cval", [0.0, 1.0])
def test_closed_form_breadth_first(cval):
    B, D = 7, 15
    conf = np.full((B, D), cval, np.float32)
    for K in [B, B + 1, 2 * B - 1, 3 * B + 4, 100, B * (D + 1)]:
        out = osel.select(conf, np.zeros((B, D + 1), np.int32), np.zeros(B, np.int32), [K], [1.0])
        q, r = divmod(K - B, B)
        want = [1 + q + (1 if i < r else 0) for i in range(B)]
        assert out["keep_len"].tolist() == want


def test_closed_form_extremes_and_cost_shapes():
    rng = np.random.default_rng(7)
    B, D = 6, 15
    conf = _conf(rng, B, D, "beta")
    conf = np.maximum(conf, np.float32(0.5))      # every score >= 2^-15, so u > 0 everywhere
    grid = [B * m for m in range(1, D + 2)]
    dz = np.zeros((B, D + 1), np.int32)
    z = np.zeros(B, np.int32)
    assert osel.select(conf, dz, z, [B], [1.0])["keep_len"].tolist() == [1] * B
    assert osel.select(conf, dz, z, [B * (D + 1)], [1.0])["keep_len"].tolist() == [D + 1] * B
    # constant cost: benefit strictly increases with K, so the largest budget wins
    out = osel.select(conf, dz, z, grid, [2.0] * len(grid))
    assert int(out["choice"][0]) == grid[-1]
    # cost proportional to K: the top-K mean never increases, so K = B wins
    out = osel.select(conf, dz, z, grid, [0.1 * K for K in grid])
    assert int(out["choice"][0]) == B


def test_paper_budget_table():
    g = json.load(open(os.path.join(GOLD, "cost_table_tab3.json")))
    for bi, B in enumerate(g["B"]):
        got = [osel.budget_from_ratio(B, g["D"], n, d) for n, d in g["ratios"]]
        assert got == g["budget_from_caption"][bi]
    # lower clamp of Eq. dcut-budget: every request keeps its bonus
    assert osel.budget_from_ratio(10, 0, 1, 4) == 10
    assert osel.budget_from_ratio(3, 3, 1, 3) == 4      # ceil(12/3) = 4
    assert osel.budget_from_ratio(3, 3, 1, 5) == 3      # ceil(2.4) = 3 = B


def test_paper_cost_rows_as_costs():
    """The printed cost rows drive a valid selection; r* maximises benefit/cost by brute force."""
    g = json.load(open(os.path.join(GOLD, "cost_table_tab3.json")))
    rng = np.random.default_rng(11)
    B, D = 4, 15
    for key in ("H20_ms", "H800_ms"):
        budgets = [osel.budget_from_ratio(B, D, n, d) for n, d in g["ratios"]]
        for row in g[key]:
            conf = _conf(rng, B, D, "beta")
            out = osel.select(conf, np.zeros((B, D + 1), np.int32), np.zeros(B, np.int32), budgets, row)
            _, best, r = _brute(conf, budgets, row)
            assert int(out["choice"][1]) == r


@pytest.mark.parametrize("seed", range(20))
def test_invariants(seed):
    rng = np.random.default_rng(seed)
    B = int(rng.integers(1, 40))
    D = int(rng.integers(0, 20))
    conf = _conf(rng, B, D, ["beta", "coarse", "tiny"][seed % 3])
    draft = rng.integers(0, 500, size=(B, D + 1)).astype(np.int32)
    ctx = rng.integers(0, 1000, size=B).astype(np.int32)
    prev = np.zeros(B, np.int32)
    for K in range(B, B * (D + 1) + 1, max(1, B // 2)):
        out = osel.select(conf, draft, ctx, [K], [1.0])
        kl = out["keep_len"]
        assert kl.min() >= 1 and int(kl.sum()) == K           # progress + exact budget
        assert (kl >= prev).all()                             # monotone in K
        prev = kl
        cu = out["cu"]
        assert cu[0] == 0 and int(cu[B]) == K and (np.diff(cu) == kl).all()
        t = np.arange(K)
        req = out["packed_req"][:K]
        k = t - cu[req]
        assert ((0 <= k) & (k < kl[req])).all()
        assert (out["packed_pos"][:K] - ctx[req] == k).all()
        assert (out["packed_tok"][:K] == draft[req, k]).all()


def test_data_faults():
    base = np.full((2, 3), 0.5, np.float32)
    for bad in [np.nan, -0.25, 1.5, -0.0]:
        c = base.copy()
        c[1, 2] = bad
        with pytest.raises(DcutDataError) as e:
            osel.select(c, np.zeros((2, 4), np.int32), np.zeros(2, np.int32), [4], [1.0])
        assert e.value.bits == DERR_CONF


def test_arg_errors():
    c = np.full((2, 3), 0.5, np.float32)
    dz = np.zeros((2, 4), np.int32)
    z = np.zeros(2, np.int32)
    for budgets, costs in [([1], [1.0]), ([9], [1.0]), ([5, 4], [1.0, 1.0]), ([4], [0.0]),
                           ([4], [float("nan")]), ([4], [float("inf")]), ([], []), ([4], [])]:
        with pytest.raises(DcutArgError):
            osel.select(c, dz, z, budgets, costs)
    with pytest.raises(DcutArgError):
        osel.select(np.zeros((1, 64), np.float32), np.zeros((1, 65), np.int32), z[:1], [1], [1.0])
    with pytest.raises(DcutArgError):
        osel.budget_from_ratio(4, 15, 5, 4)


def test_fixed_point_exactness():
    s = np.array([1.0, 0.5, 2.0 ** -40, 2.0 ** -41, np.float32(0.1)], np.float32)
    u = osel.fixed_point(s)
    assert u.tolist() == [2 ** 40, 2 ** 39, 1, 0, int(float(np.float32(0.1)) * 2 ** 40)]
    # sequential float32 products keep subnormals
    p = osel.prefix_scores(np.array([[2.0 ** -70, 2.0 ** -70]], np.float32))
    assert p[0, 1] == np.float32(2.0 ** -70) and p[0, 2] == np.float32(2.0 ** -140)  # subnormal kept
    z = osel.prefix_scores(np.array([[2.0 ** -80, 2.0 ** -80]], np.float32))
    assert z[0, 2] == np.float32(0.0)
    q = osel.prefix_scores(np.array([[2.0 ** -63, 2.0 ** -63]], np.float32))
    assert q[0, 2] == np.float32(2.0 ** -126)
