"""Pins of the rejection-sampling oracle (App. B) against hand-worked values,
alternative formulations, the causality property the appendix proves, and the
output distribution RS must reproduce."""
import json
import math
import os

import numpy as np
import pytest
from scipy import stats

from oracle import rs
from oracle import select as osel
from oracle.errors import DcutArgError, DcutDataError

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _load(name):
    return json.load(open(os.path.join(GOLD, name)))


# ---------------------------------------------------------------- shifted scores

def test_shifted_scores_hand_values():
    conf = np.array([[0.5, 0.25, 0.75]], np.float32)
    s = rs.shifted_scores(conf)
    assert s.dtype == np.float32
    assert s.tolist() == [[1.0, 1.0, 0.5, 0.125]]          # c_3 never enters
    assert rs.shifted_scores(np.zeros((3, 0), np.float32)).tolist() == [[1.0]] * 3


def test_shifted_scores_are_the_unshifted_ones_moved_by_one_depth():
    rng = np.random.default_rng(3)
    conf = rng.random((7, 9)).astype(np.float32)
    s, t = rs.shifted_scores(conf), osel.prefix_scores(conf)
    assert np.array_equal(s[:, 0], np.ones(7, np.float32))
    assert np.array_equal(s[:, 1:], t[:, :-1])
    # depth k never depends on c_k or later
    conf2 = conf.copy()
    conf2[:, 4:] = rng.random((7, 5)).astype(np.float32)
    assert np.array_equal(rs.shifted_scores(conf2)[:, :5], s[:, :5])


def test_shifted_scores_reject_bad_confidence():
    for bad in [np.nan, -0.0, 1.5]:
        c = np.full((2, 3), 0.5, np.float32)
        c[1, 2] = bad
        with pytest.raises(DcutDataError):
            rs.shifted_scores(c)


# ---------------------------------------------------------------- cost curve

def test_cost_curve_knots_linear_and_flat_ends():
    C = rs.cost_curve(4, 3, [6, 10, 16], [2.0, 4.0, 7.0])
    assert C.shape == (17,)
    assert C[6] == 2.0 and C[10] == 4.0 and C[16] == 7.0
    assert C[8] == 3.0 and C[13] == 5.5
    assert np.all(C[:6] == 2.0)                     # below the first budget: its cost
    assert np.all(np.diff(C) >= 0)


def test_cost_curve_single_budget_and_duplicates():
    assert np.all(rs.cost_curve(2, 3, [5], [1.5]) == 1.5)
    # equal budgets: the last one's cost holds at that K, then interpolate onward
    C = rs.cost_curve(2, 3, [2, 4, 4, 8], [1.0, 2.0, 3.0, 5.0])
    assert C[3] == 1.5 and C[4] == 3.0 and C[6] == 4.0 and C[8] == 5.0


def test_cost_curve_exact_on_integer_affine_costs():
    B, D = 5, 6
    N = B * (D + 1)
    C = rs.cost_curve(B, D, [B, N], [float(B), float(N)])
    assert np.array_equal(C[B:], np.arange(B, N + 1, dtype=np.float64))


# ---------------------------------------------------------------- causal scan

def test_scan_hand_example():
    g = _load("rs_scan_example.json")
    conf = np.array(g["conf"], np.float32)
    for case in g["cases"]:
        C = rs.cost_curve(2, 2, g["budgets"], case["costs"])
        assert np.allclose(C, case["curve"], rtol=0, atol=1e-15)
        o = rs.select_rs(conf, np.zeros((2, 3), np.int32), np.array([5, 9]), rs.SCAN,
                         g["budgets"], case["costs"])
        assert o["choice"].tolist() == [case["K"], case["r"]]
        assert o["keep_len"].tolist() == case["keep_len"]
        assert o["objective"] == pytest.approx(case["objective"], rel=1e-15)
        assert int(o["cu"][-1]) == case["K"]


def _first_stop(s, curve):
    """Alternative formulation: walk the global ranking of the shifted scores
    and stop at the first K >= B whose next objective is not larger."""
    B, D1 = s.shape
    order = osel.rank_order(s)
    u = osel.fixed_point(s).ravel()[order]
    P = np.concatenate([[0], np.cumsum(u.astype(object))])
    N = B * D1
    J = lambda K: (float(P[K]) * 2.0 ** -40) / curve[K]
    K = B
    while K < N and J(K + 1) > J(K):
        K += 1
    kept = np.zeros(N, bool)
    kept[order[:K]] = True
    return K, kept.reshape(B, D1)


def _random_instance(rng, B, D, R):
    conf = rng.choice([0.0, 0.25, 0.5, 0.75, 1.0], size=(B, D)).astype(np.float32)
    if rng.random() < 0.5:
        conf = rng.random((B, D)).astype(np.float32)
    N = B * (D + 1)
    budgets = sorted(int(x) for x in rng.integers(B, N + 1, size=R))
    costs = sorted(float(x) for x in rng.uniform(0.5, 3.0, size=R))
    if rng.random() < 0.3:
        costs = [float(x) for x in rng.uniform(0.5, 3.0, size=R)]      # not monotone
    return conf, budgets, costs


def test_scan_equals_first_local_maximum_over_the_ranking():
    rng = np.random.default_rng(11)
    for _ in range(300):
        B, D, R = int(rng.integers(1, 6)), int(rng.integers(0, 6)), int(rng.integers(1, 5))
        conf, budgets, costs = _random_instance(rng, B, D, R)
        s = rs.shifted_scores(conf)
        curve = rs.cost_curve(B, D, budgets, costs)
        sc = rs.causal_scan(s, curve)
        K, kept = _first_stop(s, curve)
        assert sc["K"] == K
        assert np.array_equal(sc["admitted"], kept)
        # admission order is the ranking itself
        assert [i * (D + 1) + k for i, k in sc["order"]] == list(osel.rank_order(s)[:K])


def _retention(conf, budgets, costs, mode, shifted=True):
    B, D = conf.shape
    if shifted:
        return rs.select_rs(conf, np.zeros((B, D + 1), np.int32), np.zeros(B, np.int32), mode,
                            budgets, costs)["kept"]
    s = osel.prefix_scores(conf)          # unshifted scores through the same scan
    return rs.causal_scan(s, rs.cost_curve(B, D, budgets, costs))["admitted"]


def _retrospective(conf, budgets, costs):
    """Global argmax over the buckets applied to shifted scores (not causal)."""
    B, D = conf.shape
    s = rs.shifted_scores(conf)
    order = osel.rank_order(s)
    u = osel.fixed_point(s).ravel()[order]
    P = np.concatenate([[0], np.cumsum(u.astype(object))])
    objs = [(float(P[K]) * 2.0 ** -40) / c for K, c in zip(budgets, costs)]
    K = budgets[int(np.argmax(objs))]
    kept = np.zeros(B * (D + 1), bool)
    kept[order[:K]] = True
    return kept.reshape(B, D + 1)


def _violations(select_fn, rng, trials):
    """Count positions (i, k) whose retention changes when z_{i,k} and later
    proposals of request i change (their confidences c_{i,k..D} redrawn)."""
    bad = 0
    for _ in range(trials):
        B, D, R = int(rng.integers(2, 5)), int(rng.integers(2, 6)), int(rng.integers(2, 5))
        conf, budgets, costs = _random_instance(rng, B, D, R)
        base = select_fn(conf, budgets, costs)
        for i in range(B):
            for k in range(1, D + 1):
                c2 = conf.copy()
                c2[i, k - 1:] = rng.random(D - k + 1).astype(np.float32)
                if select_fn(c2, budgets, costs)[i, k] != base[i, k]:
                    bad += 1
    return bad


def test_scan_and_fixed_budget_are_causal():
    """App. B, distributional correctness: whether (i, k) is kept never
    depends on z_{i,k} or any later proposal of request i."""
    rng = np.random.default_rng(5)
    assert _violations(lambda c, b, co: _retention(c, b, co, rs.SCAN), rng, 120) == 0
    rng = np.random.default_rng(6)
    assert _violations(lambda c, b, co: _retention(c, b[:1], co[:1], rs.FIXED), rng, 120) == 0


def test_non_causal_variants_are_caught():
    """The appendix's two counterexamples: unshifted scores, and shifted scores
    with a retrospective choice of the budget, both let a proposal decide its
    own retention.  The causality check above must see that."""
    rng = np.random.default_rng(7)
    assert _violations(lambda c, b, co: _retention(c, b, co, rs.SCAN, shifted=False), rng, 60) > 0
    rng = np.random.default_rng(8)
    assert _violations(_retrospective, rng, 200) > 0


def test_scan_closed_forms():
    rng = np.random.default_rng(2)
    B, D = 6, 5
    N = B * (D + 1)
    conf = rng.uniform(0.05, 1.0, (B, D)).astype(np.float32)
    z = np.zeros((B, D + 1), np.int32)
    L = np.zeros(B, np.int32)
    # constant cost: every position with a positive score improves the objective
    o = rs.select_rs(conf, z, L, rs.SCAN, [B], [2.0])
    assert o["choice"][0] == N and np.all(o["keep_len"] == D + 1)
    # cost exactly K and every score 1: the objective stays 1, nothing beyond the bonus
    ones = np.ones((B, D), np.float32)
    o = rs.select_rs(ones, z, L, rs.SCAN, [B, N], [float(B), float(N)])
    assert o["choice"].tolist() == [B, 0] and np.all(o["keep_len"] == 1)
    # cost K + 1 and every score 1: the objective K/(K+1) rises to the full block
    o = rs.select_rs(ones, z, L, rs.SCAN, [B, N], [float(B + 1), float(N + 1)])
    assert o["choice"].tolist() == [N, 1]
    # zero confidences: depth 1 (shifted score 1) may still enter, depth 2 never
    zero = np.zeros((B, D), np.float32)
    o = rs.select_rs(zero, z, L, rs.SCAN, [B, N], [1.0, 1.0 + 1e-9])
    assert np.all(o["keep_len"] <= 2) and o["choice"][0] >= B


def test_fixed_budget_is_global_top_k_of_shifted_scores():
    rng = np.random.default_rng(9)
    for _ in range(50):
        B, D = int(rng.integers(1, 6)), int(rng.integers(0, 6))
        N = B * (D + 1)
        conf = rng.random((B, D)).astype(np.float32)
        K = int(rng.integers(B, N + 1))
        z = rng.integers(0, 50, (B, D + 1)).astype(np.int32)
        L = rng.integers(0, 20, B).astype(np.int32)
        o = rs.select_rs(conf, z, L, rs.FIXED, [K], [1.0])
        s = rs.shifted_scores(conf)
        # brute force: the K largest (score, -depth, -request) triples
        trip = sorted(((float(s[i, k]), -k, -i) for i in range(B) for k in range(D + 1)), reverse=True)
        keep = np.zeros((B, D + 1), bool)
        for _, mk, mi in trip[:K]:
            keep[-mi, -mk] = True
        assert np.array_equal(o["kept"], keep)
        assert int(o["cu"][-1]) == K and o["choice"].tolist() == [K, 0]
        for i in range(B):
            for k in range(o["keep_len"][i]):
                t = o["cu"][i] + k
                assert (o["packed_tok"][t], o["packed_pos"][t], o["packed_req"][t]) == (z[i, k], L[i] + k, i)


def test_history_budget_is_carried_and_causal():
    """HISTORY: K* is the state passed in (clamped), retention is then causal,
    and the state passed on is the retrospective bucket choice of this block
    (brute force over the candidate budgets)."""
    rng = np.random.default_rng(13)
    for _ in range(60):
        B, D, R = int(rng.integers(1, 6)), int(rng.integers(0, 6)), int(rng.integers(1, 5))
        conf, budgets, costs = _random_instance(rng, B, D, R)
        N = B * (D + 1)
        z = np.zeros((B, D + 1), np.int32)
        L = np.zeros(B, np.int32)
        k_in = int(rng.integers(-3, N + 5))
        o = rs.select_rs(conf, z, L, rs.HISTORY, budgets, costs, k_state=k_in)
        assert int(o["choice"][0]) == min(max(k_in, B), N)
        fx = rs.select_rs(conf, z, L, rs.FIXED, [min(max(k_in, B), N)], [1.0])
        assert np.array_equal(o["kept"], fx["kept"])
        # brute force: objective of every candidate from its own top-K sum
        s = rs.shifted_scores(conf)
        vals = sorted(((float(s[i, k]), -k, -i) for i in range(B) for k in range(D + 1)), reverse=True)
        u = [int(np.trunc(np.float64(v[0]) * 2.0 ** 40)) for v in vals]
        objs = [(float(sum(u[:K])) * 2.0 ** -40) / c for K, c in zip(budgets, costs)]
        best = max(range(R), key=lambda r: (objs[r], -r))
        assert o["k_next"] == budgets[best]
    rng = np.random.default_rng(14)
    assert _violations(lambda c, b, co: _retention_hist(c, b, co), rng, 80) == 0


def _retention_hist(conf, budgets, costs):
    B, D = conf.shape
    return rs.select_rs(conf, np.zeros((B, D + 1), np.int32), np.zeros(B, np.int32), rs.HISTORY,
                        budgets, costs, k_state=budgets[len(budgets) // 2])["kept"]


def test_select_rs_argument_errors():
    conf = np.full((2, 3), 0.5, np.float32)
    z = np.zeros((2, 4), np.int32)
    L = np.zeros(2, np.int32)
    with pytest.raises(DcutArgError):
        rs.select_rs(conf, z, L, rs.FIXED, [2, 4], [1.0, 2.0])
    with pytest.raises(DcutArgError):
        rs.select_rs(conf, z, L, 7, [2], [1.0])
    with pytest.raises(DcutArgError):
        rs.select_rs(conf, z, L, rs.SCAN, [1], [1.0])


# ---------------------------------------------------------------- RS acceptance

def _blocks(n_req, D, L0=100):
    keep_len = np.full(n_req, D + 1, np.int32)
    cu = np.zeros(n_req + 1, np.int32)
    cu[1:] = np.cumsum(keep_len)
    return keep_len, cu, np.full(n_req, L0, np.int32)


def _logits_of(p):
    return np.log(np.asarray(p, np.float64))


def test_accept_uniforms_are_uniform_and_keyed():
    u = rs.accept_uniform(np.arange(20000) % 97, np.arange(20000) // 97, 5)
    assert stats.kstest(u, "uniform").pvalue > 1e-3
    assert np.array_equal(rs.accept_uniform([3, 3], [8, 8], 5), rs.accept_uniform([3, 3], [8, 8], 5))
    assert rs.accept_uniform([3], [8], 5)[0] != rs.accept_uniform([3], [8], 6)[0]


def test_rs_055_example():
    """App. B's one-position example: proposal-dependent retention plus
    unchanged RS emits A with probability 0.55; a retention decision that
    does not look at the proposal gives p(A) = 0.5."""
    g = _load("rs_055_example.json")
    p, q = np.array(g["p"]), np.array(g["q"])
    n = 20000
    rng = np.random.default_rng(1)
    z1 = (rng.random(n) >= q[0]).astype(np.int32)          # 0 = A with probability 0.9
    draft = np.stack([np.zeros(n, np.int32), z1], axis=1)
    qq = np.broadcast_to(q, (n, 1, 2))
    logits = np.broadcast_to(_logits_of(p), (2 * n, 2))
    L = np.full(n, 50, np.int32)

    def emitted_A(keep_len):
        cu = np.zeros(n + 1, np.int32)
        cu[1:] = np.cumsum(keep_len)
        o = rs.rs_accept(draft, keep_len, cu, L, qq, logits, 1.0, 123)
        first = np.where(o["accept_len"] >= 1, z1, o["next_tok"])
        return float(np.mean(first == 0))

    biased = emitted_A(np.where(q[z1] > g["keep_threshold"], 2, 1).astype(np.int32))
    causal = emitted_A(np.full(n, 2, np.int32))
    sd = math.sqrt(0.25 / n)
    assert abs(biased - g["biased_p_A"]) < 4 * sd
    assert abs(causal - g["target_p_A"]) < 4 * sd


def test_rs_output_follows_the_target_joint_distribution():
    """Token 1 ~ p_0; given token 1 = x came from an accepted draft, token 2 ~ p_1(. | x)."""
    V, n = 3, 12000
    rng = np.random.default_rng(4)
    p0 = np.array([0.5, 0.3, 0.2])
    p1 = np.array([[0.1, 0.6, 0.3], [0.7, 0.2, 0.1], [0.2, 0.2, 0.6]])      # p_1(. | token 1)
    q1 = np.array([0.2, 0.7, 0.1])
    q2 = np.array([[0.3, 0.3, 0.4], [0.8, 0.1, 0.1], [0.05, 0.05, 0.9]])    # q_2(. | z_1)
    z1 = np.array([rng.choice(V, p=q1) for _ in range(n)], np.int32)
    z2 = np.array([rng.choice(V, p=q2[a]) for a in z1], np.int32)
    draft = np.stack([np.zeros(n, np.int32), z1, z2], axis=1)
    q = np.stack([np.broadcast_to(q1, (n, V)), q2[z1]], axis=1)
    keep_len, cu, L = _blocks(n, 2)
    logits = np.empty((3 * n, V))
    logits[0::3] = _logits_of(p0)
    logits[1::3] = _logits_of(p1[z1])
    logits[2::3] = 0.0                                                      # bonus row: uniform
    o = rs.rs_accept(draft, keep_len, cu, L, q, logits, 1.0, 77)
    a = o["accept_len"]
    t1 = np.where(a >= 1, z1, o["next_tok"])
    f1 = np.bincount(t1, minlength=V)
    assert stats.chisquare(f1, n * p0).pvalue > 1e-3
    t2 = np.where(a >= 2, z2, o["next_tok"])
    for x in range(V):
        m = (a >= 1) & (z1 == x)
        f2 = np.bincount(t2[m], minlength=V)
        assert m.sum() > 500
        assert stats.chisquare(f2, m.sum() * p1[x]).pvalue > 1e-3


def test_rs_residual_distribution():
    """After a rejection the committed token follows (p - q)_+ normalised."""
    V, n = 4, 20000
    p = np.array([0.1, 0.4, 0.3, 0.2])
    q = np.array([0.5, 0.1, 0.3, 0.1])
    rng = np.random.default_rng(8)
    z1 = np.array(rng.choice(V, size=n, p=q), np.int32)
    draft = np.stack([np.zeros(n, np.int32), z1], axis=1)
    keep_len, cu, L = _blocks(n, 1)
    logits = np.broadcast_to(_logits_of(p), (2 * n, V))
    o = rs.rs_accept(draft, keep_len, cu, L, np.broadcast_to(q, (n, 1, V)), logits, 1.0, 9)
    rej = o["accept_len"] == 0
    # rejection probability = total variation distance between p and q
    tv = 0.5 * np.abs(p - q).sum()
    assert abs(rej.mean() - tv) < 4 * math.sqrt(tv * (1 - tv) / n)
    res = np.maximum(p - q, 0) / np.maximum(p - q, 0).sum()
    f = np.bincount(o["next_tok"][rej], minlength=V)
    assert f[res == 0].sum() == 0
    keep = res > 0
    assert stats.chisquare(f[keep], rej.sum() * res[keep]).pvalue > 1e-3
    assert np.array_equal(np.flatnonzero(o["rej_row"] >= 0), np.flatnonzero(rej))
    assert np.all(o["rej_row"][rej] == cu[:-1][rej])


def test_rs_special_cases():
    V, n = 5, 400
    rng = np.random.default_rng(10)
    keep_len, cu, L = _blocks(n, 3)
    draft = rng.integers(0, V, (n, 4)).astype(np.int32)
    logits = rng.normal(size=(4 * n, V))
    # q equal to p at every row: every draft is accepted, the bonus comes from p
    q = np.empty((n, 3, V))
    for i in range(n):
        for j in range(3):
            q[i, j] = rs.target_probs(logits[cu[i] + j], 1.0)
    o = rs.rs_accept(draft, keep_len, cu, L, q, logits, 1.0, 3)
    assert np.all(o["accept_len"] == 3) and o["total"][0] == 4 * n
    from oracle import sampling
    bonus = sampling.sample_tokens(logits[cu[:-1] + 3], np.arange(n), L + 3, 1.0, 3)["token"]
    assert np.array_equal(o["next_tok"], bonus)
    # a draft the target gives probability 0 is always rejected, never re-emitted
    lg = logits.copy()
    lg[np.arange(0, 4 * n, 4), draft[:, 1]] = -np.inf
    o = rs.rs_accept(draft, keep_len, cu, L, q, lg, 1.0, 3)
    assert np.all(o["accept_len"] == 0) and np.all(o["next_tok"] != draft[:, 1])
    # a one-hot target emits its token whatever happens
    oh = np.full((4 * n, V), -1e9)
    oh[:, 2] = 0.0
    qu = np.full((n, 3, V), 1.0 / V)
    o = rs.rs_accept(draft, keep_len, cu, L, qu, oh, 1.0, 3)
    acc = o["accept_len"]
    assert np.all(o["next_tok"] == 2)
    for i in range(n):
        assert np.all(draft[i, 1:acc[i] + 1] == 2)
        if acc[i] < 3:
            assert draft[i, acc[i] + 1] != 2


def test_rs_accept_respects_keep_len_and_temperature():
    V, n = 6, 50
    rng = np.random.default_rng(12)
    keep_len = rng.integers(1, 5, n).astype(np.int32)
    cu = np.zeros(n + 1, np.int32)
    cu[1:] = np.cumsum(keep_len)
    L = rng.integers(0, 30, n).astype(np.int32)
    draft = rng.integers(0, V, (n, 5)).astype(np.int32)
    logits = rng.normal(size=(int(cu[-1]), V)) * 3
    q = rng.dirichlet(np.ones(V), size=(n, 4))
    o = rs.rs_accept(draft, keep_len, cu, L, q, logits, 0.7, 1)
    assert np.all(o["accept_len"] <= keep_len - 1)
    assert o["total"][0] == int((o["accept_len"] + 1).sum())
    assert np.all((o["next_tok"] >= 0) & (o["next_tok"] < V))
    with pytest.raises(ValueError):
        rs.rs_accept(draft, keep_len, cu, L, q, logits, 0.0, 1)
    lse = rs.lse_rows(logits, 0.7)
    assert np.allclose(np.exp(logits / 0.7 - lse[:, None]).sum(axis=1), 1.0)
