"""Rejection-sampling verification on the GPU versus the oracle (App. B).

- dcut_select_rs: shifted scores, the causal early-stopping scan and the fixed
  budget; keep depths, offsets, packing, choice and benefits bit for bit.
- dcut_accept_rs on oracle-made inputs (logits, log-partition values, the
  target's draws): accepted lengths wherever the deciding comparison
  u q(z) < p(z) is not within 1e-4 (log scale) of a tie, committed tokens
  wherever the residual draw's top-2 gap exceeds 1e-3.
- dcut_lm_head_sample's logits and log-partition outputs within the logit
  tolerance.
- One whole RS step (select_rs, verify, sampled LM head, accept_rs) against
  the oracle's float64 step, gated by the logit tolerance carried into the
  decisions.
"""
import json
import os

import numpy as np
import pytest
import torch

from oracle import layer as olay
from oracle import lm_head as olm
from oracle import rs as ors
from oracle import sampling as osm
from paper_2607_14647_amd import lib as L
from paper_2607_14647_amd import runner
from paper_2607_14647_amd import workload as wl
from tests.gpu_common import LOGIT_RTOL, need_gpu, note, row_rel_err, tiny_variants, to_dev, workload

pytestmark = pytest.mark.gpu
VARIANTS = tiny_variants()
GOLD = os.path.join(os.path.dirname(__file__), "golden")
SEED = 0x51D_0_5EED


# ---------------------------------------------------------------- selection

def gpu_select_rs(conf, draft, ctx, mode, budgets, costs, k_state=None):
    B, D1 = draft.shape
    D = D1 - 1
    out = L.select_outputs(B, D, len(budgets))
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    c = to_dev(conf.astype(np.float32)) if D > 0 else torch.zeros(1, device="cuda")
    L.select_rs(B, D, c, to_dev(draft), to_dev(ctx), mode, budgets, costs, out, err, k_state=k_state)
    torch.cuda.synchronize()
    return {k: v.cpu().numpy() for k, v in out.items()}, int(err.item())


def check_select(conf, draft, ctx, mode, budgets, costs):
    got, err = gpu_select_rs(conf, draft, ctx, mode, budgets, costs)
    ref = ors.select_rs(conf, draft, ctx, mode, budgets, costs)
    assert err == 0
    K = int(ref["choice"][0])
    assert got["choice"].tolist() == ref["choice"].tolist()
    assert np.array_equal(got["keep_len"], ref["keep_len"])
    assert np.array_equal(got["cu"], ref["cu"])
    assert np.array_equal(got["benefit"][: len(budgets)].view(np.uint64), ref["benefit"])
    for k in ("packed_tok", "packed_pos", "packed_req"):
        assert np.array_equal(got[k][:K], ref[k][:K]), k
    return ref


def _costs(rng, budgets, monotone=True):
    K = np.asarray(budgets, dtype=np.float64)
    a, b, c = rng.uniform(0.1, 5.0), rng.uniform(0.0, 0.02), rng.uniform(0.0, 2e-5)
    cost = a + b * K + c * K * K
    if not monotone:
        cost = cost * rng.uniform(0.7, 1.3, size=len(budgets))
    return cost.tolist()


SEL_CASES = [(cid, seed) for cid in (1, 2, 3, 4, 5) for seed in range(4)] + [(1, s) for s in range(4, 40)]


@pytest.mark.parametrize("cid,seed", SEL_CASES)
def test_select_rs_configs(cid, seed):
    need_gpu()
    cfg = wl.CONFIGS[cid]
    st = wl.make_step_inputs(cfg, seed)
    rng = np.random.default_rng(2000 + seed)
    budgets = list(cfg.budgets)
    note(f"select_rs cfg{cid} seed{seed} B={cfg.B}")
    ref = check_select(st["conf"], st["draft"], st["ctx_len"], L.RS_SCAN, budgets, _costs(rng, budgets))
    assert int(ref["choice"][0]) >= cfg.B
    check_select(st["conf"], st["draft"], st["ctx_len"], L.RS_SCAN, budgets, _costs(rng, budgets, False))
    K = int(rng.integers(cfg.B, cfg.B * (cfg.D + 1) + 1))
    check_select(st["conf"], st["draft"], st["ctx_len"], L.RS_FIXED, [K], [1.0])


@pytest.mark.parametrize("cid", [1, 2, 3, 4, 5])
def test_select_rs_history_chain(cid):
    """History-based K over four consecutive blocks: each step's budget is the
    previous block's choice, carried in the device state word."""
    need_gpu()
    cfg = wl.CONFIGS[cid]
    budgets = list(cfg.budgets) if len(cfg.budgets) > 1 else [cfg.B, cfg.budgets[0], cfg.B * (cfg.D + 1)]
    rng = np.random.default_rng(77 + cid)
    costs = _costs(rng, budgets)
    k_state = torch.full((1,), budgets[-1], dtype=torch.int32, device="cuda")
    k_ref = budgets[-1]
    for t in range(4):
        st = wl.make_step_inputs(cfg, 100 + t)
        got, err = gpu_select_rs(st["conf"], st["draft"], st["ctx_len"], L.RS_HISTORY, budgets, costs, k_state)
        ref = ors.select_rs(st["conf"], st["draft"], st["ctx_len"], ors.HISTORY, budgets, costs, k_state=k_ref)
        note(f"history cfg{cid} step {t}: K*={int(ref['choice'][0])} next={ref['k_next']}")
        assert err == 0
        assert got["choice"].tolist() == ref["choice"].tolist()
        assert np.array_equal(got["keep_len"], ref["keep_len"])
        assert np.array_equal(got["benefit"][: len(budgets)].view(np.uint64), ref["benefit"])
        assert int(k_state.item()) == ref["k_next"]
        k_ref = ref["k_next"]


def test_select_rs_hand_example():
    need_gpu()
    g = json.load(open(os.path.join(GOLD, "rs_scan_example.json")))
    conf = np.array(g["conf"], np.float32)
    z = np.array([[5, 6, 7], [8, 9, 10]], np.int32)
    for case in g["cases"]:
        got, err = gpu_select_rs(conf, z, np.array([3, 4], np.int32), L.RS_SCAN, g["budgets"], case["costs"])
        assert err == 0
        assert got["choice"].tolist() == [case["K"], case["r"]]
        assert got["keep_len"].tolist() == case["keep_len"]


@pytest.mark.parametrize("B,D,R", [(1024, 7, 8), (4096, 1, 3), (512, 15, 16), (1, 63, 4), (300, 0, 1),
                                   (64, 15, 64)])
def test_select_rs_shapes(B, D, R):
    """Several ranks per thread (B(D+1) = 8192), the largest batch, one
    request, a bonus-only block, and the most candidate budgets."""
    need_gpu()
    rng = np.random.default_rng(B * 131 + D)
    conf = rng.random((B, D)).astype(np.float32) ** 0.3
    conf[rng.random((B, D)) < 0.05] = 0.0
    conf[rng.random((B, D)) < 0.05] = 1.0
    draft = rng.integers(0, 1000, (B, D + 1)).astype(np.int32)
    ctx = rng.integers(0, 5000, B).astype(np.int32)
    N = B * (D + 1)
    budgets = sorted(int(x) for x in rng.integers(B, N + 1, size=R))
    note(f"select_rs shapes B={B} D={D} R={R}")
    check_select(conf, draft, ctx, L.RS_SCAN, budgets, _costs(rng, budgets))
    check_select(conf, draft, ctx, L.RS_SCAN, budgets, _costs(rng, budgets, False))
    check_select(conf, draft, ctx, L.RS_FIXED, [budgets[-1]], [2.0])


def test_select_rs_closed_forms():
    need_gpu()
    B, D = 64, 15
    N = B * (D + 1)
    z = np.zeros((B, D + 1), np.int32)
    L0 = np.zeros(B, np.int32)
    ones = np.ones((B, D), np.float32)
    got, _ = gpu_select_rs(ones, z, L0, L.RS_SCAN, [B, N], [float(B), float(N)])
    assert got["choice"].tolist() == [B, 0]
    got, _ = gpu_select_rs(ones, z, L0, L.RS_SCAN, [B, N], [float(B + 1), float(N + 1)])
    assert got["choice"].tolist() == [N, 1]
    rng = np.random.default_rng(1)
    conf = rng.uniform(0.05, 1.0, (B, D)).astype(np.float32)
    got, _ = gpu_select_rs(conf, z, L0, L.RS_SCAN, [B], [3.0])
    assert got["choice"][0] == N


def test_select_rs_flags_bad_confidence():
    need_gpu()
    rng = np.random.default_rng(3)
    B, D = 8, 5
    conf = rng.random((B, D)).astype(np.float32)
    conf[2, 1] = np.nan
    conf[5, 4] = 1.5                  # the last depth's confidence enters no shifted score
    z = np.zeros((B, D + 1), np.int32)
    got, err = gpu_select_rs(conf, z, np.zeros(B, np.int32), L.RS_FIXED, [20], [1.0])
    assert err & L.DERR_CONF
    clean = conf.copy()
    clean[2, 1] = 0.0
    clean[5, 4] = 0.0
    ref = ors.select_rs(clean, z, np.zeros(B, np.int32), ors.FIXED, [20], [1.0])
    assert np.array_equal(got["keep_len"], ref["keep_len"])


# ---------------------------------------------------------------- acceptance on oracle-made inputs

def _rs_inputs(seed, B, D, V, T, scale=2.0, q_mode="related"):
    """Logits, proposals and drafts with a tunable target/proposal overlap."""
    rng = np.random.default_rng(seed)
    rows = B * (D + 1)
    keep_len = rng.integers(1, D + 2, B).astype(np.int32)
    cu = np.zeros(B + 1, np.int32)
    cu[1:] = np.cumsum(keep_len)
    ctx = rng.integers(0, 3000, B).astype(np.int32)
    logits = (rng.standard_normal((rows, V)) * scale).astype(np.float32)
    q = np.empty((B, D, V), np.float32)
    draft = np.zeros((B, D + 1), np.int32)
    draft[:, 0] = rng.integers(0, V, B)
    for i in range(B):
        for j in range(1, D + 1):
            r = cu[i] + j - 1 if j < keep_len[i] else rows - 1
            if q_mode == "related":       # the target's row, perturbed and sharpened
                g = logits[r].astype(np.float64) / T + rng.standard_normal(V) * 0.7
                g *= rng.uniform(0.8, 1.6)
            else:
                g = rng.standard_normal(V) * 3.0
            e = np.exp(g - g.max())
            q[i, j - 1] = (e / e.sum()).astype(np.float32)
            cdf = np.cumsum(q[i, j - 1].astype(np.float64))
            draft[i, j] = min(int((cdf < rng.random() * cdf[-1]).sum()), V - 1)
    req = np.zeros(rows, np.int32)
    pos = np.zeros(rows, np.int32)
    for i in range(B):
        for k in range(keep_len[i]):
            req[cu[i] + k] = i
            pos[cu[i] + k] = ctx[i] + k
    K = int(cu[-1])
    lse = ors.lse_rows(logits[:K], T).astype(np.float32)
    token = osm.sample_tokens(logits[:K], req[:K], pos[:K], T, SEED)["token"]
    return dict(keep_len=keep_len, cu=cu, ctx=ctx, logits=logits, q=q, draft=draft, pos=pos, K=K, lse=lse,
                token=token)


def gpu_accept_rs(x, B, D, V, T, ctx_inout=None):
    rows = B * (D + 1)
    lse = np.zeros(rows, np.float32)
    lse[: x["K"]] = x["lse"]
    tok = np.zeros(rows, np.int32)
    tok[: x["K"]] = x["token"]
    i32 = dict(dtype=torch.int32, device="cuda")
    acc, nxt, tot = torch.zeros(B, **i32), torch.zeros(B, **i32), torch.zeros(1, **i32)
    err = torch.zeros(1, **i32)
    cfg = L.LayerCfg(8, 1, 1, 8, 8, 0, 0, 0, V, 8, 1e-5, 1e4)
    ws = L.workspace(L.workspace_bytes(4, cfg, B, D))
    q = to_dev(x["q"]) if D > 0 else torch.zeros(1, device="cuda")
    L.accept_rs(B, D, V, T, SEED, to_dev(x["draft"]), q, to_dev(x["keep_len"]), to_dev(x["cu"]),
                to_dev(x["pos"]), to_dev(x["logits"]), to_dev(lse), to_dev(tok), acc, nxt, tot, ws,
                ctx_inout, err)
    torch.cuda.synchronize()
    return acc.cpu().numpy(), nxt.cpu().numpy(), int(tot.item()), int(err.item())


def _compare(x, got_acc, got_nxt, got_tot, T, min_frac=0.9):
    ref = ors.rs_accept(x["draft"], x["keep_len"], x["cu"], x["ctx"], x["q"],
                        x["logits"].astype(np.float64), T, SEED)
    dec = ref["margin"] > 1e-4
    drawn = dec & ((ref["rej_row"] < 0) | (ref["gap"] > 1e-3))
    B = len(dec)
    note(f"  requests {B}: decisions checked {dec.sum()}, tokens checked {drawn.sum()}, "
         f"rejections {int((ref['rej_row'] >= 0).sum())}, accepted {int(ref['accept_len'].sum())}")
    assert dec.sum() >= min_frac * B and drawn.sum() >= min_frac * B
    assert np.array_equal(got_acc[dec], ref["accept_len"][dec])
    assert np.array_equal(got_nxt[drawn], ref["next_tok"][drawn])
    if dec.all():
        assert got_tot == int(ref["total"][0])
    return ref


@pytest.mark.parametrize("B,D,V,T,scale,qm", [
    (32, 15, 1024, 1.0, 2.0, "related"), (32, 15, 1024, 0.7, 1.5, "related"),
    (16, 7, 5000, 1.0, 3.0, "related"), (24, 15, 1024, 1.0, 1.0, "unrelated"),
    (8, 3, 130, 1.0, 2.0, "related"), (200, 3, 64, 1.0, 1.0, "related"), (4, 15, 32768, 1.0, 2.5, "related"),
])
def test_accept_rs_parity(B, D, V, T, scale, qm):
    need_gpu()
    note(f"accept_rs B={B} D={D} V={V} T={T} {qm}")
    x = _rs_inputs(B * 7 + V, B, D, V, T, scale, qm)
    acc, nxt, tot, err = gpu_accept_rs(x, B, D, V, T)
    assert err == 0
    ref = _compare(x, acc, nxt, tot, T)
    assert np.all(acc <= x["keep_len"] - 1)


def test_accept_rs_all_accepted_and_bonus_only():
    need_gpu()
    B, D, V, T = 16, 7, 700, 1.0
    x = _rs_inputs(5, B, D, V, T)
    # proposals equal to the target rows: every kept draft passes (u < 1)
    for i in range(B):
        for j in range(1, int(x["keep_len"][i])):
            x["q"][i, j - 1] = ors.target_probs(x["logits"][x["cu"][i] + j - 1], T).astype(np.float32)
    acc, nxt, tot, err = gpu_accept_rs(x, B, D, V, T)
    assert np.array_equal(acc, x["keep_len"] - 1)
    assert np.array_equal(nxt, x["token"][x["cu"][1:] - 1])
    assert tot == int(x["keep_len"].sum())
    # D = 0: the bonus position only
    x0 = _rs_inputs(6, B, 0, V, T)
    ctx_io = to_dev(x0["ctx"].copy())
    acc, nxt, tot, err = gpu_accept_rs(x0, B, 0, V, T, ctx_inout=ctx_io)
    assert np.all(acc == 0) and np.array_equal(nxt, x0["token"][x0["cu"][:-1]]) and tot == B
    assert np.array_equal(ctx_io.cpu().numpy(), x0["ctx"] + 1)


def test_accept_rs_target_excludes_a_draft():
    """A draft the target gives probability 0 is rejected and never re-emitted."""
    need_gpu()
    B, D, V, T = 12, 5, 300, 1.0
    x = _rs_inputs(8, B, D, V, T)
    x["keep_len"][:] = D + 1
    x["cu"][1:] = np.cumsum(x["keep_len"])
    rows = x["cu"][:-1]
    x["logits"][rows, x["draft"][:, 1]] = -np.inf
    pos = np.zeros(B * (D + 1), np.int32)
    req = np.zeros(B * (D + 1), np.int32)
    for i in range(B):
        for k in range(D + 1):
            pos[x["cu"][i] + k] = x["ctx"][i] + k
            req[x["cu"][i] + k] = i
    x["pos"] = pos
    x["K"] = int(x["cu"][-1])
    lg = x["logits"][: x["K"]]
    x["lse"] = ors.lse_rows(lg, T).astype(np.float32)
    x["token"] = osm.sample_tokens(lg, req[: x["K"]], pos[: x["K"]], T, SEED)["token"]
    acc, nxt, tot, err = gpu_accept_rs(x, B, D, V, T)
    assert np.all(acc == 0) and np.all(nxt != x["draft"][:, 1])
    _compare(x, acc, nxt, tot, T)


def test_accept_rs_flags_invalid_drafts():
    need_gpu()
    B, D, V, T = 6, 4, 256, 1.0
    x = _rs_inputs(9, B, D, V, T)
    x["keep_len"][:] = D + 1
    x["cu"][1:] = np.cumsum(x["keep_len"])
    x["K"] = int(x["cu"][-1])
    x["lse"] = ors.lse_rows(x["logits"][: x["K"]], T).astype(np.float32)
    x["token"] = np.zeros(x["K"], np.int32)
    for i in range(B):
        x["q"][i] = 1.0 / V                                  # uniform proposals ...
        x["logits"][x["cu"][i]: x["cu"][i] + D + 1] = 0.0    # ... against a uniform target: all pass
    x["lse"] = ors.lse_rows(x["logits"][: x["K"]], T).astype(np.float32)
    x["draft"][2, 3] = V + 5
    x["draft"][4, 1] = -1
    acc, nxt, tot, err = gpu_accept_rs(x, B, D, V, T)
    assert err & L.DERR_TOKEN
    assert acc[2] == 2 and acc[4] == 0
    assert np.all(np.delete(acc, [2, 4]) == D)


# ---------------------------------------------------------------- LM head outputs and the whole step

def _lm_rows(cfg, st, w64, kv, sel):
    lay = olay.verify_layer(cfg.layer, w64, kv, sel["cu"], sel["packed_tok"], sel["packed_pos"],
                            sel["packed_req"], st["ctx_len"], cfg.D)
    K = int(sel["cu"][-1])
    lm = olm.lm_head_argmax(lay["x_out"][:K], w64["final_norm"], cfg.layer.rms_eps, w64["w_lm"])
    return lay, lm


@pytest.mark.parametrize("name", ["cfg1", "split", "long"])
@pytest.mark.parametrize("T", [1.0, 0.6])
def test_rs_step(name, T):
    need_gpu()
    cfg = VARIANTS[name]
    st, w, kv = workload(cfg, 0)
    prop = wl.make_proposals(cfg, 0, st["draft"][:, 0])
    st = dict(st, conf=prop["conf"], draft=prop["draft"])
    w64 = olay.prepare_weights(w)
    N = cfg.B * (cfg.D + 1)
    budgets = sorted({cfg.B, max(cfg.B, N // 4), max(cfg.B, N // 2), N})
    rng = np.random.default_rng(11)
    costs = _costs(rng, budgets)
    note(f"rs step {name} T={T} budgets={budgets}")
    vs = runner.VerifyStep(cfg, w, st, kv)
    vs.enable_rs(prop["q"])
    vs.temperature, vs.seed = T, SEED
    vs.select_rs(L.RS_SCAN, budgets, costs)
    vs.verify()
    vs.lm_head()
    vs.accept_rs()
    torch.cuda.synchronize()
    assert int(vs.dev_err.item()) == 0
    sel = ors.select_rs(st["conf"], st["draft"], st["ctx_len"], ors.SCAN, budgets, costs)
    K = int(sel["cu"][-1])
    assert vs.host("choice").tolist() == sel["choice"].tolist()
    assert np.array_equal(vs.host("keep_len"), sel["keep_len"])
    _, lm = _lm_rows(cfg, st, w64, kv, sel)
    # LM-head outputs: logits and the log-partition function of every kept row
    lg = vs.logits[:K].cpu().numpy()
    assert row_rel_err(lg, lm["logits"]).max() <= LOGIT_RTOL
    scale = np.abs(lm["logits"]).max(axis=1)
    lse_ref = ors.lse_rows(lm["logits"], T)
    assert np.all(np.abs(vs.lse[:K].cpu().numpy() - lse_ref) <= LOGIT_RTOL * scale / T + 1e-5)
    # acceptance, gated by how far the logit tolerance can move each decision
    ref = ors.rs_accept(st["draft"], sel["keep_len"], sel["cu"], st["ctx_len"], prop["q"], lm["logits"], T, SEED)
    tol = np.array([2 * LOGIT_RTOL * scale[sel["cu"][i]: sel["cu"][i + 1]].max() / T for i in range(cfg.B)])
    dec = ref["margin"] > tol
    drawn = dec & (ref["gap"] > tol)
    acc, nxt = vs.host("accept_len"), vs.host("next_tok")
    note(f"  K*={K}: decisions checked {dec.sum()}/{cfg.B}, tokens checked {drawn.sum()}, "
         f"rejections {int((ref['rej_row'] >= 0).sum())}")
    assert dec.sum() >= cfg.B // 2
    assert np.array_equal(acc[dec], ref["accept_len"][dec])
    assert np.array_equal(nxt[drawn], ref["next_tok"][drawn])
    assert np.all(acc <= sel["keep_len"] - 1)
    assert int(vs.total.item()) == int((acc + 1).sum())
