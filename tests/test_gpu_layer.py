"""Verify layer + LM head + accept on the GPU versus the float64 oracle (tiny layer and its variants).

Tolerances (written here, derived in the design notes): logits and residual
rows within 2e-2 of the oracle, relative to the row's largest magnitude;
argmax identical wherever the oracle's top-2 gap exceeds 1e-2; selection,
offsets and acceptance bit-exact.  Determinism and causality are bitwise.
"""
import numpy as np
import pytest
import torch

from oracle import accept as oacc
from oracle import drafts as odr
from oracle import layer as olay
from oracle import lm_head as olm
from oracle import select as osel
from paper_2607_14647_amd import lib as L
from paper_2607_14647_amd import runner
from tests.gpu_common import (ARGMAX_GAP, LOGIT_RTOL, ROUTER_GAP, X_RTOL, edge_variants, need_gpu, note,
                              row_rel_err, tiny_variants, workload)

pytestmark = pytest.mark.gpu
VARIANTS = tiny_variants()
EDGES = edge_variants()


def _gpu_run(cfg, st, w, kv, budgets, costs, draft=None):
    vs = runner.VerifyStep(cfg, w, st, kv)
    if draft is not None:
        vs.set_draft(draft)
    logits = torch.zeros(vs.rows, cfg.layer.vocab, dtype=torch.float32, device="cuda")
    vs.select(budgets, costs)
    vs.verify()
    vs.lm_head(logits=logits)
    vs.accept()
    torch.cuda.synchronize()
    return vs, logits.cpu().numpy()


def _oracle(cfg, st, w64, kv, K, draft=None):
    z = st["draft"] if draft is None else draft
    sel = osel.select(st["conf"], z, st["ctx_len"], [K], [1.0])
    lay = olay.verify_layer(cfg.layer, w64, kv, sel["cu"], sel["packed_tok"], sel["packed_pos"],
                            sel["packed_req"], st["ctx_len"], cfg.D)
    lm = olm.lm_head_argmax(lay["x_out"], w64["final_norm"], cfg.layer.rms_eps, w64["w_lm"])
    acc = oacc.accept(z, sel["keep_len"], sel["cu"], lm["argmax"])
    return sel, lay, lm, acc


@pytest.mark.parametrize("name", list(VARIANTS))
@pytest.mark.parametrize("seed", [0, 1])
def test_layer_parity(name, seed):
    need_gpu()
    _layer_parity(VARIANTS[name], name, seed)


@pytest.mark.parametrize("name", list(EDGES))
def test_layer_parity_at_the_limits(name):
    need_gpu()
    _layer_parity(EDGES[name], name, 0)


def _layer_parity(cfg, name, seed):
    st, w, kv = workload(cfg, seed)
    w64 = olay.prepare_weights(w)
    K = cfg.budgets[0]
    note(f"layer parity {name} seed{seed} B={cfg.B} K={K}")
    vs, logits = _gpu_run(cfg, st, w, kv, [K], [1.0])
    sel, lay, lm, acc = _oracle(cfg, st, w64, kv, K)
    assert int(vs.dev_err.item()) == 0
    assert np.array_equal(vs.host("cu"), sel["cu"])
    x = vs.x.cpu().numpy()[:K]
    # MoE: rows whose routing is a near-tie in the oracle are not compared
    ok = lay["router_gap"] > ROUTER_GAP if "router_gap" in lay else np.ones(K, bool)
    ex = row_rel_err(x[ok], lay["x_out"][ok])
    ly = cfg.layer
    # appended keys / values, and every other cache slot untouched
    kg = vs.kv["k"].cpu().numpy().view(np.uint16)
    vg = vs.kv["v"].cpu().numpy().view(np.uint16)
    hd, nkv = ly.head_dim, ly.n_kv
    ek = []
    touched = np.zeros(kg.shape, bool)
    for t in range(K):
        i = int(sel["packed_req"][t])
        slot = int(sel["packed_pos"][t])
        cap, base = int(kv["cap"][i]), int(kv["base"][i])
        for g in range(nkv):
            off = base + (g * cap + slot) * hd
            touched[off: off + hd] = True
            gk = olay.bf16_bits_to_f64(kg[off: off + hd])
            gv = olay.bf16_bits_to_f64(vg[off: off + hd])
            ek.append(np.abs(gk - lay["new_k"][t, g]).max() / np.abs(lay["new_k"][t, g]).max())
            ek.append(np.abs(gv - lay["new_v"][t, g]).max() / np.abs(lay["new_v"][t, g]).max())
    assert np.array_equal(kg[~touched], kv["k"][~touched])
    assert np.array_equal(vg[~touched], kv["v"][~touched])
    el = row_rel_err(logits[:K][ok], lm["logits"][ok])
    am = vs.host("argmax")[:K]
    sure = (lm["gap"] > ARGMAX_GAP) & ok
    note(f"  max rel err x={ex.max():.2e} kv={max(ek):.2e} logits={el.max():.2e}; "
         f"argmax rows checked {sure.sum()}/{K}; rows compared {ok.sum()}/{K}")
    assert ex.max() <= X_RTOL and max(ek) <= X_RTOL and el.max() <= LOGIT_RTOL
    assert np.array_equal(am[sure], lm["argmax"][sure])
    # max_logit is the logit at the argmax
    ml = vs.max_logit.cpu().numpy()[:K]
    assert np.array_equal(ml, logits[np.arange(K), am])


@pytest.mark.parametrize("name", ["plan", "plan1024"])
def test_attention_plan_runs_every_item(name):
    """The layer scratch is filled with NaN bit patterns before the call, so an attention
    work item that the longest-first plan dropped would leave NaN partials or rows."""
    need_gpu()
    cfg = {**VARIANTS, **EDGES}[name]
    st, w, kv = workload(cfg, 0)
    K = cfg.budgets[0]
    vs = runner.VerifyStep(cfg, w, st, kv)
    vs.ws_layer.fill_(255)
    vs.select([K], [1.0])
    vs.verify()
    torch.cuda.synchronize()
    sel, lay, _, _ = _oracle(cfg, st, olay.prepare_weights(w), kv, K)
    x = vs.x.cpu().numpy()[:K]
    assert np.isfinite(x).all()
    ex = row_rel_err(x, lay["x_out"])
    note(f"plan variant {name}: B={cfg.B}, {K} rows, x err {ex.max():.2e}")
    assert ex.max() <= X_RTOL


@pytest.mark.parametrize("name", ["cfg1", "long"])
def test_end_to_end_accept_with_forced_drafts(name):
    """Drafts forced from the oracle's greedy tokens; acceptance must match the oracle."""
    need_gpu()
    cfg = VARIANTS[name]
    st, w, kv = workload(cfg, 0)
    w64 = olay.prepare_weights(w)
    z = odr.force_matches(cfg.layer, w64, kv, st["conf"], st["draft"], st["match_u"],
                          st["ctx_len"], cfg.D)
    B, D = cfg.B, cfg.D
    checked = 0
    for K in (cfg.budgets[0], B * (D + 1)):
        vs, _ = _gpu_run(cfg, st, w, kv, [K], [1.0], draft=z)
        sel, lay, lm, acc = _oracle(cfg, st, w64, kv, K, draft=z)
        ga, gn = vs.host("accept_len"), vs.host("next_tok")
        cu = sel["cu"]
        excluded = 0
        for i in range(B):
            a = int(acc["accept_len"][i])
            decisive = lm["gap"][cu[i]: cu[i] + min(a, sel["keep_len"][i] - 1) + 1]
            if (decisive <= ARGMAX_GAP).any():
                excluded += 1
                continue
            assert ga[i] == a and gn[i] == acc["next_tok"][i]
            checked += 1
        note(f"e2e {name} K={K}: accepted {int(acc['total'][0])} tokens, "
             f"requests with a near-tie decisive row (not compared) {excluded}/{B}")
    assert checked >= 2


@pytest.mark.parametrize("name", ["cfg1", "long", "wide", "deep", "moe", "moe128"])
def test_determinism_and_causality(name):
    """Same inputs -> identical bits; a kept row's outputs do not depend on the budget."""
    need_gpu()
    cfg = VARIANTS[name]
    st, w, kv = workload(cfg, 0)
    B, D = cfg.B, cfg.D
    full = B * (D + 1)
    v1, l1 = _gpu_run(cfg, st, w, kv, [full], [1.0])
    x1, a1 = v1.x.cpu().numpy(), v1.host("argmax")
    v2, l2 = _gpu_run(cfg, st, w, kv, [full], [1.0])
    assert np.array_equal(x1, v2.x.cpu().numpy()) and np.array_equal(l1, l2)
    Kp = cfg.budgets[0]
    vp, lp = _gpu_run(cfg, st, w, kv, [Kp], [1.0])
    cf, cp = v1.host("cu"), vp.host("cu")
    kl = vp.host("keep_len")
    xp, ap = vp.x.cpu().numpy(), vp.host("argmax")
    n = 0
    for i in range(B):
        for k in range(int(kl[i])):
            tf, tp = cf[i] + k, cp[i] + k
            assert np.array_equal(x1[tf], xp[tp]), (i, k)
            assert np.array_equal(l1[tf], lp[tp]), (i, k)
            assert a1[tf] == ap[tp]
            n += 1
    note(f"causality {name}: {n} kept rows bitwise equal at K={Kp} and K={full}")


def test_argmax_tie_rule():
    """Duplicate LM-head rows give exactly equal logits; the lower id must win."""
    need_gpu()
    cfg = VARIANTS["cfg1"]
    st, w, kv = workload(cfg, 0)
    w = dict(w)
    lm = w["w_lm"].copy()
    lm[512:1024] = lm[0:512]
    w["w_lm"] = lm
    vs, logits = _gpu_run(cfg, st, w, kv, [cfg.budgets[0]], [1.0])
    K = cfg.budgets[0]
    am = vs.host("argmax")[:K]
    assert (am < 512).all()
    assert np.array_equal(am, np.argmax(logits[:K], axis=1))
