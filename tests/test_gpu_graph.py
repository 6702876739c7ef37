"""Whole verify steps captured into HIP graphs replay the eager results bit for bit.

One graph per batch size: every size the calls take comes from the host and
K* stays on the device, so a captured adaptive step picks its budget anew on
each replay.  Each replay follows eager work that overwrites the outputs (a
different budget), and every replay is compared with the eager step and,
for the greedy steps, with the oracle (selection, packing and acceptance bit
for bit; residual rows, logits and argmax to their tolerances).
"""
import numpy as np
import pytest
import torch

from paper_2607_14647_amd import lib as L
from paper_2607_14647_amd import runner
from paper_2607_14647_amd import workload as wl
from oracle import layer as olay
from tests.gpu_common import check_step, full_workload, need_gpu, note, oracle_step, tiny_variants, workload

pytestmark = pytest.mark.gpu
VARIANTS = tiny_variants()


def _snapshot(vs, logits=None):
    K = int(vs.sel["cu"][-1].item())
    out = {k: vs.host(k) for k in ("choice", "keep_len", "cu", "accept_len", "next_tok", "total")}
    out["argmax"] = vs.host("argmax")[:K]
    out["x"] = vs.x[:K].cpu().numpy()
    if logits is not None:
        out["logits"] = logits[:K].cpu().numpy()
    if vs.q is not None:
        out["lse"] = vs.lse[:K].cpu().numpy()
        out["k_state"] = vs.k_state.cpu().numpy()
    return out


def _check_oracle(ref, snap, what):
    check_step(ref, snap["choice"], snap["keep_len"], snap["cu"], snap["x"], snap["argmax"], snap["accept_len"],
               snap["next_tok"], logits=snap.get("logits"), what=what)


def _same(a, b):
    assert a.keys() == b.keys()
    for k in a:
        assert np.array_equal(a[k], b[k]), k


def _candidates(cfg):
    N = cfg.B * (cfg.D + 1)
    budgets = sorted({cfg.B, cfg.budgets[0], (cfg.B + N) // 2, N})
    costs = [1.0 + 0.002 * K + (0.5 if K > cfg.budgets[0] else 0.0) for K in budgets]
    return budgets, costs


@pytest.mark.parametrize("name", ["cfg1", "split", "qkvsplit", "moe", "long", "plan"])
def test_graph_greedy_step(name):
    need_gpu()
    cfg = VARIANTS[name]
    st, w, kv = workload(cfg, 0)
    vs = runner.VerifyStep(cfg, w, st, kv)
    budgets, costs = _candidates(cfg)
    logits = torch.zeros(vs.rows, cfg.layer.vocab, dtype=torch.float32, device="cuda")

    def step():
        vs.select(budgets, costs)
        vs.verify()
        vs.lm_head(logits=logits)
        vs.accept()
    step()
    torch.cuda.synchronize()
    ref = _snapshot(vs, logits)
    note(f"graph greedy {name}: K*={ref['choice'][0]}")
    oref = oracle_step(cfg, st, olay.prepare_weights(w), kv, budgets, costs)
    _check_oracle(oref, ref, f"eager {name}")
    g = vs.capture(step)
    for rep in range(3):
        vs.step([cfg.B * (cfg.D + 1)], [1.0])          # eager work that overwrites every output
        logits.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        snap = _snapshot(vs, logits)
        _same(snap, ref)
        _check_oracle(oref, snap, f"replay {rep} {name}")


@pytest.mark.parametrize("mode", [L.RS_SCAN, L.RS_HISTORY])
def test_graph_rs_step(mode):
    need_gpu()
    cfg = VARIANTS["cfg1"]
    st, w, kv = workload(cfg, 0)
    prop = wl.make_proposals(cfg, 0, st["draft"][:, 0])
    st = dict(st, conf=prop["conf"], draft=prop["draft"])
    vs = runner.VerifyStep(cfg, w, st, kv)
    vs.enable_rs(prop["q"])
    vs.temperature, vs.seed, vs.rs_mode = 1.0, 99, mode
    budgets, costs = _candidates(cfg)
    step = lambda: vs.step_rs(budgets, costs)
    # eager sequence (the history mode carries its budget from step to step)
    vs.k_state.fill_(budgets[-1])
    eager = []
    for _ in range(3):
        step()
        torch.cuda.synchronize()
        eager.append(_snapshot(vs))
    note(f"graph rs mode {mode}: K* per step {[int(e['choice'][0]) for e in eager]}")
    vs.k_state.fill_(budgets[-1])
    g = vs.capture(step)                 # capture runs the step once more: restart the state
    for rep in range(3):
        if rep == 0:
            vs.k_state.fill_(budgets[-1])
        vs.step([cfg.B], [1.0])           # eager greedy-budget work in between
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        _same(_snapshot(vs), eager[rep])


def test_graph_fullsize_step():
    """The batch-64 step (dense 8B-shaped layer, V = 128256, all candidate budgets) captured
    once and replayed after eager steps at another budget: every replay reproduces the eager
    step bit for bit, including the attention work order built inside the graph."""
    need_gpu()
    cfg, st, w, kv, w64 = full_workload(3, 0)
    vs = runner.VerifyStep(cfg, w, st, kv)
    budgets = list(cfg.budgets)
    costs = [1.0 + K / (2.0 * cfg.B) for K in budgets]
    logits = torch.zeros(vs.rows, cfg.layer.vocab, dtype=torch.float32, device="cuda")

    def step():
        vs.select(budgets, costs)
        vs.verify()
        vs.lm_head(logits=logits)
        vs.accept()
    step()
    torch.cuda.synchronize()
    ref = _snapshot(vs, logits)
    note(f"graph cfg3: K*={ref['choice'][0]}")
    g = vs.capture(step)
    for rep in range(3):
        vs.step([budgets[-1]], [1.0])
        logits.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        snap = _snapshot(vs, logits)
        _same(snap, ref)
    note("graph cfg3: oracle on every kept row of the replayed step")
    _check_oracle(oracle_step(cfg, st, w64, kv, budgets, costs), snap, "replay cfg3")
