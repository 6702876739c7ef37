"""The startup cost-table protocol of App. C on the GPU.

One graph-captured verify step per captured batch size and ratio bucket,
each forced to its bucket's budget K_rho(B_c) (Eq. dcut-budget) and timed by
HIP events (`costtable.profile` with `event_timer`).  The table's budgets
must equal the oracle's exact ceiling rule, every replay must keep exactly
its forced budget, and a live batch then takes the row of its nearest
captured batch size (ties to the larger): the selection that row drives on
the GPU, and the whole step after it, must match the oracle.
"""
import dataclasses

import numpy as np
import pytest
import torch

from oracle import layer as olay
from oracle import select as osel
from paper_2607_14647_amd import costtable as ct
from paper_2607_14647_amd import runner
from paper_2607_14647_amd import workload as wl
from tests.gpu_common import check_step, need_gpu, note, oracle_step

pytestmark = pytest.mark.gpu


def _batch(Bc):
    base = wl.CONFIGS[1]
    return dataclasses.replace(base, B=Bc, budgets=tuple(Bc * m for m in range(1, base.D + 2)))


def test_cost_table_protocol():
    need_gpu()
    base = wl.CONFIGS[1]
    w = wl.make_weights(base, 0)
    steps, keep, seen = {}, [], {}
    for Bc in (1, 2, 4, 8):
        c2 = _batch(Bc)
        st2 = wl.make_step_inputs(c2, 0)
        kv2 = wl.make_kv(c2, 0, st2["ctx_len"])
        v2 = runner.VerifyStep(c2, w, st2, kv2)
        graphs = {}

        def run(budgets, v2=v2, graphs=graphs, Bc=Bc):
            K = budgets[0]
            if K not in graphs:
                graphs[K] = v2.capture(lambda: v2.step([K], [1.0]))
            graphs[K].replay()
            seen.setdefault(Bc, []).append((K, v2))
        steps[Bc] = run
        keep.append((v2, graphs))
    t = ct.profile(steps, base.D, ct.PAPER_RATIOS, time_ms=ct.event_timer(), reps=5, warmup=1)
    note("cost table (ms): " + "; ".join(f"B={B}: " + ", ".join(f"{x:.3f}" for x in r)
                                         for B, r in zip(t.batch, t.ms)))
    assert t.batch == [1, 2, 4, 8]
    for b, Bc in enumerate(t.batch):
        expect = [osel.budget_from_ratio(Bc, base.D, n, d) for n, d in ct.PAPER_RATIOS]
        assert t.budgets(Bc) == expect
        assert all(np.isfinite(x) and x > 0 for x in t.ms[b])
    # every replay kept exactly its forced budget (the last replay of each batch size is checked)
    for Bc, (v2, graphs) in zip((1, 2, 4, 8), keep):
        K_last = seen[Bc][-1][0]
        torch.cuda.synchronize()
        assert int(v2.host("choice")[0]) == K_last and int(v2.host("cu")[-1]) == K_last
    # a live batch of 3 reads the row of captured size 4 (tie between 2 and 4 goes to the larger)
    live = _batch(3)
    assert t.row(3)[0] == 4
    budgets, costs = t.candidates(3)
    assert budgets == [osel.budget_from_ratio(3, base.D, n, d) for n, d in ct.PAPER_RATIOS]
    assert costs == t.ms[t.batch.index(4)]
    st = wl.make_step_inputs(live, 0)
    kv = wl.make_kv(live, 0, st["ctx_len"])
    vs = runner.VerifyStep(live, w, st, kv)
    vs.step(budgets, costs)
    torch.cuda.synchronize()
    note(f"live batch 3: budgets {budgets}, costs {[round(c, 4) for c in costs]}, K*={vs.host('choice')[0]}")
    ref = oracle_step(live, st, olay.prepare_weights(w), kv, budgets, costs)
    K = int(vs.host("cu")[-1])
    check_step(ref, vs.host("choice"), vs.host("keep_len"), vs.host("cu"), vs.x[:K].cpu().numpy(),
               vs.host("argmax")[:K], vs.host("accept_len"), vs.host("next_tok"), what="cost-table row step")
    assert np.array_equal(vs.host("benefit")[: len(budgets)].astype(np.uint64), ref["sel"]["benefit"])
