"""The startup cost-table protocol (App. C) on the host: budgets per captured
batch size, nearest-batch lookup, profiling order and medians (fake timer)."""
import json
import os

import pytest

from oracle import select as osel
from paper_2607_14647_amd import costtable as ct

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_profile_runs_every_bucket_and_takes_medians():
    calls = []
    steps = {B: (lambda budgets, B=B: calls.append((B, tuple(budgets)))) for B in (16, 1, 8)}

    def timer(fn, n):
        fn_calls = []
        for _ in range(n):
            fn()
            fn_calls.append(calls[-1])
        B, (K,) = fn_calls[-1]
        return [float(B * 1000 + K + j % 3) for j in range(n)]   # median = B*1000 + K + 1

    t = ct.profile(steps, 15, time_ms=timer, reps=5, warmup=1)
    assert t.batch == [1, 8, 16]
    for b, B in enumerate(t.batch):
        Ks = [osel.budget_from_ratio(B, 15, n, d) for n, d in ct.PAPER_RATIOS]
        assert t.ms[b] == [B * 1000 + K + 1 for K in Ks]
        assert [c for c in calls if c[0] == B] == [(B, (K,)) for K in Ks for _ in range(6)]


def test_lookup_uses_the_nearest_captured_batch():
    g = json.load(open(os.path.join(ROOT, "tests", "golden", "cost_table_tab3.json")))
    t = ct.CostTable(g["D"], [tuple(r) for r in g["ratios"]], list(g["B"]), [list(r) for r in g["H20_ms"]])
    assert t.row(64) == (64, list(g["H20_ms"][-1]))
    assert t.row(12)[0] == 16            # tie between 8 and 16 goes to the larger
    assert t.row(40)[0] == 32
    assert t.row(1000)[0] == 64
    budgets, costs = t.candidates(20)
    assert budgets == [osel.budget_from_ratio(20, g["D"], n, d) for n, d in t.ratios]
    assert costs == list(g["H20_ms"][t.batch.index(16)])
    assert ct.CostTable.from_json(t.to_json()) == t


def test_profile_needs_a_timer():
    with pytest.raises(ValueError):
        ct.profile({1: lambda b: None}, 15)
