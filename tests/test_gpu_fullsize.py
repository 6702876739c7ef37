"""Full-size configurations: the GPU step at its real shapes, checked on every kept row.

The whole batch runs on the GPU exactly as the benchmark launches it (all
candidate budgets, device-side K*).  Selection, offsets and packing are
compared bit for bit over the whole batch; the float64 oracle recomputes the
layer and LM head of every kept row of every request, and acceptance is
compared for every request whose deciding rows clear the argmax gap.
Causality at full size: every row kept under a smaller budget (the smallest,
and the quarter budget 4B the benchmark's cost row picks at batch 64) is
bitwise identical, logits and argmax, to the same row at the adaptive budget.
"""
import numpy as np
import pytest
import torch

from oracle import layer as olay
from oracle import lm_head as olm
from oracle import select as osel
from paper_2607_14647_amd import runner
from paper_2607_14647_amd import workload as wl
from tests.gpu_common import (ARGMAX_GAP, LOGIT_RTOL, check_step, full_workload, need_gpu, note,
                              oracle_step, row_rel_err)

pytestmark = pytest.mark.gpu


def _costs(budgets, B):
    # a fixed cost plus a per-position cost: the chosen K* lands inside the grid
    return [1.0 + K / (2.0 * B) for K in budgets]


@pytest.mark.timeout(900)
@pytest.mark.parametrize("cid", [2, 4, 5, 3])   # the batch-64 shape last: later tests reuse it
def test_fullsize_every_row(cid):
    need_gpu()
    note(f"cfg{cid}: generating workload")
    cfg, st, w, kv, w64 = full_workload(cid, 0)
    budgets = list(cfg.budgets)
    costs = _costs(budgets, cfg.B)
    note(f"cfg{cid}: uploading")
    vs = runner.VerifyStep(cfg, w, st, kv)
    ly = cfg.layer
    logits = torch.zeros(vs.rows, ly.vocab, dtype=torch.float32, device="cuda")
    vs.select(budgets, costs)
    vs.verify()
    vs.lm_head(logits=logits)
    vs.accept()
    torch.cuda.synchronize()
    assert int(vs.dev_err.item()) == 0
    K = int(vs.host("cu")[-1])
    note(f"cfg{cid}: K*={K}")
    cu_f, kl_f = vs.host("cu"), vs.host("keep_len")
    x_gpu = vs.x[:K].cpu().numpy()
    lg_gpu = logits[:K].cpu().numpy()
    am_gpu = vs.host("argmax")[:K]
    out = dict(choice=vs.host("choice"), keep_len=kl_f, cu=cu_f, accept_len=vs.host("accept_len"),
               next_tok=vs.host("next_tok"))
    # causality: rows kept under smaller budgets are bitwise the adaptive step's rows
    for Kc in sorted({budgets[0], 4 * cfg.B} & set(budgets)):
        vs.select([Kc], [1.0])
        vs.verify()
        vs.lm_head(logits=logits)
        torch.cuda.synchronize()
        cu_p, kl_p = vs.host("cu"), vs.host("keep_len")
        rows_p = np.concatenate([cu_p[i] + np.arange(min(kl_p[i], kl_f[i])) for i in range(cfg.B)])
        rows_f = np.concatenate([cu_f[i] + np.arange(min(kl_p[i], kl_f[i])) for i in range(cfg.B)])
        note(f"cfg{cid}: causality at K={Kc}: {len(rows_p)} rows")
        lg_p = logits[torch.from_numpy(rows_p).cuda()].cpu().numpy()
        assert np.array_equal(lg_p, lg_gpu[rows_f]), f"logits changed with the budget (K={Kc})"
        # the argmax too, whichever LM-head tile each live row count takes
        assert np.array_equal(vs.host("argmax")[rows_p], am_gpu[rows_f]), f"argmax changed with the budget (K={Kc})"
    del logits, vs
    torch.cuda.empty_cache()
    note(f"cfg{cid}: oracle on every kept row")
    ref = oracle_step(cfg, st, w64, kv, budgets, costs)
    assert np.array_equal(ref["rows"], np.arange(K))
    check_step(ref, out["choice"], out["keep_len"], out["cu"], x_gpu, am_gpu, out["accept_len"], out["next_tok"],
               logits=lg_gpu, what=f"cfg{cid}")


def test_fullsize_sampled_lm_head():
    """dcut_lm_head_sample at the batch-64 shape (V = 128256, 256 kept rows, the budget the
    benchmark picks) with float32 logits and log-partition outputs, as the rejection-sampling step
    launches it: sampled requests against the float64 oracle (logits within the logit tolerance,
    the log-partition within that tolerance over T, the drawn token wherever the top-2 gap of the
    noisy scores exceeds ARGMAX_GAP / T)."""
    from oracle import rs as ors
    from oracle import sampling as osm
    from paper_2607_14647_amd import lib as L

    need_gpu()
    cfg, st, w, kv, w64 = full_workload(3, 0)
    ly = cfg.layer
    K, T, seed = 4 * cfg.B, 1.0, 0x5EED_0001
    vs = runner.VerifyStep(cfg, w, st, kv)
    vs.select([K], [1.0])
    vs.verify()
    logits = torch.zeros(vs.rows, ly.vocab, dtype=torch.float32, device="cuda")
    lse = torch.zeros(vs.rows, dtype=torch.float32, device="cuda")
    L.lm_head_sample(ly.hidden, ly.vocab, cfg.B, cfg.D, vs.sel["cu"], vs.sel["packed_req"], vs.sel["packed_pos"],
                     vs.x, vs.w["final_norm"], ly.rms_eps, vs.w["w_lm"], T, seed, vs.argmax, vs.ws_lm,
                     max_score=vs.max_logit, logits=logits, lse=lse)
    torch.cuda.synchronize()
    assert int(vs.dev_err.item()) == 0
    sel = osel.select(st["conf"], st["draft"], st["ctx_len"], [K], [1.0])
    assert np.array_equal(vs.host("cu"), sel["cu"])
    kl = sel["keep_len"]
    sample = list(dict.fromkeys([int(np.argmax(kl)), int(np.argmin(kl)), int(np.argmax(st["ctx_len"]))]))
    rows = np.concatenate([np.arange(sel["cu"][i], sel["cu"][i + 1]) for i in sample])
    idx = torch.from_numpy(rows).cuda()
    lg_gpu = logits[idx].cpu().numpy()
    lse_gpu = lse[idx].cpu().numpy().astype(np.float64)
    tok_gpu = vs.host("argmax")[rows]
    del logits
    note(f"cfg3 sampled LM head: oracle on requests {sample} ({len(rows)} rows)")
    lay = olay.verify_layer(ly, w64, kv, sel["cu"], sel["packed_tok"], sel["packed_pos"], sel["packed_req"],
                            st["ctx_len"], cfg.D, requests=sample)
    ref = osm.lm_head_sample(lay["x_out"][rows], w64["final_norm"], ly.rms_eps, w64["w_lm"],
                             sel["packed_req"][rows], sel["packed_pos"][rows], T, seed)
    el = row_rel_err(lg_gpu, ref["logits"])
    scale = np.abs(ref["logits"]).max(axis=1)
    e_lse = np.abs(lse_gpu - ors.lse_rows(ref["logits"], T)) / scale
    sure = ref["gap"] > ARGMAX_GAP / T
    note(f"  max rel err logits={el.max():.2e} lse={e_lse.max():.2e}; tokens checked {sure.sum()}/{len(rows)}")
    assert el.max() <= LOGIT_RTOL and e_lse.max() <= LOGIT_RTOL / T
    assert sure.sum() >= len(rows) // 2
    assert np.array_equal(tok_gpu[sure], ref["token"][sure])
