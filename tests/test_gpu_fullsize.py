"""Full-size dense configurations: the GPU step at its real shapes, checked on sampled requests.

The whole batch runs on the GPU exactly as the benchmark launches it (all
candidate budgets, device-side K*); selection is compared bit for bit over
the whole batch, and the float64 oracle recomputes every kept row of a few
sampled requests (the largest and smallest keep depth and the longest
context).  Causality at full size: the sampled rows are bitwise identical
under the smallest budget and under the quarter budget 4B (the budget the
benchmark's cost row picks at batch 64).
"""
import numpy as np
import pytest
import torch

from oracle import layer as olay
from oracle import lm_head as olm
from oracle import select as osel
from paper_2607_14647_amd import runner
from paper_2607_14647_amd import workload as wl
from tests.gpu_common import ARGMAX_GAP, LOGIT_RTOL, ROUTER_GAP, X_RTOL, need_gpu, note, row_rel_err

pytestmark = pytest.mark.gpu


def _costs(budgets, B):
    # a fixed cost plus a per-position cost: the chosen K* lands inside the grid
    return [1.0 + K / (2.0 * B) for K in budgets]


@pytest.mark.parametrize("cid", [2, 3, 4, 5])
def test_fullsize_sampled_requests(cid):
    need_gpu()
    cfg = wl.CONFIGS[cid]
    seed = 0
    note(f"cfg{cid}: generating workload")
    st = wl.make_step_inputs(cfg, seed)
    w = wl.make_weights(cfg, seed)
    kv = wl.make_kv(cfg, seed, st["ctx_len"])
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
    sel = osel.select(st["conf"], st["draft"], st["ctx_len"], budgets, costs)
    K = int(sel["choice"][0])
    note(f"cfg{cid}: K*={K}")
    assert vs.host("choice").tolist() == sel["choice"].tolist()
    assert np.array_equal(vs.host("keep_len"), sel["keep_len"])
    assert int(vs.dev_err.item()) == 0
    kl = sel["keep_len"]
    sample = list(dict.fromkeys([int(np.argmax(kl)), int(np.argmin(kl)), int(np.argmax(st["ctx_len"]))]))
    rows = np.concatenate([np.arange(sel["cu"][i], sel["cu"][i + 1]) for i in sample])
    x_gpu = vs.x[torch.from_numpy(rows).cuda()].cpu().numpy()
    lg_gpu = logits[torch.from_numpy(rows).cuda()].cpu().numpy()
    am_gpu = vs.host("argmax")[rows]
    # more runs at other budgets for the causality check
    for Kc in sorted({budgets[0], 4 * cfg.B} & set(budgets)):
        vs.select([Kc], [1.0])
        vs.verify()
        vs.lm_head(logits=logits)
        torch.cuda.synchronize()
        cu_p = vs.host("cu")
        kl_p = vs.host("keep_len")
        rows_p, rows_f = [], []
        for i in sample:
            for k in range(min(int(kl_p[i]), int(kl[i]))):
                rows_p.append(cu_p[i] + k)
                rows_f.append(int(np.where(rows == sel["cu"][i] + k)[0][0]))
        note(f"cfg{cid}: causality at K={Kc}: {len(rows_p)} rows")
        lg_p = logits[torch.tensor(rows_p, device="cuda")].cpu().numpy()
        assert np.array_equal(lg_p, lg_gpu[rows_f]), f"logits changed with the budget (K={Kc})"
        # the argmax too, whichever LM-head tile each live row count takes
        assert np.array_equal(vs.host("argmax")[rows_p], am_gpu[rows_f]), f"argmax changed with the budget (K={Kc})"
    del logits
    note(f"cfg{cid}: oracle on requests {sample} ({len(rows)} rows)")
    w64 = olay.prepare_weights(w)
    lay = olay.verify_layer(ly, w64, kv, sel["cu"], sel["packed_tok"], sel["packed_pos"],
                            sel["packed_req"], st["ctx_len"], cfg.D, requests=sample)
    lm = olm.lm_head_argmax(lay["x_out"][rows], w64["final_norm"], ly.rms_eps, w64["w_lm"])
    ok = lay["router_gap"][rows] > ROUTER_GAP if "router_gap" in lay else np.ones(len(rows), bool)
    ex = row_rel_err(x_gpu[ok], lay["x_out"][rows][ok])
    el = row_rel_err(lg_gpu[ok], lm["logits"][ok])
    sure = (lm["gap"] > ARGMAX_GAP) & ok
    note(f"cfg{cid}: max rel err x={ex.max():.2e} logits={el.max():.2e}; argmax rows {sure.sum()}/{len(rows)}; "
         f"rows compared {ok.sum()}/{len(rows)}")
    assert ex.max() <= X_RTOL and el.max() <= LOGIT_RTOL
    assert np.array_equal(am_gpu[sure], lm["argmax"][sure])


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
    cfg = wl.CONFIGS[3]
    ly = cfg.layer
    st = wl.make_step_inputs(cfg, 0)
    w = wl.make_weights(cfg, 0)
    kv = wl.make_kv(cfg, 0, st["ctx_len"])
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
    w64 = olay.prepare_weights(w)
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
