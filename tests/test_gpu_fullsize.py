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
