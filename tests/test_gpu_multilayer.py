"""A stack of decoder layers (the target's depth) on the GPU versus the oracle.

Each layer has its own seeded weights and KV cache; the residual stream runs
through every layer in place (x_in = x_out) and the LM head reads the last.
Residual rows, every layer's appended keys and values, and logits are
compared with the float64 oracle under the single-layer tolerances; MoE rows
whose routing is a near-tie in any layer are left out.
"""
import numpy as np
import pytest
import torch

from oracle import layer as olay
from oracle import lm_head as olm
from oracle import select as osel
from paper_2607_14647_amd import runner
from paper_2607_14647_amd import workload as wl
from tests.gpu_common import (ARGMAX_GAP, LOGIT_RTOL, ROUTER_GAP, X_RTOL, need_gpu, note, row_rel_err,
                              tiny_variants, workload)

pytestmark = pytest.mark.gpu
VARIANTS = tiny_variants()


def _kv_err(kg, vg, kv, lay, sel, ly, rows):
    hd, nkv = ly.head_dim, ly.n_kv
    err = [0.0]
    for t in rows:
        i, slot = int(sel["packed_req"][t]), int(sel["packed_pos"][t])
        cap, base = int(kv["cap"][i]), int(kv["base"][i])
        for g in range(nkv):
            off = base + (g * cap + slot) * hd
            for got, ref in ((kg, lay["new_k"]), (vg, lay["new_v"])):
                a = olay.bf16_bits_to_f64(got[off: off + hd])
                err.append(np.abs(a - ref[t, g]).max() / np.abs(ref[t, g]).max())
    return max(err)


@pytest.mark.parametrize("name,n_layers", [("cfg1", 4), ("split", 3), ("qkvsplit", 2), ("moe", 3), ("long", 2)])
def test_layer_stack(name, n_layers):
    need_gpu()
    cfg = VARIANTS[name]
    st, w, kv = workload(cfg, 0)
    extra = [(wl.make_weights(cfg, 0, layer=l), wl.make_kv(cfg, 0, st["ctx_len"], layer=l))
             for l in range(1, n_layers)]
    K = cfg.budgets[0]
    note(f"layer stack {name}: {n_layers} layers, K={K}")
    vs = runner.VerifyStep(cfg, w, st, kv)
    for wx, kx in extra:
        vs.add_layer(wx, kx)
    logits = torch.zeros(cfg.B * (cfg.D + 1), cfg.layer.vocab, dtype=torch.float32, device="cuda")
    vs.select([K], [1.0])
    vs.verify()
    vs.lm_head(logits=logits)
    torch.cuda.synchronize()
    assert int(vs.dev_err.item()) == 0

    sel = osel.select(st["conf"], st["draft"], st["ctx_len"], [K], [1.0])
    layers = [(w, kv)] + extra
    x, ok, kv_errs = None, np.ones(K, bool), []
    caches = [(vs.kv["k"], vs.kv["v"])] + [(kt["k"], kt["v"]) for _, _, kt, _ in vs.extra]
    for (wx, kx), (gk, gv) in zip(layers, caches):
        lay = olay.verify_layer(cfg.layer, olay.prepare_weights(wx), kx, sel["cu"], sel["packed_tok"],
                                sel["packed_pos"], sel["packed_req"], st["ctx_len"], cfg.D, x_in=x)
        x = lay["x_out"]
        # this layer's keys and values depend on the routing of the layers before it only
        kv_errs.append(_kv_err(gk.cpu().numpy().view(np.uint16), gv.cpu().numpy().view(np.uint16),
                               kx, lay, sel, cfg.layer, np.flatnonzero(ok)))
        if "router_gap" in lay:
            ok &= lay["router_gap"] > ROUTER_GAP
            # later rows of a request attend to the earlier ones in the next layers
            for i in range(cfg.B):
                seg = np.flatnonzero(~ok[sel["cu"][i]: sel["cu"][i + 1]])
                if seg.size:
                    ok[sel["cu"][i] + seg[0]: sel["cu"][i + 1]] = False
    w64 = olay.prepare_weights(w)
    lm = olm.lm_head_argmax(x, w64["final_norm"], cfg.layer.rms_eps, w64["w_lm"])
    ex = row_rel_err(vs.x.cpu().numpy()[:K][ok], x[ok])
    el = row_rel_err(logits.cpu().numpy()[:K][ok], lm["logits"][ok])
    sure = (lm["gap"] > ARGMAX_GAP) & ok
    note(f"  rows {ok.sum()}/{K}: x err {ex.max():.2e}, kv err per layer "
         f"{', '.join(f'{e:.1e}' for e in kv_errs)}, logits err {el.max():.2e}, argmax rows {sure.sum()}")
    assert ok.sum() >= K // 2
    assert ex.max() <= X_RTOL and max(kv_errs) <= X_RTOL and el.max() <= LOGIT_RTOL
    assert np.array_equal(vs.host("argmax")[:K][sure], lm["argmax"][sure])
