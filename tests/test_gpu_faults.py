"""Faults in device-resident data on the layer call, and operands past 2 GiB.

The layer call's contract: a packed token outside [0, vocab) (with the
embedding gathered, x_in = NULL) sets DCUT_DERR_TOKEN, and a request whose
context does not leave room for its block (ctx_len < 0 or ctx_len + D + 1 >
cap) sets DCUT_DERR_CAPACITY; the affected request's outputs are unspecified,
every access stays in bounds (the norm kernel reads embedding row 0 for a bad
token, the attention clamps the usable context to cap - D - 1 and the cache
append skips slots outside [0, cap)), and the other requests' rows are exactly
what they would have been, so they still match the oracle.

The LM head at H = 8192, V = 152064 has 2.49 GB of weights: every column tile
addresses its own slice of W, so rows past 2 GiB are read like any other; its
logits and argmax match the oracle on every column.
"""
import dataclasses

import numpy as np
import pytest
import torch

from oracle import layer as olay
from oracle import lm_head as olm
from oracle import select as osel
from paper_2607_14647_amd import lib as L
from paper_2607_14647_amd import runner
from paper_2607_14647_amd import workload as wl
from tests.gpu_common import (ARGMAX_GAP, LOGIT_RTOL, X_RTOL, need_gpu, note, row_rel_err, tiny_variants,
                              workload)

pytestmark = pytest.mark.gpu
VARIANTS = tiny_variants()


def _run(cfg, st, w, kv, budgets, ctx_dev=None, tok_patch=None):
    """Select on the device, optionally overwrite packed tokens (device data), run the layer
    with the embedding gathered; returns (VerifyStep, host outputs)."""
    vs = runner.VerifyStep(cfg, w, st, kv)
    if ctx_dev is not None:
        vs.ctx_len.copy_(torch.from_numpy(ctx_dev))
    vs.select(budgets, [1.0] * len(budgets))
    torch.cuda.synchronize()
    if tok_patch is not None:
        for row, tok in tok_patch:
            vs.sel["packed_tok"][row] = int(tok)
    vs.dev_err.zero_()
    vs.verify()
    torch.cuda.synchronize()
    return vs


def _check_others(cfg, st, w, kv, vs, ctx_host, skip):
    K = int(vs.host("cu")[-1])
    sel = osel.select(st["conf"], st["draft"], ctx_host, list(cfg.budgets), [1.0] * len(cfg.budgets))
    assert np.array_equal(vs.host("cu"), sel["cu"])
    others = [i for i in range(cfg.B) if i not in skip]
    lay = olay.verify_layer(cfg.layer, olay.prepare_weights(w), kv, sel["cu"], sel["packed_tok"], sel["packed_pos"],
                            sel["packed_req"], ctx_host, cfg.D, requests=others)
    rows = np.concatenate([np.arange(sel["cu"][i], sel["cu"][i + 1]) for i in others])
    x = vs.x[:K].cpu().numpy()
    err = row_rel_err(x[rows], lay["x_out"][rows])
    note(f"  unaffected requests {others}: {len(rows)} rows, max rel err {err.max():.2e}")
    assert err.max() <= X_RTOL


@pytest.mark.parametrize("name", ["cfg1", "plan"])
def test_bad_token_sets_token_bit(name):
    need_gpu()
    cfg = VARIANTS[name]
    st, w, kv = workload(cfg, 0)
    sel = osel.select(st["conf"], st["draft"], st["ctx_len"], list(cfg.budgets), [1.0] * len(cfg.budgets))
    j = int(np.argmax(sel["keep_len"]))
    r0 = int(sel["cu"][j])
    patch = [(r0, cfg.layer.vocab + 5), (r0 + 1, -3)] if sel["keep_len"][j] > 1 else [(r0, cfg.layer.vocab)]
    note(f"{name}: request {j} rows {[p[0] for p in patch]} get tokens {[p[1] for p in patch]}")
    vs = _run(cfg, st, w, kv, list(cfg.budgets), tok_patch=patch)
    assert int(vs.dev_err.item()) & L.DERR_TOKEN
    _check_others(cfg, st, w, kv, vs, st["ctx_len"], {j})


@pytest.mark.parametrize("name", ["cfg1", "plan"])
def test_capacity_overflow_sets_capacity_bit(name):
    need_gpu()
    cfg = VARIANTS[name]
    st, w, kv = workload(cfg, 0)
    cap = kv["cap"].astype(np.int64)
    ctx = st["ctx_len"].copy()
    j1, j2 = 1, cfg.B - 1
    ctx[j1] = cap[j1] - cfg.D                # L + D + 1 = cap + 1: the last block slot falls outside
    ctx[j2] = -2                             # a negative context
    note(f"{name}: ctx_len[{j1}] = {ctx[j1]} (cap {cap[j1]}), ctx_len[{j2}] = {ctx[j2]}")
    vs = _run(cfg, st, w, kv, list(cfg.budgets), ctx_dev=ctx)
    assert int(vs.dev_err.item()) & L.DERR_CAPACITY
    assert not int(vs.dev_err.item()) & L.DERR_TOKEN
    _check_others(cfg, st, w, kv, vs, ctx, {j1, j2})


@pytest.mark.timeout(900)
def test_lm_head_weights_past_2gib():
    need_gpu()
    base = wl.CONFIGS[1]
    cfg = dataclasses.replace(base, cid=92, B=1, D=3, budgets=(4,),
                              layer=dataclasses.replace(base.layer, hidden=8192, vocab=152064))
    H, V = cfg.layer.hidden, cfg.layer.vocab
    note(f"LM head H={H} V={V}: {V * H * 2 / 2 ** 30:.2f} GiB of weights; generating")
    w = wl.make_weights(cfg, 0, with_embed=False)
    x = np.random.default_rng(11).standard_normal((4, H)).astype(np.float32)
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a.view(np.int16) if a.dtype == np.uint16 else a)).cuda()
    w_lm, fnorm, xd = dev(w["w_lm"]), dev(w["final_norm"]), dev(x)
    cu = torch.tensor([0, 4], dtype=torch.int32, device="cuda")
    amax = torch.zeros(4, dtype=torch.int32, device="cuda")
    logits = torch.zeros(4, V, dtype=torch.float32, device="cuda")
    lcfg = L.layer_cfg(cfg.layer, 64)
    ws = L.workspace(L.workspace_bytes(2, lcfg, cfg.B, cfg.D))
    L.lm_head_argmax(H, V, cfg.B, cfg.D, cu, xd, fnorm, cfg.layer.rms_eps, w_lm, amax, ws, logits=logits)
    torch.cuda.synchronize()
    lg = logits.cpu().numpy()
    am = amax.cpu().numpy()
    del w_lm, logits
    torch.cuda.empty_cache()
    note("  oracle (float64 weights)")
    ref = olm.lm_head_argmax(x.astype(np.float64), olay.bf16_bits_to_f64(w["final_norm"]), cfg.layer.rms_eps,
                             olay.bf16_bits_to_f64(w["w_lm"]))
    err = row_rel_err(lg, ref["logits"])
    # the weight rows that start past byte 2^31 of W: vocabulary columns from 131072 on
    tail = row_rel_err(lg[:, 131072:], ref["logits"][:, 131072:])
    sure = ref["gap"] > ARGMAX_GAP
    note(f"  max rel err {err.max():.2e} (columns past 2 GiB {tail.max():.2e}); argmax {am.tolist()} "
         f"vs {ref['argmax'].tolist()}")
    assert err.max() <= LOGIT_RTOL and tail.max() <= LOGIT_RTOL
    assert np.array_equal(am[sure], ref["argmax"][sure])
