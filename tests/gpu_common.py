"""Shared helpers of the GPU parity tests (inputs from the seeded generator, expected values from the oracle)."""
import dataclasses
import functools
import sys

import numpy as np
import torch

from oracle import accept as oacc
from oracle import layer as olay
from oracle import lm_head as olm
from oracle import select as osel
from paper_2607_14647_amd import workload as wl

LOGIT_RTOL = 2e-2      # max |l_gpu - l_ref| / max |l_ref| per row (bf16 path vs float64 oracle)
ARGMAX_GAP = 1e-2      # argmax must match wherever the oracle's top-2 gap exceeds this
ROUTER_GAP = 1e-2      # MoE rows compared where the oracle's k-th / (k+1)-th router-logit gap exceeds this
X_RTOL = 2e-2          # residual rows and appended keys/values, same row-relative measure


def need_gpu():
    assert torch.cuda.is_available(), "these tests need an MI355X GPU"


def note(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


def tiny_variants():
    c1 = wl.CONFIGS[1]
    return {
        "cfg1": c1,
        # several 512-key chunks per request plus a ragged last chunk
        "long": dataclasses.replace(c1, cid=81, B=12, ctx=("uniform", 500, 1600), budgets=(100,)),
        # many row tiles, contexts down to zero
        "wide": dataclasses.replace(c1, cid=82, B=40, ctx=("uniform", 0, 40), budgets=(300,)),
        # block of one position (bonus only)
        "d0": dataclasses.replace(c1, cid=83, D=0, budgets=(4,)),
        # a deep MLP: the down projection runs split-K
        "deep": dataclasses.replace(c1, cid=84, B=8, budgets=(50,),
                                    layer=dataclasses.replace(c1.layer, inter=2048)),
        # routed MoE MLPs: 6 experts top-2; 128 experts top-8 with 8 query heads per kv head
        "moe": dataclasses.replace(c1, cid=85, budgets=(30,),
                                   layer=dataclasses.replace(c1.layer, inter=0, n_exp=6, top_k=2,
                                                             exp_inter=40, rope_theta=1e6)),
        "moe128": dataclasses.replace(c1, cid=86, B=16, budgets=(120,), ctx=("uniform", 300, 700),
                                      layer=dataclasses.replace(c1.layer, n_q=8, n_kv=1, inter=0,
                                                                n_exp=128, top_k=8, exp_inter=64,
                                                                rope_theta=1e6)),
        # more than 512 attention work items (72 requests x 2 kv heads x 4 chunks of 512 keys),
        # so they run in the longest-first planned order; contexts down to zero
        "plan": dataclasses.replace(c1, cid=88, B=72, ctx=("uniform", 0, 2000), budgets=(200,)),
        # head_dim 128, split-K O and down projections, and a vocabulary wide enough for the
        # 256 x 256 LM-head tiles
        "split": dataclasses.replace(c1, cid=87, budgets=(40,),
                                     layer=dataclasses.replace(c1.layer, hidden=1024, n_q=16, n_kv=4,
                                                               head_dim=128, inter=2048, vocab=65536)),
        # split-K QKV (RoPE and the cache append in the reduce pass) as well: K = 2048
        "qkvsplit": dataclasses.replace(c1, cid=91, budgets=(40,),
                                        layer=dataclasses.replace(c1.layer, hidden=2048, n_q=16, n_kv=4,
                                                                  head_dim=128, inter=2048, vocab=1024)),
    }


def edge_variants():
    """The tiny layer at the size limits of the layer call."""
    c1 = wl.CONFIGS[1]
    return {
        # the largest batch and row count: B = 4096, B(D+1) = 8192; attention work items in
        # chunk-slowest order (batches above 1024 are not planned)
        "maxb": dataclasses.replace(c1, cid=89, B=4096, D=1, ctx=("uniform", 0, 64), budgets=(6000,)),
        # the largest planned batch: one request per thread of the planning workgroup, with full
        # and ragged chunks of 1024 keys
        "plan1024": dataclasses.replace(c1, cid=90, B=1024, D=3, ctx=("uniform", 0, 2500), budgets=(2500,)),
    }


@functools.lru_cache(maxsize=8)
def workload(cfg: wl.Config, seed: int, with_kv: bool = True):
    st = wl.make_step_inputs(cfg, seed)
    w = wl.make_weights(cfg, seed)
    kv = wl.make_kv(cfg, seed, st["ctx_len"]) if with_kv else None
    return st, w, kv


@functools.lru_cache(maxsize=1)
def full_workload(cid: int, seed: int):
    """A full-size configuration's inputs with the oracle's float64 weights (the last one
    asked for is kept: several tests share the batch-64 shape)."""
    cfg = wl.CONFIGS[cid]
    st = wl.make_step_inputs(cfg, seed)
    w = wl.make_weights(cfg, seed)
    kv = wl.make_kv(cfg, seed, st["ctx_len"])
    return cfg, st, w, kv, olay.prepare_weights(w)


def oracle_step(cfg: wl.Config, st, w64, kv, budgets, costs, draft=None, requests=None):
    """The oracle's whole greedy step: selection, layer and LM head over the kept rows of
    `requests` (default all), in float64 (for the residual and logit tolerances) and with
    the path's bf16 activations (for the argmax and acceptance decisions, which are integers
    decided by floating point and so are taken in the path's precision)."""
    draft = st["draft"] if draft is None else draft
    sel = osel.select(st["conf"], draft, st["ctx_len"], list(budgets), list(costs))
    args = (cfg.layer, w64, kv, sel["cu"], sel["packed_tok"], sel["packed_pos"], sel["packed_req"],
            st["ctx_len"], cfg.D)
    lay = olay.verify_layer(*args, requests=requests)
    lay16 = olay.verify_layer(*args, requests=requests, act_bf16=True)
    reqs = range(cfg.B) if requests is None else requests
    rows = np.concatenate([np.arange(sel["cu"][i], sel["cu"][i + 1]) for i in reqs]).astype(np.int64)
    lm = olm.lm_head_argmax(lay["x_out"][rows], w64["final_norm"], cfg.layer.rms_eps, w64["w_lm"])
    lm16 = olm.lm_head_argmax(lay16["x_out"][rows], w64["final_norm"], cfg.layer.rms_eps, w64["w_lm"],
                              act_bf16=True)
    return dict(sel=sel, lay=lay, lm=lm, lm16=lm16, rows=rows, draft=draft)


def check_step(ref, choice, keep_len, cu, x, argmax, accept_len=None, next_tok=None, logits=None,
               what=""):
    """GPU step outputs against oracle_step's: selection and packing bit for bit; residual rows
    (and logits when given) within their row-relative tolerance of the float64 oracle on every
    compared row; argmax where the bf16-activation oracle's top-2 gap exceeds ARGMAX_GAP;
    acceptance bit for bit for every request whose decisive rows all clear that gap (on that
    oracle's argmax).  x, argmax and logits hold the compared rows in the order of ref["rows"]."""
    sel, lay, lm, rows = ref["sel"], ref["lay"], ref["lm"], ref["rows"]
    lm16 = ref["lm16"]
    assert np.asarray(choice).tolist() == sel["choice"].tolist(), what
    assert np.array_equal(keep_len, sel["keep_len"]), what
    assert np.array_equal(cu, sel["cu"]), what
    ok = lay["router_gap"][rows] > ROUTER_GAP if "router_gap" in lay else np.ones(len(rows), bool)
    ex = row_rel_err(np.asarray(x)[ok], lay["x_out"][rows][ok])
    sure = (lm16["gap"] > ARGMAX_GAP) & ok
    msg = (f"{what}: {len(rows)} rows, {ok.sum()} compared, max rel err x={ex.max(initial=0):.2e}, "
           f"argmax rows {sure.sum()} (float64 oracle's argmax differs on {int((lm['argmax'] != argmax).sum())}, "
           f"at gaps {np.round(np.sort(lm['gap'][lm['argmax'] != argmax]), 4).tolist()})")
    if logits is not None:
        el = row_rel_err(np.asarray(logits)[ok], lm["logits"][ok])
        msg += f", logits {el.max(initial=0):.2e}"
        assert el.max(initial=0) <= LOGIT_RTOL, msg
    assert ex.max(initial=0) <= X_RTOL, msg
    assert sure.sum() >= len(rows) // 2, msg
    assert np.array_equal(np.asarray(argmax)[sure], lm16["argmax"][sure]), msg
    if accept_len is not None:
        # the oracle's argmax at every compared row; a request is decided when all rows
        # cu[i] .. cu[i] + min(a_i, n_i) clear the gap
        g = np.zeros(int(sel["cu"][-1]), dtype=np.int32)
        g[rows] = lm16["argmax"]
        sure_row = np.zeros(len(g), bool)
        sure_row[rows] = sure
        acc = oacc.accept(ref["draft"], sel["keep_len"], sel["cu"], g)
        B = len(sel["keep_len"])
        in_rows = np.zeros(len(g), bool)
        in_rows[rows] = True
        decided = np.array([in_rows[sel["cu"][i]] and
                            sure_row[sel["cu"][i]: sel["cu"][i] + acc["accept_len"][i] + 1].all() for i in range(B)])
        msg += f", acceptance decided for {decided.sum()}/{B} requests"
        assert np.array_equal(np.asarray(accept_len)[decided], acc["accept_len"][decided]), msg
        assert np.array_equal(np.asarray(next_tok)[decided], acc["next_tok"][decided]), msg
    note(msg)


def row_rel_err(got: np.ndarray, ref: np.ndarray) -> np.ndarray:
    got = got.reshape(got.shape[0], -1).astype(np.float64)
    ref = ref.reshape(ref.shape[0], -1).astype(np.float64)
    return np.abs(got - ref).max(axis=1) / np.maximum(np.abs(ref).max(axis=1), 1e-30)


def to_dev(a: np.ndarray) -> torch.Tensor:
    if a.dtype == np.uint16:
        a = a.view(np.int16)
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()
