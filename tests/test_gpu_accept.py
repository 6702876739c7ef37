"""dcut_accept on the GPU versus the oracle, bit-exact, on generator-made target tokens."""
import numpy as np
import pytest
import torch

from oracle import accept as oacc
from oracle import select as osel
from paper_2607_14647_amd import lib as L
from paper_2607_14647_amd import workload as wl
from tests.gpu_common import need_gpu, note, to_dev

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("cid,seed", [(c, s) for c in (1, 2, 3, 4, 5) for s in range(3)])
def test_accept_configs(cid, seed):
    need_gpu()
    cfg = wl.CONFIGS[cid]
    st = wl.make_step_inputs(cfg, seed)
    g_full = wl.synthetic_argmax(cfg, seed, st["draft"], st["match_u"], st["conf"])
    B, D = cfg.B, cfg.D
    for K in (cfg.budgets[0], cfg.budgets[len(cfg.budgets) // 2], B * (D + 1)):
        sel = osel.select(st["conf"], st["draft"], st["ctx_len"], [K], [1.0])
        kl, cu = sel["keep_len"], sel["cu"]
        argmax = np.zeros(B * (D + 1), np.int32)
        for i in range(B):
            argmax[cu[i]: cu[i + 1]] = g_full[i, : kl[i]]
        ref = oacc.accept(st["draft"], kl, cu, argmax)
        i32 = dict(dtype=torch.int32, device="cuda")
        acc, nxt, tot = torch.zeros(B, **i32), torch.zeros(B, **i32), torch.zeros(1, **i32)
        ctx = to_dev(st["ctx_len"])
        L.accept(B, D, to_dev(st["draft"]), to_dev(kl), to_dev(cu), to_dev(argmax), acc, nxt, tot, ctx)
        torch.cuda.synchronize()
        note(f"accept cfg{cid} seed{seed} K={K} total={int(ref['total'][0])}")
        assert np.array_equal(acc.cpu().numpy(), ref["accept_len"])
        assert np.array_equal(nxt.cpu().numpy(), ref["next_tok"])
        assert int(tot.item()) == int(ref["total"][0])
        assert np.array_equal(ctx.cpu().numpy(), st["ctx_len"] + ref["accept_len"] + 1)
