"""The allocation-free LM head (dcut_lm_head_argmax_static) against the workspace one.

Two calls in a row through the C ABI on the static scratch array, the second
with a smaller input, each compared bit for bit (argmax, max logit, logits)
with dcut_lm_head_argmax on a caller workspace: the same kernels run on the
same inputs, so the outputs are identical.  The first call is the batch-64
LM head at its largest row count (B(D+1) = 1024, V = 128256, H = 4096).
"""
import dataclasses

import numpy as np
import pytest
import torch

from paper_2607_14647_amd import lib as L
from paper_2607_14647_amd import workload as wl
from tests.gpu_common import need_gpu, note

pytestmark = pytest.mark.gpu


def _inputs(B, D, H, rng):
    keep = rng.integers(1, D + 2, size=B)
    cu = np.zeros(B + 1, dtype=np.int32)
    cu[1:] = np.cumsum(keep)
    x = rng.standard_normal((B * (D + 1), H)).astype(np.float32)
    return cu, x


def test_static_lm_head_matches_workspace_call():
    need_gpu()
    base = wl.CONFIGS[3]
    cfg = dataclasses.replace(wl.CONFIGS[1], cid=93, layer=dataclasses.replace(wl.CONFIGS[1].layer, hidden=4096,
                                                                               vocab=base.layer.vocab))
    H, V, eps = cfg.layer.hidden, cfg.layer.vocab, cfg.layer.rms_eps
    w = wl.make_weights(cfg, 0, with_embed=False)
    w_lm = torch.from_numpy(w["w_lm"].view(np.int16)).cuda()
    fnorm = torch.from_numpy(w["final_norm"].view(np.int16)).cuda()
    rng = np.random.default_rng(2024)
    assert L.lm_head_static_scratch_bytes() == 32 << 20
    for call, (B, D) in enumerate([(64, 15), (16, 15)]):
        cu_h, x_h = _inputs(B, D, H, rng)
        M, K = B * (D + 1), int(cu_h[-1])
        note(f"call {call}: B={B} D={D} rows={M} K*={K} V={V}")
        cu, x = torch.from_numpy(cu_h).cuda(), torch.from_numpy(x_h).cuda()
        out = {}
        for which in ("static", "workspace"):
            am = torch.full((M,), -7, dtype=torch.int32, device="cuda")
            ml = torch.full((M,), -7.0, dtype=torch.float32, device="cuda")
            lg = torch.full((M, V), -7.0, dtype=torch.float32, device="cuda")
            if which == "static":
                L.lm_head_argmax_static(H, V, B, D, cu, x, fnorm, eps, w_lm, am, max_logit=ml, logits=lg)
            else:
                lcfg = L.layer_cfg(cfg.layer, 64)
                ws = L.workspace(L.workspace_bytes(2, lcfg, B, D))
                L.lm_head_argmax(H, V, B, D, cu, x, fnorm, eps, w_lm, am, ws, max_logit=ml, logits=lg)
            torch.cuda.synchronize()
            out[which] = (am[:K].cpu().numpy(), ml[:K].cpu().numpy(), lg[:K].cpu().numpy())
            del lg
        for a, b in zip(out["static"], out["workspace"]):
            assert np.array_equal(a, b)
        # the argmax is the logits' first maximum and max_logit its value
        am_s, ml_s, lg_s = out["static"]
        assert np.array_equal(am_s, np.argmax(lg_s, axis=1))
        assert np.array_equal(ml_s, lg_s.max(axis=1))
        note(f"  identical on {K} rows")
