"""Forced-match draft construction with the oracle (test infrastructure only).

The paper's drafter is unavailable, so synthetic drafts stand in for it:
draft z_{i,k} (k >= 1) is replaced by the target's greedy token at block
position k-1 when the stored uniform v_{i,k} < c_{i,k}, so depth k survives
with probability prod_{t<=k} c_{i,t} = s_{i,k}, the survival probability the
scores model (Sec. 3.2).  Because a row only sees its own block prefix, the
target token at position k-1 depends on z_{i,0..k-1} alone; the D passes run
in depth order and each one needs only block prefixes of length k.
"""
from __future__ import annotations

from typing import Optional, Sequence

import numpy as np

from .layer import verify_layer
from .lm_head import lm_head_argmax


def force_matches(ly, w64, kv, conf: np.ndarray, draft: np.ndarray, match_u: np.ndarray,
                  ctx_len: np.ndarray, D: int,
                  requests: Optional[Sequence[int]] = None) -> np.ndarray:
    B = draft.shape[0]
    z = np.array(draft, dtype=np.int32, copy=True)
    reqs = list(range(B)) if requests is None else list(requests)
    for k in range(1, D + 1):
        keep = np.full(B, k, dtype=np.int32)
        cu = np.zeros(B + 1, dtype=np.int32)
        cu[1:] = np.cumsum(keep)
        rows = int(cu[B])
        tok = np.zeros(rows, dtype=np.int32)
        pos = np.zeros(rows, dtype=np.int32)
        req = np.zeros(rows, dtype=np.int32)
        for i in range(B):
            for j in range(k):
                tok[cu[i] + j] = z[i, j]
                pos[cu[i] + j] = ctx_len[i] + j
                req[cu[i] + j] = i
        lay = verify_layer(ly, w64, kv, cu, tok, pos, req, ctx_len, D, requests=reqs)
        last = np.array([cu[i] + k - 1 for i in reqs])
        g = lm_head_argmax(lay["x_out"][last], w64["final_norm"], ly.rms_eps, w64["w_lm"])["argmax"]
        for n, i in enumerate(reqs):
            if match_u[i, k - 1] < conf[i, k - 1]:
                z[i, k] = g[n]
    return z
