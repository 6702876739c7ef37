"""Oracle for the final norm, LM head and greedy argmax (test infrastructure only).

The target's greedy choice at every kept row (Sec. 3.1: the target model
scores the packed positions; Sec. 4.1: greedy target decoding):
  f = x / sqrt(mean(x^2) + eps) * g_final;  logits = f W_lm^T;
  argmax = the lowest vocabulary id among the maxima (np.argmax returns the
  first occurrence).  Also returns the gap between the two largest logits,
  which the parity tests use to decide where the argmax is well defined
  under bf16 rounding.  float64 throughout; `act_bf16=True` rounds the
  normalised rows f to bf16 first, as the path stores them (see the layer
  oracle's act_bf16).
"""
from __future__ import annotations

from typing import Dict

import numpy as np

from .layer import rmsnorm, round_bf16


def lm_head_argmax(x: np.ndarray, final_norm64: np.ndarray, eps: float,
                   w_lm64: np.ndarray, chunk: int = 16384, act_bf16: bool = False) -> Dict[str, np.ndarray]:
    x = np.asarray(x, dtype=np.float64)
    f = rmsnorm(x, final_norm64, eps)
    if act_bf16:
        f = round_bf16(f)
    V = w_lm64.shape[0]
    n = f.shape[0]
    logits = np.empty((n, V), dtype=np.float64)
    for c0 in range(0, V, chunk):
        logits[:, c0:c0 + chunk] = f @ w_lm64[c0:c0 + chunk].T
    am = np.argmax(logits, axis=1).astype(np.int32)
    top2 = np.sort(logits, axis=1)[:, -2:] if V >= 2 else np.zeros((n, 2))
    gap = top2[:, 1] - top2[:, 0]
    return dict(logits=logits, argmax=am, max_logit=logits[np.arange(n), am], gap=gap)
