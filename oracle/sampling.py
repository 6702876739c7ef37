"""Oracle for temperature-T target sampling at every kept row (test infrastructure only).

Temperature-1 target sampling with target-only verification is the paper's
second regime (Sec. 4, robustness across sampling regimes; App. A, the
correctness paragraph): the target draws its token at each kept row from
softmax(logits / T) and a draft is accepted while it equals the target's
token at the previous row, exactly as in greedy verification.

Draws use the Gumbel-max identity: with G_c = -ln(-ln u_c) and u_c
independent uniforms on (0, 1), argmax_c (logits_c / T + G_c) is distributed
as softmax(logits / T)_c (Gumbel, 1954).  The uniforms come from
Philox4x32-10 (Salmon, Moraes, Dror and Shaw, "Parallel random numbers: as
easy as 1, 2, 3", SC 2011), keyed by the 64-bit seed (low word first):

  counter(c) = (32 * (c >> 7) + (c & 31), pos, req, 0),  word(c) = (c >> 5) & 3
  u_c = (philox(counter(c), key)[word(c)] + 0.5) / 2^32

so a (request, absolute position) pair always sees the same noise, whatever
else the batch keeps.  Logits, noise and scores are float64 here.
"""
from __future__ import annotations

from typing import Dict

import numpy as np

from .lm_head import lm_head_argmax

_M0 = np.uint64(0xD2511F53)
_M1 = np.uint64(0xCD9E8D57)
_W0 = 0x9E3779B9
_W1 = 0xBB67AE85
_MASK = np.uint64(0xFFFFFFFF)


def _round(c0, c1, c2, c3, k0, k1):
    p0 = c0.astype(np.uint64) * _M0
    p1 = c2.astype(np.uint64) * _M1
    hi0, lo0 = (p0 >> np.uint64(32)).astype(np.uint32), (p0 & _MASK).astype(np.uint32)
    hi1, lo1 = (p1 >> np.uint64(32)).astype(np.uint32), (p1 & _MASK).astype(np.uint32)
    return hi1 ^ c1 ^ k0, lo1, hi0 ^ c3 ^ k1, lo0


def philox4x32_10(ctr, key):
    """Philox4x32 with 10 rounds: ctr is four uint32 arrays (broadcastable),
    key two uint32 scalars; returns the four output words as uint32 arrays.
    The key is bumped by the Weyl constants before every round after the first."""
    c0, c1, c2, c3 = (np.asarray(c, dtype=np.uint32) for c in ctr)
    c0, c1, c2, c3 = np.broadcast_arrays(c0, c1, c2, c3)
    k0, k1 = int(key[0]) & 0xFFFFFFFF, int(key[1]) & 0xFFFFFFFF
    for r in range(10):
        if r > 0:
            k0 = (k0 + _W0) & 0xFFFFFFFF
            k1 = (k1 + _W1) & 0xFFFFFFFF
        c0, c1, c2, c3 = _round(c0, c1, c2, c3, np.uint32(k0), np.uint32(k1))
    return c0, c1, c2, c3


def uniforms(req: np.ndarray, pos: np.ndarray, V: int, seed: int) -> np.ndarray:
    """u[row, c] in (0, 1) for rows (req, pos) and columns c < V."""
    req = np.asarray(req, dtype=np.int64)
    pos = np.asarray(pos, dtype=np.int64)
    c = np.arange(V, dtype=np.int64)
    c0 = (32 * (c >> 7) + (c & 31)).astype(np.uint32)[None, :]
    word = ((c >> 5) & 3)[None, :]
    key = (seed & 0xFFFFFFFF, (seed >> 32) & 0xFFFFFFFF)
    out = philox4x32_10((c0, pos.astype(np.uint32)[:, None], req.astype(np.uint32)[:, None], np.uint32(0)), key)
    w = np.choose(np.broadcast_to(word, (len(req), V)), out)
    return (w.astype(np.float64) + 0.5) / 4294967296.0


def gumbel(req, pos, V: int, seed: int) -> np.ndarray:
    """Standard Gumbel noise G = -ln(-ln u)."""
    return -np.log(-np.log(uniforms(req, pos, V, seed)))


def sample_tokens(logits: np.ndarray, req, pos, temperature: float, seed: int) -> Dict[str, np.ndarray]:
    """Sampled token per row of `logits`: argmax of logits / T + G (lowest id on
    ties), the winning score and the gap to the runner-up (used to gate
    comparisons)."""
    if not temperature > 0.0:
        raise ValueError("temperature must be positive")
    logits = np.asarray(logits, dtype=np.float64)
    y = logits / float(temperature) + gumbel(req, pos, logits.shape[1], seed)
    tok = np.argmax(y, axis=1).astype(np.int32)
    n = y.shape[0]
    top2 = np.sort(y, axis=1)[:, -2:] if y.shape[1] >= 2 else np.zeros((n, 2))
    return dict(score=y, token=tok, max_score=y[np.arange(n), tok], gap=top2[:, 1] - top2[:, 0])


def lm_head_sample(x: np.ndarray, final_norm64: np.ndarray, eps: float, w_lm64: np.ndarray,
                   req: np.ndarray, pos: np.ndarray, temperature: float, seed: int) -> Dict[str, np.ndarray]:
    """Final norm, logits, then the sampled token of every row."""
    lm = lm_head_argmax(x, final_norm64, eps, w_lm64)
    out = sample_tokens(lm["logits"], req, pos, temperature, seed)
    out["logits"] = lm["logits"]
    return out
