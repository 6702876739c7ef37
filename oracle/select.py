"""Oracle for cross-request draft selection and packing (test infrastructure only).

Follows Sec. 3.2 (Eq. dcut-prefix-score: s_{i,0} = 1, s_{i,k} = prod_{t<=k} c_{i,t};
the estimated advance of keep depth n is the sum of s_{i,0..n}), Sec. 3.3
(Eq. dcut-budget for the ratio buckets, Eq. dcut-objective for the budget
choice) and Alg. 1 (flatten, rank with ties toward smaller depth, sum the
top-K scores per candidate budget, pick the best ratio, keep the per-request
prefixes, pack them).  App. A proves that the kept set of each request is a
contiguous prefix; `select` asserts it.

Readings fixed here where the paper leaves the arithmetic open:
  * s is the sequential float32 product (one rounding per factor, in depth
    order).  The paper's complexity paragraph mentions log-confidences; the
    product is the equation's definition, and float32 is the precision in
    which the GPU takes the same integer decisions.
  * ranking order: score descending, then depth ascending (Alg. 1), then
    request index ascending (the tie rule stated in App. B, used for all
    variants here).
  * benefit sums are exact: each score becomes u = trunc(s * 2^40) as an
    unsigned 64-bit integer and the top-K sums are integer sums.
  * objective: float64(P[K]) * 2^-40 / C_r with one IEEE division; the first
    candidate with the strictly largest objective wins, so among equal
    objectives the smaller budget is chosen (candidates are given with
    non-decreasing budgets).
  * exactly K positions are kept, including positions whose score is 0.
"""
from __future__ import annotations

import math
from typing import Dict, Sequence

import numpy as np

from .errors import DcutArgError, DcutDataError, DERR_CONF

MAX_BLOCK = 64          # D + 1 limit
MAX_BATCH = 4096
MAX_ROWS = 8192         # B (D + 1) limit
MAX_CANDIDATES = 64
FIX_SHIFT = 40          # benefit fixed point: units of 2^-40


def budget_from_ratio(B: int, D: int, num: int, den: int) -> int:
    """Eq. dcut-budget: K_rho(B) = max(B, ceil(rho * B * (D + 1))), rho = num/den exactly."""
    if den <= 0 or num < 0 or num > den:
        raise DcutArgError("ratio must be num/den with 0 <= num <= den, den > 0")
    total = B * (D + 1)
    k = -((-num * total) // den)          # exact integer ceiling
    return max(B, k)


def check_args(B: int, D: int, budgets: Sequence[int], costs: Sequence[float]) -> None:
    if B < 1 or B > MAX_BATCH:
        raise DcutArgError(f"batch {B} outside [1, {MAX_BATCH}]")
    if D < 0 or D + 1 > MAX_BLOCK:
        raise DcutArgError(f"block D+1={D + 1} outside [1, {MAX_BLOCK}]")
    if B * (D + 1) > MAX_ROWS:
        raise DcutArgError(f"B(D+1)={B * (D + 1)} above {MAX_ROWS}")
    R = len(budgets)
    if R < 1 or R > MAX_CANDIDATES or len(costs) != R:
        raise DcutArgError("need 1..64 candidates with one cost each")
    prev = -1
    for K in budgets:
        if K < B or K > B * (D + 1):
            raise DcutArgError(f"budget {K} outside [B, B(D+1)]")
        if K < prev:
            raise DcutArgError("budgets must be non-decreasing")
        prev = K
    for c in costs:
        if not math.isfinite(c) or c <= 0.0:
            raise DcutArgError("costs must be finite and positive")


def prefix_scores(conf: np.ndarray) -> np.ndarray:
    """Eq. dcut-prefix-score, one float32 multiply per depth, in depth order."""
    conf = np.asarray(conf, dtype=np.float32)
    bad = np.isnan(conf) | np.signbit(conf) | (conf > np.float32(1.0))
    if bad.any():
        raise DcutDataError(DERR_CONF, "confidence NaN, negative or above 1")
    B, D = conf.shape
    s = np.empty((B, D + 1), dtype=np.float32)
    s[:, 0] = np.float32(1.0)
    for k in range(1, D + 1):
        s[:, k] = s[:, k - 1] * conf[:, k - 1]
    return s


def fixed_point(s: np.ndarray) -> np.ndarray:
    """u = trunc(s * 2^40), exact for float32 s in [0, 1]."""
    return np.trunc(s.astype(np.float64) * float(2 ** FIX_SHIFT)).astype(np.uint64)


def rank_order(s: np.ndarray) -> np.ndarray:
    """Flattened positions (i, k) in rank order: s desc, k asc, i asc (Alg. 1)."""
    B, D1 = s.shape
    ii, kk = np.meshgrid(np.arange(B), np.arange(D1), indexing="ij")
    order = np.lexsort((ii.ravel(), kk.ravel(), -s.astype(np.float64).ravel()))
    return order          # flat indices i*(D+1)+k


def select(conf: np.ndarray, draft: np.ndarray, ctx_len: np.ndarray,
           budgets: Sequence[int], costs: Sequence[float]) -> Dict[str, np.ndarray]:
    """Full selection + packing.  Returns the same outputs as the library call.

    keep_len[i] = n_i + 1; cu = exclusive prefix sum of keep_len (cu[B] = K*);
    packed rows t = cu[i] + k carry token z_{i,k}, position L_i + k, request i;
    choice = (K*, r*); benefit[r] = sum of u over the top-K_r positions."""
    conf = np.asarray(conf, dtype=np.float32)
    B, D = conf.shape
    check_args(B, D, budgets, costs)
    s = prefix_scores(conf)
    u = fixed_point(s).ravel()
    order = rank_order(s)
    P = np.zeros(B * (D + 1) + 1, dtype=np.uint64)
    P[1:] = np.cumsum(u[order], dtype=np.uint64)
    benefit = np.array([P[K] for K in budgets], dtype=np.uint64)
    best_r, best_obj = 0, -1.0
    for r, (K, C) in enumerate(zip(budgets, costs)):
        obj = (float(P[K]) * 2.0 ** -FIX_SHIFT) / float(C)
        if obj > best_obj:
            best_r, best_obj = r, obj
    Kstar = int(budgets[best_r])
    kept = np.zeros(B * (D + 1), dtype=bool)
    kept[order[:Kstar]] = True
    kept = kept.reshape(B, D + 1)
    keep_len = kept.sum(axis=1).astype(np.int32)
    for i in range(B):            # App. A: kept positions are exactly {0..n_i}
        assert kept[i, : keep_len[i]].all() and not kept[i, keep_len[i]:].any()
    cu = np.zeros(B + 1, dtype=np.int32)
    cu[1:] = np.cumsum(keep_len)
    rows = B * (D + 1)
    ptok = np.zeros(rows, dtype=np.int32)
    ppos = np.zeros(rows, dtype=np.int32)
    preq = np.zeros(rows, dtype=np.int32)
    for i in range(B):
        for k in range(keep_len[i]):
            t = cu[i] + k
            ptok[t] = draft[i, k]
            ppos[t] = ctx_len[i] + k
            preq[t] = i
    return dict(scores=s, keep_len=keep_len, cu=cu, packed_tok=ptok, packed_pos=ppos,
                packed_req=preq, choice=np.array([Kstar, best_r], dtype=np.int32),
                benefit=benefit, objective=best_obj)
