"""Oracle for the rejection-sampling (RS) extension (test infrastructure only).

App. B (causality under rejection sampling) extends D-cut to drafters that
expose their per-position proposal distributions q_{i,k} and to targets that
verify with standard rejection sampling.  Three pieces are defined there:

  * shifted scores, Eq. dcut-shifted-score:  s~_{i,0} = 1 and
    s~_{i,k} = prod_{t=1}^{k-1} q_{i,t}(z_{i,t}) for k = 1..D, so the score
    that admits depth k depends only on the proposals before k;
  * causal budget selection, either the early-stopping scan (one frontier
    per request; the frontier with the largest shifted score is admitted
    for good while the utility-cost objective improves, and the scan stops
    at the first position that does not improve it), or a budget K fixed
    beforehand from earlier steps followed by the global top-K of the
    shifted scores; ties go to the shallower depth, then the smaller request;
  * RS acceptance: draft z_{i,j} is accepted with probability
    min(1, p(z)/q(z)) against the target distribution p of the previous
    block position; at the first rejection the committed token is drawn from
    the residual distribution proportional to (p - q)_+; when every kept
    draft is accepted the bonus token is drawn from p at the last kept row.

Readings fixed here where the paper leaves the arithmetic open:
  * shifted scores are sequential float32 products in depth order (the same
    arithmetic as the unshifted scores of Eq. dcut-prefix-score), so
    s~_{i,1} = 1 and s~_{i,k} equals the unshifted s_{i,k-1};
  * the scan starts from the B bonus positions (the clamp K >= B of
    Eq. dcut-budget) and evaluates the objective of Eq. dcut-objective,
    float64(P(K)) * 2^-40 / C(K), with P the exact fixed-point sum of
    trunc(s~ * 2^40) over the admitted positions; "improves" means strictly
    larger;
  * the objective at an arbitrary K needs a cost there, while the cost table
    holds the ratio buckets: C(K) interpolates it linearly between
    consecutive budgets (K_r, C_r) and is constant outside [K_0, K_{R-1}];
    where several budgets coincide, the last one's cost holds at that K;
  * the fixed-budget variant takes exactly one budget;
  * history-based K: the budget of this step is the one the cost model picks
    (Eq. dcut-objective over the candidate budgets, first strict maximum)
    on the previous step's shifted scores, carried in one integer of state
    (clamped to [B, B(D+1)]); it is fixed before the current block is seen;
  * the target distribution of a kept row is softmax(logits / T);
    acceptance compares u * q(z) < p(z) in float64, with u one Philox4x32-10
    uniform per row (counter (0, pos, req, 1), word 0, u = (w + 0.5) / 2^32);
  * both samples use the row's Gumbel noise of the target sampler (counter
    (32 (c >> 7) + (c & 31), pos, req, 0), word (c >> 5) & 3): the bonus is
    argmax_c logits_c / T + G_c and the residual draw is
    argmax_c ln((p_c - q_c)_+) + G_c.  A row is consulted for at most one of
    the two, so their sharing the noise leaves them independent.  If no
    column has p_c > q_c the residual draw falls back to the bonus rule.
"""
from __future__ import annotations

import math
from typing import Dict, Sequence

import numpy as np

from .errors import DcutArgError, DcutDataError, DERR_CONF
from .sampling import gumbel, philox4x32_10
from .select import FIX_SHIFT, check_args, fixed_point

SCAN = 0        # causal early-stopping scan over the interpolated cost curve
FIXED = 1       # budget fixed beforehand, global top-K
HISTORY = 2     # budget carried over from the previous block, global top-K


def shifted_scores(conf: np.ndarray) -> np.ndarray:
    """Eq. dcut-shifted-score: s~_{i,0} = s~_{i,1} = 1, s~_{i,k} = s~_{i,k-1} * c_{i,k-1}
    (one float32 multiply per depth, in depth order)."""
    conf = np.asarray(conf, dtype=np.float32)
    bad = np.isnan(conf) | np.signbit(conf) | (conf > np.float32(1.0))
    if bad.any():
        raise DcutDataError(DERR_CONF, "confidence NaN, negative or above 1")
    B, D = conf.shape
    s = np.empty((B, D + 1), dtype=np.float32)
    s[:, 0] = np.float32(1.0)
    if D >= 1:
        s[:, 1] = np.float32(1.0)
    for k in range(2, D + 1):
        s[:, k] = s[:, k - 1] * conf[:, k - 2]
    return s


def cost_curve(B: int, D: int, budgets: Sequence[int], costs: Sequence[float]) -> np.ndarray:
    """C(K) for K = 0..B(D+1): linear between consecutive budgets, constant outside.

    Between K_r <= K < K_{r+1} (r the last budget not above K):
        C(K) = C_r + ((C_{r+1} - C_r) * (K - K_r)) / (K_{r+1} - K_r)
    in that order of float64 operations."""
    N = B * (D + 1)
    R = len(budgets)
    C = np.empty(N + 1, dtype=np.float64)
    for K in range(N + 1):
        r = -1
        for t in range(R):
            if budgets[t] <= K:
                r = t
        if r < 0:
            C[K] = float(costs[0])
        elif r == R - 1:
            C[K] = float(costs[R - 1])
        else:
            ka, kb = int(budgets[r]), int(budgets[r + 1])
            ca, cb = float(costs[r]), float(costs[r + 1])
            C[K] = ca + ((cb - ca) * float(K - ka)) / float(kb - ka)
    return C


def _objective(P: int, C: float) -> float:
    return (float(P) * 2.0 ** -FIX_SHIFT) / C


def causal_scan(s: np.ndarray, curve: np.ndarray) -> Dict[str, object]:
    """The early-stopping scan of App. B over shifted scores `s` [B][D+1].

    Every request's bonus position is admitted first (K = B).  Then, while
    some request still has a frontier depth <= D, the frontier with the
    largest score (ties: smaller depth, then smaller request) is tried: it is
    admitted if the objective at K + 1 is strictly larger than at K, and the
    scan stops otherwise."""
    B, D1 = s.shape
    u = fixed_point(s)
    admitted = np.zeros((B, D1), dtype=bool)
    admitted[:, 0] = True
    frontier = np.ones(B, dtype=np.int64)
    K = B
    P = int(u[:, 0].astype(object).sum())
    J = _objective(P, curve[K])
    order = [(i, 0) for i in range(B)]
    req = np.arange(B)
    while True:
        live = frontier < D1
        if not live.any():
            break
        # the frontier with the largest score; ties to the smaller depth, then request
        f = np.minimum(frontier, D1 - 1)
        sc = np.where(live, s[req, f].astype(np.float64), -1.0)
        top = sc == sc.max()
        dep = np.where(top, f, D1)
        i = int(np.flatnonzero(top & (dep == dep.min()))[0])
        k = int(frontier[i])
        P2 = P + int(u[i, k])
        J2 = _objective(P2, curve[K + 1])
        if not J2 > J:
            break
        admitted[i, k] = True
        frontier[i] += 1
        K, P, J = K + 1, P2, J2
        order.append((i, k))
    return dict(K=K, admitted=admitted, benefit=P, objective=J, order=order)


def _pack(draft, ctx_len, keep_len):
    B = len(keep_len)
    rows = draft.shape[0] * draft.shape[1]
    cu = np.zeros(B + 1, dtype=np.int32)
    cu[1:] = np.cumsum(keep_len)
    ptok = np.zeros(rows, dtype=np.int32)
    ppos = np.zeros(rows, dtype=np.int32)
    preq = np.zeros(rows, dtype=np.int32)
    for i in range(B):
        for k in range(int(keep_len[i])):
            t = cu[i] + k
            ptok[t] = draft[i, k]
            ppos[t] = ctx_len[i] + k
            preq[t] = i
    return cu, ptok, ppos, preq


def select_rs(conf: np.ndarray, draft: np.ndarray, ctx_len: np.ndarray, mode: int,
              budgets: Sequence[int], costs: Sequence[float], k_state: int = 0) -> Dict[str, np.ndarray]:
    """RS-safe selection and packing; the same outputs as the unshifted selection.

    choice = (K*, r) with r the last budget index whose K_r <= K* (-1 if none);
    benefit[r] = exact fixed-point sum of the shifted scores over the top-K_r
    positions of the global ranking.  With HISTORY, K* = k_state clamped to
    [B, B(D+1)], and k_next is the budget for the next step."""
    conf = np.asarray(conf, dtype=np.float32)
    draft = np.asarray(draft)
    B, D = conf.shape
    check_args(B, D, budgets, costs)
    if mode not in (SCAN, FIXED, HISTORY):
        raise DcutArgError("mode must be SCAN, FIXED or HISTORY")
    if mode == FIXED and len(budgets) != 1:
        raise DcutArgError("a fixed budget takes exactly one candidate")
    s = shifted_scores(conf)
    u = fixed_point(s).ravel()
    ii, kk = np.meshgrid(np.arange(B), np.arange(D + 1), indexing="ij")
    order = np.lexsort((ii.ravel(), kk.ravel(), -s.astype(np.float64).ravel()))
    P = np.zeros(B * (D + 1) + 1, dtype=np.uint64)
    P[1:] = np.cumsum(u[order], dtype=np.uint64)
    benefit = np.array([P[K] for K in budgets], dtype=np.uint64)
    k_next = None
    if mode == HISTORY:
        # this block's retrospective choice, the budget of the next step
        best_r, best_obj = 0, -1.0
        for r, (K, C) in enumerate(zip(budgets, costs)):
            obj = _objective(int(P[K]), float(C))
            if obj > best_obj:
                best_r, best_obj = r, obj
        k_next = int(budgets[best_r])
    if mode == SCAN:
        sc = causal_scan(s, cost_curve(B, D, budgets, costs))
        Kstar, kept = int(sc["K"]), sc["admitted"]
        objective = sc["objective"]
    else:
        Kstar = int(budgets[0]) if mode == FIXED else min(max(int(k_state), B), B * (D + 1))
        kept = np.zeros(B * (D + 1), dtype=bool)
        kept[order[:Kstar]] = True
        kept = kept.reshape(B, D + 1)
        objective = _objective(int(P[Kstar]), float(costs[0])) if mode == FIXED else None
    keep_len = kept.sum(axis=1).astype(np.int32)
    for i in range(B):            # kept positions form a prefix (s~ is non-increasing in depth)
        assert kept[i, : keep_len[i]].all() and not kept[i, keep_len[i]:].any()
    r_of = -1
    for r, K in enumerate(budgets):
        if K <= Kstar:
            r_of = r
    cu, ptok, ppos, preq = _pack(draft, ctx_len, keep_len)
    return dict(scores=s, keep_len=keep_len, cu=cu, packed_tok=ptok, packed_pos=ppos,
                packed_req=preq, choice=np.array([Kstar, r_of], dtype=np.int32),
                benefit=benefit, objective=objective, kept=kept, k_next=k_next)


def accept_uniform(req, pos, seed: int) -> np.ndarray:
    """The acceptance uniform of each (request, position) row."""
    req = np.asarray(req, dtype=np.int64).astype(np.uint32)
    pos = np.asarray(pos, dtype=np.int64).astype(np.uint32)
    key = (seed & 0xFFFFFFFF, (seed >> 32) & 0xFFFFFFFF)
    w = philox4x32_10((np.uint32(0), pos, req, np.uint32(1)), key)[0]
    return (w.astype(np.float64) + 0.5) / 4294967296.0


def target_probs(logits_row: np.ndarray, temperature: float) -> np.ndarray:
    """softmax(logits / T) in float64."""
    y = np.asarray(logits_row, dtype=np.float64) / float(temperature)
    e = np.exp(y - y.max())
    return e / e.sum()


def rs_accept(draft: np.ndarray, keep_len: np.ndarray, cu: np.ndarray, ctx_len: np.ndarray,
              q: np.ndarray, logits: np.ndarray, temperature: float, seed: int) -> Dict[str, np.ndarray]:
    """RS verification of every request's kept block.

    draft [B][D+1] (column 0 the bonus token), q [B][D][V] with q[i, j-1] the
    proposal distribution of z_{i,j}, logits [rows][V] of the packed rows.
    Row cu_i + j - 1 (position L_i + j - 1) verifies z_{i,j}.

    Returns accept_len a_i, next_tok (the token committed after the accepted
    drafts), total = sum(a_i + 1), rej_row (the rejecting row or -1), and for
    gating: margin = |ln(u q(z)) - ln p(z)| of the deciding row of each
    request (the smallest over its consulted rows) and gap = the top-2 gap of
    the final draw."""
    if not temperature > 0.0 or not math.isfinite(temperature):
        raise ValueError("temperature must be positive and finite")
    draft = np.asarray(draft)
    B = draft.shape[0]
    V = logits.shape[1]
    acc = np.zeros(B, dtype=np.int32)
    nxt = np.zeros(B, dtype=np.int32)
    rej = np.full(B, -1, dtype=np.int32)
    margin = np.full(B, np.inf)
    gap = np.zeros(B)
    # the acceptance uniform of every position a request could consult
    D1 = draft.shape[1]
    U = accept_uniform(np.repeat(np.arange(B), D1),
                       (np.asarray(ctx_len, dtype=np.int64)[:, None] + np.arange(D1)[None, :]).ravel(),
                       seed).reshape(B, D1)
    for i in range(B):
        n = int(keep_len[i]) - 1
        a = 0
        rejected = False
        while a < n:
            j = a + 1
            r = int(cu[i]) + j - 1
            z = int(draft[i, j])
            p = target_probs(logits[r], temperature)
            qz = float(q[i, j - 1, z])
            uu = float(U[i, j - 1])          # position L_i + j - 1
            if uu * qz > 0.0 and p[z] > 0.0:
                margin[i] = min(margin[i], abs(math.log(uu * qz) - math.log(p[z])))
            if uu * qz < p[z]:
                a += 1
                continue
            rejected = True
            break
        r = int(cu[i]) + a
        pos = int(ctx_len[i]) + a
        G = gumbel([i], [pos], V, seed)[0]
        if rejected:
            rej[i] = r
            p = target_probs(logits[r], temperature)
            res = p - np.asarray(q[i, a], dtype=np.float64)
            with np.errstate(divide="ignore"):
                y = np.where(res > 0.0, np.log(np.where(res > 0.0, res, 1.0)), -np.inf) + G
            if not np.isfinite(y).any():
                y = np.asarray(logits[r], dtype=np.float64) / temperature + G
        else:
            y = np.asarray(logits[r], dtype=np.float64) / temperature + G
        t = int(np.argmax(y))
        nxt[i] = t
        acc[i] = a
        fin = np.sort(y[np.isfinite(y)])
        gap[i] = fin[-1] - fin[-2] if fin.size >= 2 else np.inf
    total = np.array([int((acc.astype(np.int64) + 1).sum())], dtype=np.int32)
    return dict(accept_len=acc, next_tok=nxt, total=total, rej_row=rej, margin=margin, gap=gap)


def lse_rows(logits: np.ndarray, temperature: float) -> np.ndarray:
    """ln sum_c exp(logits_c / T) per row, float64."""
    y = np.asarray(logits, dtype=np.float64) / float(temperature)
    m = y.max(axis=1)
    return m + np.log(np.exp(y - m[:, None]).sum(axis=1))
