"""Oracle for the packed ragged verify forward of one decoder layer (test infrastructure only).

What is computed is the plain definition of one pre-norm decoder layer over
the packed rows (App. C: the kept prefixes are concatenated into one batch
with block and position metadata, and every kept position is scored against
its request's accepted prefix).  The paper names the target models but not
their internals, so the layer follows the usual Llama/Qwen form:

  x    = x_in[t]            or  E[token_t]                  (residual, float64)
  h    = x / sqrt(mean(x^2) + eps) * g1                     (RMSNorm)
  q,k,v = h W_qkv^T split by heads; RoPE on q and k at pos_t
  RoPE: pairs (j, j + hd/2), angle pos * theta^(-2j/hd), i.e. the complex
        rotation (x_j + i x_{j+hd/2}) * exp(i * angle)
  attn: row (i, k), head h, kv group h // (n_q / n_kv) attends to the cached
        keys 0..L_i-1 and to its own block's keys 0..k; scale 1/sqrt(hd);
        max-subtracted softmax
  y    = x + attn W_o^T
  h2   = RMSNorm(y) * g2
  dense: out = y + (SiLU(h2 W_gate^T) * (h2 W_up^T)) W_down^T
  MoE:   p = softmax(h2 W_router^T); top_k experts by p (ties -> lower id);
         w = p / sum(p over the top_k); out = y + sum_e w_e SwiGLU_e(h2)

All arithmetic is float64 on the exact bf16 values of weights and cache.
`row_exact=True` evaluates every product one row at a time with the same
shapes, so a row's result cannot depend on which other rows are present.

`act_bf16=True` is the same definition with the tensors the verify step
holds in bf16 between its operations rounded to bf16 (nearest even) where
they are formed: the normalised rows h and h2, q after RoPE, the keys and
values appended to the (bf16) cache, the attention output and the SwiGLU
product.  Everything else stays float64.  The argmax is an integer decided
by floating point, so the tests take that decision on logits formed from the
same bf16 activations as the path under test (the logit and residual
tolerances are still checked against the plain float64 forward).
"""
from __future__ import annotations

from typing import Dict, Optional, Sequence

import numpy as np

from .errors import DcutDataError, DERR_TOKEN, DERR_CAPACITY


def bf16_bits_to_f64(u: np.ndarray) -> np.ndarray:
    """Exact value of raw bf16 bits (the top half of a float32)."""
    u32 = np.asarray(u, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return u32.view(np.float32).astype(np.float64)


def prepare_weights(w: Dict[str, np.ndarray]) -> Dict[str, np.ndarray]:
    """float64 copies of every weight (the embedding stays as bits, gathered per row)."""
    out = {}
    for name, arr in w.items():
        out[name] = arr if name == "embed" else bf16_bits_to_f64(arr)
    return out


def round_bf16(x: np.ndarray) -> np.ndarray:
    """Nearest bf16 value (ties to even) of float64 values, as float64: first to float32
    (the precision the activations are formed in), then to the 8-bit significand."""
    f = np.ascontiguousarray(x, dtype=np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) >> 16 << 16
    return u.astype(np.uint32).view(np.float32).astype(np.float64).reshape(np.shape(x))


def rmsnorm(x: np.ndarray, gain: np.ndarray, eps: float) -> np.ndarray:
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * gain


def rope(x: np.ndarray, pos: np.ndarray, theta: float) -> np.ndarray:
    """Rotate-half RoPE on the last axis; pos broadcasts against x[..., 0]."""
    hd = x.shape[-1]
    half = hd // 2
    j = np.arange(half, dtype=np.float64)
    inv_freq = theta ** (-2.0 * j / hd)
    ang = np.asarray(pos, dtype=np.float64)[..., None] * inv_freq
    c, s = np.cos(ang), np.sin(ang)
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def silu(x: np.ndarray) -> np.ndarray:
    return x / (1.0 + np.exp(-x))


def _mm(a: np.ndarray, w: np.ndarray, row_exact: bool) -> np.ndarray:
    """a [n][in] times w[out][in]^T."""
    if not row_exact:
        return a @ w.T
    out = np.empty((a.shape[0], w.shape[0]), dtype=np.float64)
    for r in range(a.shape[0]):
        out[r] = w @ np.array(a[r], dtype=np.float64, copy=True)
    return out


def attention(q: np.ndarray, k_all: np.ndarray, v_all: np.ndarray, L: int) -> np.ndarray:
    """Ragged causal attention of one request's d kept rows.

    q [d][n_q][hd]; k_all, v_all [n_kv][L + d][hd] (cache then block).
    Row r attends to keys 0 .. L + r."""
    d, nq, hd = q.shape
    nkv = k_all.shape[0]
    grp = nq // nkv
    out = np.empty_like(q)
    scale = 1.0 / np.sqrt(hd)
    for r in range(d):
        n = L + r + 1
        for h in range(nq):
            g = h // grp
            sc = (k_all[g, :n] @ q[r, h]) * scale
            p = np.exp(sc - sc.max())
            out[r, h] = (p @ v_all[g, :n]) / p.sum()
    return out


def topk_route(logits: np.ndarray, top_k: int):
    """Softmax probabilities, top_k expert ids (ties -> lower id), renormalised weights."""
    z = logits - logits.max(axis=-1, keepdims=True)
    p = np.exp(z)
    p /= p.sum(axis=-1, keepdims=True)
    order = np.argsort(-p, axis=-1, kind="stable")
    ids = order[..., :top_k]
    pt = np.take_along_axis(p, ids, axis=-1)
    w = pt / pt.sum(axis=-1, keepdims=True)
    return p, ids, w


def verify_layer(ly, w64: Dict[str, np.ndarray], kv: Dict[str, np.ndarray],
                 cu: np.ndarray, packed_tok: np.ndarray, packed_pos: np.ndarray,
                 packed_req: np.ndarray, ctx_len: np.ndarray, D: int,
                 x_in: Optional[np.ndarray] = None,
                 requests: Optional[Sequence[int]] = None,
                 row_exact: bool = False, act_bf16: bool = False) -> Dict[str, np.ndarray]:
    """Layer forward over the packed rows of `requests` (default: all).

    Returns x_out [K*][H] (rows of other requests are NaN), the appended keys
    (after RoPE) and values new_k/new_v [K*][n_kv][hd], and, for MoE layers,
    router probabilities/ids per row."""
    H, nq, nkv, hd = ly.hidden, ly.n_q, ly.n_kv, ly.head_dim
    act = round_bf16 if act_bf16 else (lambda a: a)
    B = len(ctx_len)
    Kstar = int(cu[B])
    x_out = np.full((Kstar, H), np.nan)
    new_k = np.full((Kstar, nkv, hd), np.nan)
    new_v = np.full((Kstar, nkv, hd), np.nan)
    moe = ly.n_exp > 0
    r_ids = np.full((Kstar, max(ly.top_k, 1)), -1, dtype=np.int64)
    r_gap = np.full(Kstar, np.inf)
    reqs = range(B) if requests is None else requests
    for i in reqs:
        t0, t1 = int(cu[i]), int(cu[i + 1])
        d = t1 - t0
        L = int(ctx_len[i])
        cap = int(kv["cap"][i])
        if L < 0 or L + D + 1 > cap:
            raise DcutDataError(DERR_CAPACITY, f"request {i}: L={L} cap={cap}")
        if x_in is not None:
            x = np.asarray(x_in[t0:t1], dtype=np.float64)
        else:
            tok = packed_tok[t0:t1]
            if (tok < 0).any() or (tok >= ly.vocab).any():
                raise DcutDataError(DERR_TOKEN, f"request {i}: token out of range")
            x = bf16_bits_to_f64(w64["embed"][tok])
        h = act(rmsnorm(x, w64["attn_norm"], ly.rms_eps))
        qkv = _mm(h, w64["w_qkv"], row_exact).reshape(d, nq + 2 * nkv, hd)
        pos = packed_pos[t0:t1].astype(np.float64)
        q = act(rope(qkv[:, :nq], pos[:, None], ly.rope_theta))
        kb = act(rope(qkv[:, nq:nq + nkv], pos[:, None], ly.rope_theta))
        vb = act(qkv[:, nq + nkv:])
        base = int(kv["base"][i])
        slab = nkv * cap * hd
        ck = bf16_bits_to_f64(kv["k"][base: base + slab]).reshape(nkv, cap, hd)[:, :L]
        cv = bf16_bits_to_f64(kv["v"][base: base + slab]).reshape(nkv, cap, hd)[:, :L]
        k_all = np.concatenate([ck, kb.transpose(1, 0, 2)], axis=1)
        v_all = np.concatenate([cv, vb.transpose(1, 0, 2)], axis=1)
        att = act(attention(q, k_all, v_all, L).reshape(d, nq * hd))
        y = x + _mm(att, w64["w_o"], row_exact)
        h2 = act(rmsnorm(y, w64["mlp_norm"], ly.rms_eps))
        if not moe:
            gu = _mm(h2, w64["w_gate_up"], row_exact)
            m = act(silu(gu[:, : ly.inter]) * gu[:, ly.inter:])
            out = y + _mm(m, w64["w_down"], row_exact)
        else:
            logits = _mm(h2, w64["w_router"], row_exact)
            p, ids, wts = topk_route(logits, ly.top_k)
            out = y.copy()
            Ie = ly.exp_inter
            for r in range(d):
                acc = np.zeros(H)
                for slot in range(ly.top_k):
                    e = int(ids[r, slot])
                    gu = w64["w_exp_gate_up"][e] @ h2[r]
                    m = act(silu(gu[:Ie]) * gu[Ie:])
                    acc += wts[r, slot] * (w64["w_exp_down"][e] @ m)
                out[r] += acc
            r_ids[t0:t1] = ids
            srt = np.sort(logits, axis=-1)[:, ::-1]
            r_gap[t0:t1] = srt[:, ly.top_k - 1] - srt[:, ly.top_k]
        x_out[t0:t1] = out
        new_k[t0:t1] = kb
        new_v[t0:t1] = vb
    res = dict(x_out=x_out, new_k=new_k, new_v=new_v)
    if moe:
        res["router_ids"] = r_ids
        res["router_gap"] = r_gap
    return res
