"""Seeded synthetic workloads for the D-cut verify step.

This module only draws inputs: draft confidences, draft tokens, context
lengths, weights and cached keys/values.  It holds none of the method's
arithmetic (no prefix products, no ranking, no forward pass), so both the
HIP path and the CPU oracle can consume it without sharing computation.

Every tensor comes from its own counter-based Philox stream keyed by
(seed, config id, tensor tag[, request or chunk index]), so any single
tensor, or any one request's cache slab, can be regenerated on its own.

The five configurations restate the paper's problem shapes (a batch of B
requests, each with a bonus token plus D = 15 drafts, Sec. 3.1; block of 16
positions, Tab. 5) on 8B-class dense and MoE decoder layers.  The paper's
own drafter, models and benchmark suites are not available; these seeded
stand-ins replace them (confidences from Beta(a, 1) so that easy and hard
requests differ, Sec. 2.1).
"""
from __future__ import annotations

import concurrent.futures as _cf
import dataclasses
import math
import os
from typing import Dict, Optional, Tuple

import numpy as np

BF16_ONE = np.uint16(0x3F80)

_TAGS = {
    "conf": 1, "draft": 2, "ctx": 3, "match": 4, "amix": 5, "perm": 6,
    "q": 7, "q_draw": 8, "q_beta": 9,
    "embed": 10, "w_qkv": 11, "w_o": 12, "w_gate_up": 13, "w_down": 14,
    "w_lm": 15, "w_router": 16, "w_exp_gate_up": 17, "w_exp_down": 18,
    "kv_k": 20, "kv_v": 21, "argmax": 30,
}

_CHUNK = 1 << 22  # elements per independent weight stream


@dataclasses.dataclass(frozen=True)
class LayerShape:
    hidden: int
    n_q: int
    n_kv: int
    head_dim: int
    inter: int            # dense SwiGLU width (0 for MoE)
    vocab: int
    n_exp: int = 0        # 0 -> dense layer
    top_k: int = 0
    exp_inter: int = 0
    rms_eps: float = 1e-5
    rope_theta: float = 500000.0


@dataclasses.dataclass(frozen=True)
class Config:
    cid: int
    name: str
    B: int
    D: int
    layer: LayerShape
    ctx: Tuple[str, int, int]          # ("uniform"|"loguniform", lo, hi)
    conf_model: str                    # "u18" | "mix" | "lognormal"
    budgets: Tuple[int, ...]           # candidate K grid (ascending)
    weight_std: float = 0.02

    @property
    def rows_max(self) -> int:
        return self.B * (self.D + 1)

    @property
    def max_ctx(self) -> int:
        return self.ctx[2] + self.D + 1


_DENSE8B = dict(hidden=4096, n_q=32, n_kv=8, head_dim=128, inter=14336)


def _grid(B: int, D: int) -> Tuple[int, ...]:
    return tuple(B * m for m in range(1, D + 2))


CONFIGS: Dict[int, Config] = {
    1: Config(1, "tiny-4x16-h256", 4, 15,
              LayerShape(hidden=256, n_q=4, n_kv=2, head_dim=64, inter=688, vocab=1024),
              ("uniform", 64, 128), "u18", (24,)),
    2: Config(2, "dense8b-b16", 16, 15,
              LayerShape(vocab=128256, **_DENSE8B),
              ("uniform", 1024, 2048), "u18", _grid(16, 15)),
    3: Config(3, "dense8b-b64", 64, 15,
              LayerShape(vocab=128256, **_DENSE8B),
              ("uniform", 2048, 4096), "mix", _grid(64, 15)),
    4: Config(4, "moe-b128", 128, 15,
              LayerShape(hidden=2048, n_q=32, n_kv=4, head_dim=128, inter=0, vocab=151936,
                         n_exp=128, top_k=8, exp_inter=768, rope_theta=1000000.0),
              ("uniform", 1024, 4096), "u18", _grid(128, 15)),
    5: Config(5, "dense8b-b256-ragged", 256, 15,
              LayerShape(vocab=151936, **_DENSE8B),
              ("loguniform", 512, 8192), "lognormal", _grid(256, 15)),
}


def _gen(seed: int, cid: int, tag: str, *extra: int) -> np.random.Generator:
    ss = np.random.SeedSequence([int(seed), int(cid), _TAGS[tag], *[int(e) for e in extra]])
    return np.random.Generator(np.random.Philox(ss))


def bf16_round(x: np.ndarray) -> np.ndarray:
    """float32 -> raw bf16 bits, round-to-nearest-even (inputs are finite)."""
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    lsb = (b >> np.uint32(16)) & np.uint32(1)
    b = b + (np.uint32(0x7FFF) + lsb)
    return (b >> np.uint32(16)).astype(np.uint16)


def bf16_to_f32(u: np.ndarray) -> np.ndarray:
    return (np.asarray(u, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def _normal_bf16(seed: int, cid: int, tag: str, n: int, std: float,
                 workers: Optional[int] = None, layer: int = 0) -> np.ndarray:
    """n samples of N(0, std^2), bf16-rounded, generated in fixed 4M-element streams
    (decoder layer `layer` > 0 has streams of its own)."""
    out = np.empty(n, dtype=np.uint16)
    nchunks = (n + _CHUNK - 1) // _CHUNK
    lx = () if layer == 0 else (1_000_000 + layer,)

    def work(c: int) -> None:
        lo = c * _CHUNK
        hi = min(n, lo + _CHUNK)
        g = _gen(seed, cid, tag, c, *lx)
        v = g.standard_normal(hi - lo, dtype=np.float32)
        v *= np.float32(std)
        out[lo:hi] = bf16_round(v)

    if workers is None:
        workers = min(16, len(os.sched_getaffinity(0)))
    if nchunks <= 1 or workers <= 1:
        for c in range(nchunks):
            work(c)
    else:
        with _cf.ThreadPoolExecutor(workers) as ex:
            list(ex.map(work, range(nchunks)))
    return out


# ---------------------------------------------------------------- per-step inputs

def make_step_inputs(cfg: Config, seed: int) -> Dict[str, np.ndarray]:
    """Confidences, bonus+draft tokens (unforced), match uniforms, context lengths."""
    B, D, V = cfg.B, cfg.D, cfg.layer.vocab
    g = _gen(seed, cfg.cid, "amix")
    if cfg.conf_model == "u18":
        a = g.uniform(1.0, 8.0, size=B)
    elif cfg.conf_model == "mix":
        perm = _gen(seed, cfg.cid, "perm").permutation(B)
        a = np.full(B, 1.2)
        a[perm[: B // 2]] = 6.0          # exactly half easy, half hard
    elif cfg.conf_model == "lognormal":
        a = np.exp(0.5 + g.standard_normal(B))
    else:
        raise ValueError(cfg.conf_model)
    u = _gen(seed, cfg.cid, "conf").random((B, D))
    # Beta(a,1) by inverse CDF: U^(1/a).  Computed in float64, stored as float32.
    conf = np.power(u, 1.0 / a[:, None]).astype(np.float32)
    draft = _gen(seed, cfg.cid, "draft").integers(0, V, size=(B, D + 1), dtype=np.int64).astype(np.int32)
    match_u = _gen(seed, cfg.cid, "match").random((B, D)).astype(np.float32)
    kind, lo, hi = cfg.ctx
    gc = _gen(seed, cfg.cid, "ctx")
    if kind == "uniform":
        ctx = gc.integers(lo, hi + 1, size=B)
    else:
        ctx = np.rint(np.exp(gc.uniform(math.log(lo), math.log(hi), size=B)))
        ctx = np.clip(ctx, lo, hi)
    ctx = ctx.astype(np.int32)
    return dict(a=a, conf=conf, draft=draft, match_u=match_u, ctx_len=ctx)


def kv_layout(cfg: Config, ctx_len: np.ndarray) -> Tuple[np.ndarray, np.ndarray, int]:
    """Per-request slabs [n_kv][cap_i][head_dim]; cap_i = L_i + D + 1.

    Returns (cap[B] int32, base[B] int64 element offsets, total elements)."""
    cap = (ctx_len.astype(np.int64) + cfg.D + 1)
    slab = cap * cfg.layer.n_kv * cfg.layer.head_dim
    base = np.zeros(cfg.B, dtype=np.int64)
    base[1:] = np.cumsum(slab)[:-1]
    return cap.astype(np.int32), base, int(slab.sum())


def make_kv_request(cfg: Config, seed: int, i: int, L: int, which: str, layer: int = 0) -> np.ndarray:
    """Cached entries of request i: [n_kv][L][head_dim] raw bf16 bits (of decoder layer `layer`)."""
    ly = cfg.layer
    g = _gen(seed, cfg.cid, "kv_k" if which == "k" else "kv_v", i, *(() if layer == 0 else (1_000_000 + layer,)))
    v = g.standard_normal((ly.n_kv, L, ly.head_dim), dtype=np.float32)
    v *= np.float32(cfg.weight_std)
    return bf16_round(v).reshape(ly.n_kv, L, ly.head_dim)


def make_kv(cfg: Config, seed: int, ctx_len: np.ndarray,
            requests: Optional[np.ndarray] = None, layer: int = 0) -> Dict[str, np.ndarray]:
    """Full flat caches k, v (uint16 bf16 bits) with slots >= L_i zeroed (of decoder layer `layer`)."""
    cap, base, total = kv_layout(cfg, ctx_len)
    ly = cfg.layer
    k = np.zeros(total, dtype=np.uint16)
    v = np.zeros(total, dtype=np.uint16)
    reqs = range(cfg.B) if requests is None else requests

    def work(i: int) -> None:
        L = int(ctx_len[i])
        c = int(cap[i])
        sk = k[base[i]: base[i] + ly.n_kv * c * ly.head_dim].reshape(ly.n_kv, c, ly.head_dim)
        sv = v[base[i]: base[i] + ly.n_kv * c * ly.head_dim].reshape(ly.n_kv, c, ly.head_dim)
        sk[:, :L, :] = make_kv_request(cfg, seed, i, L, "k", layer)
        sv[:, :L, :] = make_kv_request(cfg, seed, i, L, "v", layer)

    workers = min(16, len(os.sched_getaffinity(0)))
    with _cf.ThreadPoolExecutor(workers) as ex:
        list(ex.map(work, reqs))
    return dict(k=k, v=v, cap=cap, base=base)


def make_weights(cfg: Config, seed: int = 0, with_embed: bool = True, layer: int = 0) -> Dict[str, np.ndarray]:
    """Layer + LM-head weights as raw bf16 bits, PyTorch Linear layout [out][in].

    Linear/embedding weights ~ N(0, std^2) (std 0.02); norm gains are 1.0.
    The MoE router uses std 1/sqrt(hidden) so its logits are about N(0, 1)
    on unit-RMS inputs.  Decoder layer `layer` > 0 draws its layer weights
    from streams of its own and carries no embedding, final norm or LM head."""
    if layer > 0:
        return _layer_weights(cfg, seed, layer)
    ly = cfg.layer
    H, hd = ly.hidden, ly.head_dim
    s = cfg.weight_std
    w: Dict[str, np.ndarray] = {}
    nqkv = (ly.n_q + 2 * ly.n_kv) * hd
    if with_embed:
        w["embed"] = _normal_bf16(seed, cfg.cid, "embed", ly.vocab * H, s).reshape(ly.vocab, H)
    w["attn_norm"] = np.full(H, BF16_ONE, dtype=np.uint16)
    w["w_qkv"] = _normal_bf16(seed, cfg.cid, "w_qkv", nqkv * H, s).reshape(nqkv, H)
    w["w_o"] = _normal_bf16(seed, cfg.cid, "w_o", H * ly.n_q * hd, s).reshape(H, ly.n_q * hd)
    w["mlp_norm"] = np.full(H, BF16_ONE, dtype=np.uint16)
    if ly.n_exp == 0:
        w["w_gate_up"] = _normal_bf16(seed, cfg.cid, "w_gate_up", 2 * ly.inter * H, s).reshape(2 * ly.inter, H)
        w["w_down"] = _normal_bf16(seed, cfg.cid, "w_down", H * ly.inter, s).reshape(H, ly.inter)
    else:
        E, Ie = ly.n_exp, ly.exp_inter
        w["w_router"] = _normal_bf16(seed, cfg.cid, "w_router", E * H, 1.0 / math.sqrt(H)).reshape(E, H)
        w["w_exp_gate_up"] = _normal_bf16(seed, cfg.cid, "w_exp_gate_up", E * 2 * Ie * H, s).reshape(E, 2 * Ie, H)
        w["w_exp_down"] = _normal_bf16(seed, cfg.cid, "w_exp_down", E * H * Ie, s).reshape(E, H, Ie)
    w["final_norm"] = np.full(H, BF16_ONE, dtype=np.uint16)
    w["w_lm"] = _normal_bf16(seed, cfg.cid, "w_lm", ly.vocab * H, s).reshape(ly.vocab, H)
    return w


def _layer_weights(cfg: Config, seed: int, layer: int) -> Dict[str, np.ndarray]:
    ly = cfg.layer
    H, hd = ly.hidden, ly.head_dim
    s = cfg.weight_std
    nqkv = (ly.n_q + 2 * ly.n_kv) * hd
    nb = lambda tag, n, std: _normal_bf16(seed, cfg.cid, tag, n, std, layer=layer)
    w: Dict[str, np.ndarray] = {}
    w["attn_norm"] = np.full(H, BF16_ONE, dtype=np.uint16)
    w["w_qkv"] = nb("w_qkv", nqkv * H, s).reshape(nqkv, H)
    w["w_o"] = nb("w_o", H * ly.n_q * hd, s).reshape(H, ly.n_q * hd)
    w["mlp_norm"] = np.full(H, BF16_ONE, dtype=np.uint16)
    if ly.n_exp == 0:
        w["w_gate_up"] = nb("w_gate_up", 2 * ly.inter * H, s).reshape(2 * ly.inter, H)
        w["w_down"] = nb("w_down", H * ly.inter, s).reshape(H, ly.inter)
    else:
        E, Ie = ly.n_exp, ly.exp_inter
        w["w_router"] = nb("w_router", E * H, 1.0 / math.sqrt(H)).reshape(E, H)
        w["w_exp_gate_up"] = nb("w_exp_gate_up", E * 2 * Ie * H, s).reshape(E, 2 * Ie, H)
        w["w_exp_down"] = nb("w_exp_down", E * H * Ie, s).reshape(E, H, Ie)
    return w


def synthetic_argmax(cfg: Config, seed: int, draft: np.ndarray, match_u: np.ndarray,
                     conf: np.ndarray) -> np.ndarray:
    """A stand-in target argmax table g[i][k] (k = 0..D) for acceptance tests.

    g[i][k-1] equals draft[i][k] with probability conf[i][k-1] (decided by the
    stored uniforms), otherwise an unrelated uniform token."""
    B, D, V = cfg.B, cfg.D, cfg.layer.vocab
    g = _gen(seed, cfg.cid, "argmax").integers(0, V, size=(B, D + 1), dtype=np.int64).astype(np.int32)
    hit = match_u < conf
    g[:, :D] = np.where(hit, draft[:, 1:], g[:, :D])
    return g


def make_proposals(cfg: Config, seed: int, bonus: np.ndarray) -> Dict[str, np.ndarray]:
    """Proposal distributions of a stochastic drafter, for rejection-sampling tests.

    q[i][k-1] = softmax(beta_i * g) over the vocabulary with g ~ N(0, 1) per
    entry and beta_i ~ U[1, 4] per request (larger beta, more peaked), formed in
    float64 and stored as float32.  Draft z_{i,k} is drawn from q[i][k-1] by
    inverse CDF with its own stored uniform, and its confidence is
    q[i][k-1][z_{i,k}] (the drafter's probability of what it proposed).
    Column 0 of `draft` is `bonus`."""
    B, D, V = cfg.B, cfg.D, cfg.layer.vocab
    beta = _gen(seed, cfg.cid, "q_beta").uniform(1.0, 4.0, size=B)
    q = np.empty((B, D, V), dtype=np.float32)
    draft = np.zeros((B, D + 1), dtype=np.int32)
    draft[:, 0] = np.asarray(bonus, dtype=np.int32)
    conf = np.zeros((B, D), dtype=np.float32)
    for i in range(B):
        gi = _gen(seed, cfg.cid, "q", i).standard_normal((D, V)) * beta[i]
        e = np.exp(gi - gi.max(axis=1, keepdims=True))
        qi = (e / e.sum(axis=1, keepdims=True)).astype(np.float32)
        q[i] = qi
        u = _gen(seed, cfg.cid, "q_draw", i).random(D)
        cdf = np.cumsum(qi.astype(np.float64), axis=1)
        z = np.minimum((cdf < (u * cdf[:, -1])[:, None]).sum(axis=1), V - 1)
        draft[i, 1:] = z
        conf[i] = qi[np.arange(D), z]
    return dict(q=q, draft=draft, conf=conf, beta=beta)
