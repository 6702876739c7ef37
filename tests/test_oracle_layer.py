"""Pins for the layer / LM-head oracle: library routines, closed forms, special cases, causality."""
import dataclasses
import functools

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import layer as olay
from oracle import lm_head as olm
from oracle import select as osel
from paper_2607_14647_amd import workload as wl


# ------------------------------------------------------------------ building blocks

def test_rmsnorm_library_and_closed_form():
    rng = np.random.default_rng(0)
    x = rng.standard_normal((5, 33))
    g = rng.standard_normal(33)
    ref = F.rms_norm(torch.from_numpy(x), (33,), torch.from_numpy(g), eps=1e-5).numpy()
    assert np.allclose(olay.rmsnorm(x, g, 1e-5), ref, rtol=1e-12, atol=1e-12)
    c = np.full((2, 16), -3.0)
    out = olay.rmsnorm(c, np.ones(16), 0.0)
    assert np.array_equal(out, np.full((2, 16), -1.0))


def test_rope_complex_rotation():
    """RoPE equals multiplying (x_j + i x_{j+hd/2}) by exp(i pos theta^(-2j/hd))."""
    rng = np.random.default_rng(1)
    hd, theta = 16, 10000.0
    x = rng.standard_normal((3, hd))
    pos = np.array([0.0, 1.0, 777.0])
    z = x[:, : hd // 2] + 1j * x[:, hd // 2:]
    freq = np.array([theta ** (-(2.0 * j) / hd) for j in range(hd // 2)])
    zr = z * np.exp(1j * pos[:, None] * freq[None, :])
    ref = np.concatenate([zr.real, zr.imag], axis=1)
    got = olay.rope(x, pos, theta)
    assert np.allclose(got, ref, rtol=1e-12, atol=1e-12)
    assert np.array_equal(got[0], x[0])                          # pos 0: identity
    assert np.allclose(np.linalg.norm(got, axis=1), np.linalg.norm(x, axis=1))


def test_rope_hand_values():
    x = np.array([1.0, 0.0, 0.0, 1.0])          # pairs (x0, x2) = (1, 0), (x1, x3) = (0, 1)
    out = olay.rope(x, np.array(2.0), 100.0)    # freqs 1 and 100^(-1/2) = 0.1
    want = [np.cos(2.0), -np.sin(0.2), np.sin(2.0), np.cos(0.2)]
    assert np.allclose(out, want, rtol=0, atol=1e-15)


def test_silu_library():
    x = np.linspace(-20, 20, 101)
    assert np.allclose(olay.silu(x), F.silu(torch.from_numpy(x)).numpy(), rtol=1e-12, atol=1e-14)


def _sdpa_dense(q, k_all, v_all, L):
    """Per-request dense masked attention over the whole L+d sequence via torch SDPA."""
    d, nq, hd = q.shape
    nkv, n, _ = k_all.shape
    grp = nq // nkv
    kk = torch.from_numpy(np.repeat(k_all, grp, axis=0))[None]          # [1][nq][n][hd]
    vv = torch.from_numpy(np.repeat(v_all, grp, axis=0))[None]
    qq = torch.from_numpy(np.ascontiguousarray(q.transpose(1, 0, 2)))[None]  # [1][nq][d][hd]
    mask = torch.from_numpy(np.arange(n)[None, :] <= (L + np.arange(d))[:, None])
    out = F.scaled_dot_product_attention(qq, kk, vv, attn_mask=mask)
    return out[0].numpy().transpose(1, 0, 2)


@pytest.mark.parametrize("nq,nkv,L,d", [(4, 2, 37, 5), (8, 8, 0, 3), (6, 1, 100, 16), (2, 2, 5, 1)])
def test_attention_ragged_equals_dense(nq, nkv, L, d):
    rng = np.random.default_rng(nq * 100 + L)
    hd = 16
    q = rng.standard_normal((d, nq, hd))
    k_all = rng.standard_normal((nkv, L + d, hd))
    v_all = rng.standard_normal((nkv, L + d, hd))
    got = olay.attention(q, k_all, v_all, L)
    ref = _sdpa_dense(q, k_all, v_all, L)
    assert np.allclose(got, ref, rtol=1e-6, atol=1e-9)


def test_attention_special_cases():
    rng = np.random.default_rng(3)
    hd = 8
    # L = 0, first block row: its only key is itself -> output is its own value
    q = rng.standard_normal((1, 2, hd))
    k = rng.standard_normal((1, 1, hd))
    v = rng.standard_normal((1, 1, hd))
    out = olay.attention(q, k, v, 0)
    assert np.allclose(out[0, 0], v[0, 0]) and np.allclose(out[0, 1], v[0, 0])
    # zero query -> uniform weights -> mean of the visible values
    L, d = 9, 3
    k = rng.standard_normal((1, L + d, hd))
    v = rng.standard_normal((1, L + d, hd))
    out = olay.attention(np.zeros((d, 1, hd)), k, v, L)
    for r in range(d):
        assert np.allclose(out[r, 0], v[0, : L + r + 1].mean(axis=0))


def test_moe_routing_rules():
    logits = np.array([[0.0, 2.0, 2.0, 1.0, 2.0]])
    p, ids, w = olay.topk_route(logits, 2)
    assert ids.tolist() == [[1, 2]]                              # ties -> lower expert id
    assert np.allclose(w, [[0.5, 0.5]])
    p, ids, w = olay.topk_route(logits, 5)                       # top_k = E -> weights are p
    assert np.allclose(np.sort(w[0]), np.sort(p[0]))
    assert np.isclose(p.sum(), 1.0)


def test_lm_head_tie_rule_and_one_hot():
    rng = np.random.default_rng(4)
    H, V = 8, 16
    W = np.zeros((V, H))
    for j in range(V):
        W[j, j % H] = 1.0                       # rows j and j+8 are identical one-hots
    x = rng.standard_normal((6, H))
    out = olm.lm_head_argmax(x, np.ones(H), 0.0, W)
    f = x / np.sqrt((x * x).mean(axis=1, keepdims=True))
    assert np.allclose(out["logits"][:, :H], f)
    assert (out["argmax"] == np.argmax(f, axis=1)).all()        # the lower of the two twins
    assert np.allclose(out["gap"], 0.0)                          # twin rows tie exactly


# ------------------------------------------------------------------ whole layer on config 1

@functools.lru_cache(maxsize=2)
def _cfg1(seed=0, moe=False):
    cfg = wl.CONFIGS[1]
    if moe:
        ly = dataclasses.replace(cfg.layer, inter=0, n_exp=6, top_k=2, exp_inter=40)
        cfg = dataclasses.replace(cfg, layer=ly, cid=91)
    st = wl.make_step_inputs(cfg, seed)
    w = wl.make_weights(cfg, seed)
    kv = wl.make_kv(cfg, seed, st["ctx_len"])
    return cfg, st, olay.prepare_weights(w), kv


def _run(cfg, st, w64, kv, K, row_exact, x_in=None):
    sel = osel.select(st["conf"], st["draft"], st["ctx_len"], [K], [1.0])
    lay = olay.verify_layer(cfg.layer, w64, kv, sel["cu"], sel["packed_tok"], sel["packed_pos"],
                            sel["packed_req"], st["ctx_len"], cfg.D, x_in=x_in, row_exact=row_exact)
    lm = olm.lm_head_argmax(lay["x_out"], w64["final_norm"], cfg.layer.rms_eps, w64["w_lm"]) \
        if not row_exact else _lm_rows(lay["x_out"], w64, cfg)
    return sel, lay, lm


def _lm_rows(x, w64, cfg):
    rows = [olm.lm_head_argmax(x[r:r + 1].copy(), w64["final_norm"], cfg.layer.rms_eps, w64["w_lm"])
            for r in range(x.shape[0])]
    return {k: np.concatenate([r[k] for r in rows]) for k in rows[0]}


@pytest.mark.parametrize("moe", [False, True])
def test_causality_row_exact(moe):
    """A kept row's outputs do not depend on which later positions are pruned (bitwise)."""
    cfg, st, w64, kv = _cfg1(0, moe)
    B, D = cfg.B, cfg.D
    sf, lf, mf = _run(cfg, st, w64, kv, B * (D + 1), True)
    sp, lp, mp = _run(cfg, st, w64, kv, 24, True)
    for i in range(B):
        for k in range(int(sp["keep_len"][i])):
            tf, tp = sf["cu"][i] + k, sp["cu"][i] + k
            assert np.array_equal(lf["x_out"][tf], lp["x_out"][tp])
            assert np.array_equal(lf["new_k"][tf], lp["new_k"][tp])
            assert np.array_equal(mf["logits"][tf], mp["logits"][tp])


def test_causality_blocked():
    cfg, st, w64, kv = _cfg1(0)
    B, D = cfg.B, cfg.D
    sf, lf, mf = _run(cfg, st, w64, kv, B * (D + 1), False)
    sp, lp, mp = _run(cfg, st, w64, kv, 24, False)
    for i in range(B):
        for k in range(int(sp["keep_len"][i])):
            tf, tp = sf["cu"][i] + k, sp["cu"][i] + k
            assert np.allclose(mf["logits"][tf], mp["logits"][tp], rtol=1e-6, atol=1e-9)


def test_request_independence_and_x_in():
    """Reordering requests reorders rows; passing the gathered embeddings as x_in changes nothing."""
    cfg, st, w64, kv = _cfg1(0)
    B = cfg.B
    s1, l1, _ = _run(cfg, st, w64, kv, 40, False)
    x_in = olay.bf16_bits_to_f64(w64["embed"][s1["packed_tok"][:40]]).astype(np.float32)
    s2, l2, _ = _run(cfg, st, w64, kv, 40, False, x_in=x_in)
    assert np.array_equal(l1["x_out"], l2["x_out"])
    perm = np.arange(B)[::-1]
    st_p = dict(st, conf=st["conf"][perm], draft=st["draft"][perm], ctx_len=st["ctx_len"][perm])
    cap, base = kv["cap"][perm], kv["base"][perm]
    kv_p = dict(kv, cap=cap, base=base)
    s3, l3, _ = _run(cfg, st_p, w64, kv_p, 40, False)
    for j, i in enumerate(perm):
        a = l1["x_out"][s1["cu"][i]: s1["cu"][i + 1]]
        b = l3["x_out"][s3["cu"][j]: s3["cu"][j + 1]]
        assert np.allclose(a, b, rtol=1e-12, atol=1e-12)


def test_moe_identical_experts_reduce_to_dense():
    cfg, st, w64, kv = _cfg1(0, True)
    ly = cfg.layer
    w = dict(w64)
    w["w_exp_gate_up"] = np.repeat(w64["w_exp_gate_up"][:1], ly.n_exp, axis=0)
    w["w_exp_down"] = np.repeat(w64["w_exp_down"][:1], ly.n_exp, axis=0)
    dense_ly = dataclasses.replace(ly, n_exp=0, top_k=0, inter=ly.exp_inter)
    wd = dict(w, w_gate_up=w64["w_exp_gate_up"][0], w_down=w64["w_exp_down"][0])
    sel = osel.select(st["conf"], st["draft"], st["ctx_len"], [30], [1.0])
    args = (kv, sel["cu"], sel["packed_tok"], sel["packed_pos"], sel["packed_req"], st["ctx_len"], cfg.D)
    a = olay.verify_layer(ly, w, *args)["x_out"]
    b = olay.verify_layer(dense_ly, wd, *args)["x_out"]
    assert np.allclose(a, b, rtol=1e-12, atol=1e-12)


def test_forced_drafts_accept_as_constructed():
    """Drafts forced from the oracle's own greedy tokens are accepted up to the first unforced depth."""
    from oracle import drafts as odr
    from oracle import accept as oacc
    cfg, st, w64, kv = _cfg1(0)
    B, D = cfg.B, cfg.D
    z = odr.force_matches(cfg.layer, w64, kv, st["conf"], st["draft"], st["match_u"], st["ctx_len"], D)
    sel = osel.select(st["conf"], z, st["ctx_len"], [B * (D + 1)], [1.0])
    lay = olay.verify_layer(cfg.layer, w64, kv, sel["cu"], sel["packed_tok"], sel["packed_pos"],
                            sel["packed_req"], st["ctx_len"], D)
    lm = olm.lm_head_argmax(lay["x_out"], w64["final_norm"], cfg.layer.rms_eps, w64["w_lm"])
    acc = oacc.accept(z, sel["keep_len"], sel["cu"], lm["argmax"])
    hit = st["match_u"] < st["conf"]
    for i in range(B):
        first_miss = int(np.argmin(np.append(hit[i], False)))
        assert acc["accept_len"][i] >= first_miss


def test_round_bf16_matches_torch_bfloat16():
    """The oracle's bf16 rounding (float64 -> float32 -> nearest even bf16) equals torch's
    float32 -> bfloat16 conversion, ties included."""
    import torch
    rng = np.random.default_rng(5)
    x = np.concatenate([rng.standard_normal(20000) * 10.0 ** rng.integers(-6, 6, 20000),
                        [0.0, -0.0, 1.0, -1.5, 3.0e38, -3.0e38, 1e-40]])
    # exact ties: float32 values whose low 16 bits are 0x8000, with even and odd bf16 neighbours
    ties = (np.arange(0x3F800000, 0x3F800000 + 64 * 0x10000, 0x10000, dtype=np.uint32) + 0x8000).view(np.float32)
    x = np.concatenate([x, ties.astype(np.float64), -ties.astype(np.float64)])
    ref = torch.from_numpy(x.astype(np.float32)).to(torch.bfloat16).to(torch.float64).numpy()
    got = olay.round_bf16(x)
    assert np.array_equal(got, ref)
    assert np.array_equal(olay.round_bf16(got), got)          # idempotent


def test_bf16_activation_mode_rounds_only_where_stated():
    """act_bf16 changes the forward only by bf16 roundings of the stored activations: the
    appended keys and values come out bf16-representable, the results stay within a few
    bf16 ulps of the float64 forward (relative to the row), and they are not identical."""
    cfg = wl.CONFIGS[1]
    st = wl.make_step_inputs(cfg, 0)
    w = wl.make_weights(cfg, 0)
    kv = wl.make_kv(cfg, 0, st["ctx_len"])
    sel = osel.select(st["conf"], st["draft"], st["ctx_len"], [40], [1.0])
    w64 = olay.prepare_weights(w)
    args = (cfg.layer, w64, kv, sel["cu"], sel["packed_tok"], sel["packed_pos"], sel["packed_req"],
            st["ctx_len"], cfg.D)
    ref = olay.verify_layer(*args)
    got = olay.verify_layer(*args, act_bf16=True)
    for name in ("new_k", "new_v"):
        assert np.array_equal(olay.round_bf16(got[name]), got[name])
        assert np.abs(got[name] - ref[name]).max() <= 2.0 ** -8 * np.abs(ref[name]).max()
    rel = np.abs(got["x_out"] - ref["x_out"]).max(axis=1) / np.abs(ref["x_out"]).max(axis=1)
    assert 0 < rel.max() < 2e-2
    lm = olm.lm_head_argmax(ref["x_out"], w64["final_norm"], cfg.layer.rms_eps, w64["w_lm"])
    lm16 = olm.lm_head_argmax(got["x_out"], w64["final_norm"], cfg.layer.rms_eps, w64["w_lm"], act_bf16=True)
    rl = np.abs(lm16["logits"] - lm["logits"]).max(axis=1) / np.abs(lm["logits"]).max(axis=1)
    assert 0 < rl.max() < 2e-2
