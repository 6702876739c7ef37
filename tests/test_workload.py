"""The seeded generator: reproducible, per-request regenerable, shaped as the five configurations."""
import numpy as np
import torch

from paper_2607_14647_amd import workload as wl


def test_bf16_round_matches_torch():
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(10000).astype(np.float32) * 3,
                        np.array([1.00390625, 1.01171875, -2.0, 0.0, 1e-30], np.float32)])
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(wl.bf16_round(x), ref)


def test_reproducible_and_shaped():
    for cid, cfg in wl.CONFIGS.items():
        a = wl.make_step_inputs(cfg, 3)
        b = wl.make_step_inputs(cfg, 3)
        for k in a:
            assert np.array_equal(a[k], b[k])
        B, D = cfg.B, cfg.D
        assert a["conf"].shape == (B, D) and a["draft"].shape == (B, D + 1)
        assert (a["conf"] >= 0).all() and (a["conf"] <= 1).all()
        assert (a["draft"] >= 0).all() and (a["draft"] < cfg.layer.vocab).all()
        lo, hi = cfg.ctx[1], cfg.ctx[2]
        assert (a["ctx_len"] >= lo).all() and (a["ctx_len"] <= hi).all()
        assert cfg.budgets[0] >= B and cfg.budgets[-1] <= B * (D + 1)
    mix = wl.make_step_inputs(wl.CONFIGS[3], 0)["a"]
    assert (mix == 6.0).sum() == 32 and (mix == 1.2).sum() == 32


def test_kv_regenerates_per_request():
    cfg = wl.CONFIGS[1]
    st = wl.make_step_inputs(cfg, 1)
    kv = wl.make_kv(cfg, 1, st["ctx_len"])
    ly = cfg.layer
    for i in range(cfg.B):
        L, c, base = int(st["ctx_len"][i]), int(kv["cap"][i]), int(kv["base"][i])
        slab = kv["k"][base: base + ly.n_kv * c * ly.head_dim].reshape(ly.n_kv, c, ly.head_dim)
        assert np.array_equal(slab[:, :L], wl.make_kv_request(cfg, 1, i, L, "k"))
        assert not slab[:, L:].any()
        assert c == L + cfg.D + 1


def test_weights_stats():
    cfg = wl.CONFIGS[1]
    w = wl.make_weights(cfg, 0)
    x = wl.bf16_to_f32(w["w_qkv"])
    assert abs(x.std() - 0.02) < 1e-3 and abs(x.mean()) < 1e-3
    assert (w["attn_norm"] == 0x3F80).all()
    assert w["w_gate_up"].shape == (2 * 688, 256) and w["w_down"].shape == (256, 688)
