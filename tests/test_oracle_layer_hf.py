"""The oracle's composed decoder layer pinned to an independent implementation.

`oracle.layer.verify_layer` composes one pre-norm decoder layer around the
rule of App. C that every kept position is scored against its request's
accepted prefix (the cached context plus its own block up to itself).  The
paper names Llama- and Qwen-family targets but prints no worked forward, so
the composition (norm placement, residual adds, the q/k/v split and GQA head
groups, RoPE pairs, causal masking over cache plus block, the gate/up order
of SwiGLU, routed-MoE weighting) is pinned here to the Hugging Face
`transformers` implementation of the same layer:

  dense: `LlamaDecoderLayer` with eager attention, a `DynamicCache` prefilled
         with the request's cached (post-RoPE) keys and values, position ids
         L_i + k and an additive causal mask over cache plus block;
  MoE:   the same attention half with `Qwen3MoeSparseMoeBlock` as the MLP
         (softmax router, top-k, renormalised weights; expert weights in the
         library's [E][2 Ie][H] gate-then-up and [E][H][Ie] layouts);
  head:  `LlamaRMSNorm` and a matmul against the oracle's logits.

Both run in float64 on the same bf16-exact weights and cache (the library
takes its norms and softmaxes in float32, which bounds the agreement near
1e-7).  The cos/sin tables are formed in float64 from the library's default
RoPE rule and checked against its own float32 rotary embedding first.
Mutations planted in the oracle's source (on the CPU) must fail the same
comparison, so a dropped residual, swapped SwiGLU halves, a missing norm, a
wrong head group, a non-causal block or unnormalised routing cannot pass.
"""
import types

import numpy as np
import pytest
import torch

pytest.importorskip("transformers")
from transformers import LlamaConfig  # noqa: E402
from transformers.cache_utils import DynamicCache  # noqa: E402
from transformers.models.llama.modeling_llama import (  # noqa: E402
    LlamaDecoderLayer, LlamaRMSNorm, LlamaRotaryEmbedding)
from transformers.models.qwen3_moe.configuration_qwen3_moe import Qwen3MoeConfig  # noqa: E402
from transformers.models.qwen3_moe.modeling_qwen3_moe import Qwen3MoeSparseMoeBlock  # noqa: E402

import oracle.layer as olay  # noqa: E402
from oracle import lm_head as olm  # noqa: E402
from oracle import select as osel  # noqa: E402
from tests.gpu_common import tiny_variants  # noqa: E402
from paper_2607_14647_amd import workload as wl  # noqa: E402

TOL = 1e-6          # row-relative agreement of the oracle and the library
MUT_MIN = 1e-3      # a planted mistake must move some row by at least this much
ROUTER_MIN_GAP = 1e-5   # MoE rows whose k-th / (k+1)-th router logits are closer are not compared

VARIANTS = tiny_variants()
CASES = ["cfg1", "moe", "moe128", "split"]


def _llama_config(ly):
    c = LlamaConfig(hidden_size=ly.hidden, intermediate_size=max(ly.inter, 8), num_attention_heads=ly.n_q,
                    num_key_value_heads=ly.n_kv, head_dim=ly.head_dim, rms_norm_eps=ly.rms_eps,
                    vocab_size=ly.vocab, rope_theta=ly.rope_theta, attention_bias=False, mlp_bias=False,
                    hidden_act="silu")
    c._attn_implementation = "eager"
    return c


def _t(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float64))


def _rope_tables(ly, pos):
    """cos/sin [1][d][hd] in float64 by the library's default rule: inverse frequencies
    1 / theta^(2j/hd), angles pos * inv_freq, the table repeated over both halves."""
    hd = ly.head_dim
    inv = 1.0 / (ly.rope_theta ** (torch.arange(0, hd, 2, dtype=torch.float64) / hd))
    ang = torch.as_tensor(pos, dtype=torch.float64)[:, None] * inv[None, :]
    emb = torch.cat([ang, ang], dim=-1)[None]
    return emb.cos(), emb.sin()


def _hf_layer(cfg, w64):
    ly = cfg.layer
    H, nq, nkv, hd = ly.hidden, ly.n_q, ly.n_kv, ly.head_dim
    layer = LlamaDecoderLayer(_llama_config(ly), layer_idx=0).to(torch.float64).eval()
    q_end, k_end = nq * hd, (nq + nkv) * hd
    with torch.no_grad():
        layer.input_layernorm.weight.copy_(_t(w64["attn_norm"]))
        layer.post_attention_layernorm.weight.copy_(_t(w64["mlp_norm"]))
        layer.self_attn.q_proj.weight.copy_(_t(w64["w_qkv"][:q_end]))
        layer.self_attn.k_proj.weight.copy_(_t(w64["w_qkv"][q_end:k_end]))
        layer.self_attn.v_proj.weight.copy_(_t(w64["w_qkv"][k_end:]))
        layer.self_attn.o_proj.weight.copy_(_t(w64["w_o"]))
        if ly.n_exp == 0:
            I = ly.inter
            layer.mlp.gate_proj.weight.copy_(_t(w64["w_gate_up"][:I]))
            layer.mlp.up_proj.weight.copy_(_t(w64["w_gate_up"][I:]))
            layer.mlp.down_proj.weight.copy_(_t(w64["w_down"]))
        else:
            qc = Qwen3MoeConfig(hidden_size=H, num_experts=ly.n_exp, num_experts_per_tok=ly.top_k,
                                moe_intermediate_size=ly.exp_inter, norm_topk_prob=True, hidden_act="silu")
            moe = Qwen3MoeSparseMoeBlock(qc).to(torch.float64).eval()
            moe.gate.weight.copy_(_t(w64["w_router"]))
            moe.experts.gate_up_proj.copy_(_t(w64["w_exp_gate_up"]))
            moe.experts.down_proj.copy_(_t(w64["w_exp_down"]))
            layer.mlp = moe
    return layer


def _hf_request(layer, cfg, w64, kv, sel, ctx_len, i):
    """Library forward of request i's kept rows: (x_out [d][H], appended k, v [d][n_kv][hd])."""
    ly = cfg.layer
    nkv, hd = ly.n_kv, ly.head_dim
    t0, t1 = int(sel["cu"][i]), int(sel["cu"][i + 1])
    d, L, cap, base = t1 - t0, int(ctx_len[i]), int(kv["cap"][i]), int(kv["base"][i])
    x = olay.bf16_bits_to_f64(w64["embed"][sel["packed_tok"][t0:t1]])
    slab = nkv * cap * hd
    ck = olay.bf16_bits_to_f64(kv["k"][base:base + slab]).reshape(nkv, cap, hd)[:, :L]
    cv = olay.bf16_bits_to_f64(kv["v"][base:base + slab]).reshape(nkv, cap, hd)[:, :L]
    cache = DynamicCache()
    cache.update(_t(ck)[None], _t(cv)[None], 0)
    pos = np.asarray(sel["packed_pos"][t0:t1], dtype=np.int64)
    assert np.array_equal(pos, L + np.arange(d))
    mask = torch.full((1, 1, d, L + d), float("-inf"), dtype=torch.float64)
    for r in range(d):
        mask[0, 0, r, : L + r + 1] = 0.0
    with torch.no_grad():
        out = layer(_t(x)[None], attention_mask=mask, position_ids=torch.from_numpy(pos)[None],
                    past_key_values=cache, use_cache=True, position_embeddings=_rope_tables(ly, pos))
    keys = cache.layers[0].keys[0, :, L:].permute(1, 0, 2).numpy()
    vals = cache.layers[0].values[0, :, L:].permute(1, 0, 2).numpy()
    return out[0].numpy(), keys, vals


def _rel(got, ref):
    got = got.reshape(got.shape[0], -1)
    ref = ref.reshape(ref.shape[0], -1)
    return np.abs(got - ref).max(axis=1) / np.maximum(np.abs(ref).max(axis=1), 1e-300)


def _case(name):
    cfg = VARIANTS[name]
    st = wl.make_step_inputs(cfg, 0)
    w = wl.make_weights(cfg, 0)
    kv = wl.make_kv(cfg, 0, st["ctx_len"])
    sel = osel.select(st["conf"], st["draft"], st["ctx_len"], list(cfg.budgets), [1.0] * len(cfg.budgets))
    return cfg, st, olay.prepare_weights(w), kv, sel


def _compare(verify, cfg, st, w64, kv, sel):
    """Largest row-relative difference between `verify` (the oracle's verify_layer or a mutant)
    and the library over every kept row of every request (x_out, appended k and v)."""
    ly = cfg.layer
    ref = verify(ly, w64, kv, sel["cu"], sel["packed_tok"], sel["packed_pos"], sel["packed_req"], st["ctx_len"],
                 cfg.D)
    layer = _hf_layer(cfg, w64)
    worst = dict(x=0.0, k=0.0, v=0.0)
    skipped = 0
    for i in range(cfg.B):
        t0, t1 = int(sel["cu"][i]), int(sel["cu"][i + 1])
        x_hf, k_hf, v_hf = _hf_request(layer, cfg, w64, kv, sel, st["ctx_len"], i)
        keep = np.ones(t1 - t0, bool)
        if ly.n_exp > 0:
            keep = ref["router_gap"][t0:t1] > ROUTER_MIN_GAP
            skipped += int((~keep).sum())
        worst["x"] = max(worst["x"], _rel(ref["x_out"][t0:t1][keep], x_hf[keep]).max(initial=0.0))
        worst["k"] = max(worst["k"], _rel(ref["new_k"][t0:t1], k_hf).max())
        worst["v"] = max(worst["v"], _rel(ref["new_v"][t0:t1], v_hf).max())
    assert skipped <= int(sel["cu"][-1]) // 10, "too many near-tied router rows"
    return worst, ref


def test_rope_tables_match_library_rotary():
    """The float64 cos/sin tables follow the library's own rotary embedding (float32) to its
    rounding, at the largest positions the variants use."""
    for name in CASES:
        ly = VARIANTS[name].layer
        pos = np.array([0, 1, 77, 2100], dtype=np.int64)
        rot = LlamaRotaryEmbedding(_llama_config(ly))
        cos32, sin32 = rot(torch.zeros(1, dtype=torch.float32), torch.from_numpy(pos)[None])
        cos64, sin64 = _rope_tables(ly, pos)
        # float32 angles at position p carry about p * 2^-24 of absolute error
        bound = 4 * 2100 * 2.0 ** -24
        assert float((cos32.double() - cos64).abs().max()) < bound
        assert float((sin32.double() - sin64).abs().max()) < bound


@pytest.mark.parametrize("name", CASES)
def test_layer_matches_library(name):
    cfg, st, w64, kv, sel = _case(name)
    worst, ref = _compare(olay.verify_layer, cfg, st, w64, kv, sel)
    print(f"{name}: max row-relative difference x_out {worst['x']:.2e}, k {worst['k']:.2e}, v {worst['v']:.2e}")
    assert worst["x"] <= TOL and worst["k"] <= TOL and worst["v"] <= TOL


@pytest.mark.parametrize("name", ["cfg1", "split"])
def test_lm_head_matches_library(name):
    """Final RMSNorm and LM head: the oracle's logits against LlamaRMSNorm and a matmul."""
    cfg, st, w64, kv, sel = _case(name)
    ly = cfg.layer
    rng = np.random.default_rng(7)
    x = rng.standard_normal((24, ly.hidden)) * 0.3
    ref = olm.lm_head_argmax(x, w64["final_norm"], ly.rms_eps, w64["w_lm"])
    norm = LlamaRMSNorm(ly.hidden, eps=ly.rms_eps).to(torch.float64)
    with torch.no_grad():
        norm.weight.copy_(_t(w64["final_norm"]))
        logits = (norm(_t(x)) @ _t(w64["w_lm"]).T).numpy()
    assert _rel(ref["logits"], logits).max() <= TOL
    assert np.array_equal(ref["argmax"], np.argmax(logits, axis=1))


def _mutant(old: str, new: str):
    """A copy of oracle.layer with one source edit (the edit must apply exactly once)."""
    src = open(olay.__file__).read()
    assert src.count(old) == 1, f"mutation site not found once: {old!r}"
    mod = types.ModuleType("oracle.layer_mutant")
    mod.__package__ = "oracle"
    exec(compile(src.replace(old, new), olay.__file__ + " (mutant)", "exec"), mod.__dict__)
    return mod.verify_layer


MUTATIONS = {
    "drop attention residual": ("cfg1", 'y = x + _mm(att, w64["w_o"], row_exact)', 'y = _mm(att, w64["w_o"], row_exact)'),
    "drop MLP residual": ("cfg1", 'out = y + _mm(m, w64["w_down"], row_exact)', 'out = _mm(m, w64["w_down"], row_exact)'),
    "swap gate and up": ("cfg1", "m = act(silu(gu[:, : ly.inter]) * gu[:, ly.inter:])",
                         "m = act(silu(gu[:, ly.inter:]) * gu[:, : ly.inter])"),
    "no pre-attention norm": ("cfg1", 'h = act(rmsnorm(x, w64["attn_norm"], ly.rms_eps))', "h = act(x)"),
    "post-norm residual": ("cfg1", 'h2 = act(rmsnorm(y, w64["mlp_norm"], ly.rms_eps))',
                           'y = rmsnorm(y, w64["mlp_norm"], ly.rms_eps); h2 = act(y)'),
    "interleaved head groups": ("cfg1", "g = h // grp", "g = h % nkv"),
    "block not causal": ("cfg1", "n = L + r + 1", "n = L + d"),
    "MoE weights not renormalised": ("moe", "w = pt / pt.sum(axis=-1, keepdims=True)", "w = pt"),
}


@pytest.mark.parametrize("what", list(MUTATIONS))
def test_planted_mistake_fails(what):
    name, old, new = MUTATIONS[what]
    cfg, st, w64, kv, sel = _case(name)
    worst, _ = _compare(_mutant(old, new), cfg, st, w64, kv, sel)
    print(f"{what}: max row-relative difference {max(worst.values()):.2e}")
    assert max(worst.values()) > MUT_MIN
