// dcut_verify_layer: one pre-norm decoder layer over the packed kept rows (App. C).
//
// Launch sequence on the caller's stream (all grids sized for B(D+1) rows, the
// live row count K* = cu[B] is read on the device):
//   norm1    x -> x_out (float32 residual), h = RMSNorm(x) (bf16), RoPE table
//   QKV      h W_qkv^T, RoPE on q/k in the epilogue, q -> scratch, k/v -> cache
//   attn     ragged split-KV GQA attention (+ chunk merge) -> attn (bf16)
//   O        x_out += attn W_o^T
//   norm2    h = RMSNorm(x_out)
//   MLP      dense: mid = SiLU(h W_g^T) * (h W_u^T) (one GEMM, fused epilogue);
//                   x_out += mid W_down^T
//            MoE:   router, top-k, expert grouping, grouped SwiGLU GEMMs, combine
#include "dcut_internal.h"

namespace dcut {

// Split-KV chunk length (cache keys per attention work item): 1024 keys when the
// batch still gives at least 2048 work items, else 512.  A function of the
// shapes only (B, n_kv, max_ctx), never of the kept rows, so a row's partial
// sums never depend on the budget.
static int attn_chunk(const dcut_layer_cfg *c, int B) {
  const long long items = (long long)B * c->n_kv * ((c->max_ctx + 1023) / 1024);
  return items >= 2048 ? 1024 : 512;
}

struct LayerWs {
  size_t h, q, attn, rope, part, plan, mid, split, moe, total;
  int split_qkv, split_o, split_down;
};

static bool layer_cfg_ok(const dcut_layer_cfg *c, int B, int D) {
  if (!c || !batch_ok(B, D)) return false;
  if (c->hidden <= 0 || c->hidden % 8 || c->n_q <= 0 || c->n_kv <= 0 || c->n_q % c->n_kv) return false;
  if (c->head_dim <= 0 || c->vocab <= 0 || c->max_ctx < D + 1) return false;
  if (c->n_exp < 0) return false;
  if (c->n_exp == 0 && (c->inter <= 0 || c->inter % 8)) return false;
  if (c->n_exp > 0 && (c->top_k <= 0 || c->top_k > c->n_exp || c->exp_inter <= 0 || c->exp_inter % 8))
    return false;
  if (!(c->rms_eps >= 0.0f) || !(c->rope_theta > 0.0f)) return false;
  return true;
}

static bool layer_cfg_supported(const dcut_layer_cfg *c, int B, int D) {
  if (c->head_dim != 64 && c->head_dim != 128) return false;
  if ((c->n_q / c->n_kv) * (D + 1) > 256) return false;
  if (c->n_exp > 0 && !moe_supported(B * (D + 1), c->hidden, c->n_exp, c->top_k)) return false;
  // 32-bit buffer offsets: one request's key (or value) slab, and each GEMM's spans
  if ((long long)c->max_ctx * c->head_dim * 2 >= 0x7fffffffLL) return false;
  const long long H = c->hidden, QD = (long long)c->n_q * c->head_dim;
  if (!gemm_span_ok(256, H, 256, H) || !gemm_span_ok(256, QD, 256, QD)) return false;
  if (c->n_exp == 0 && (!gemm_span_ok(256, H, c->inter + 256LL, H) || !gemm_span_ok(256, c->inter, 256, c->inter)))
    return false;
  if (c->n_exp > 0 && (!gemm_span_ok((long long)B * (D + 1), H, c->exp_inter + 256LL, H) ||
                       !gemm_span_ok(256, c->exp_inter, 256, c->exp_inter)))
    return false;
  return true;
}

static LayerWs layer_ws(const dcut_layer_cfg *c, int B, int D) {
  LayerWs w;
  const size_t M = (size_t)B * (D + 1);
  const size_t qd = (size_t)c->n_q * c->head_dim;
  const int chunk = attn_chunk(c, B);
  const int mc = (c->max_ctx + chunk - 1) / chunk;
  size_t off = 0;
  w.h = off; off = align256(off + M * c->hidden * 2);
  w.q = off; off = align256(off + M * qd * 2);
  w.attn = off; off = align256(off + M * qd * 2);
  w.rope = off; off = align256(off + M * (c->head_dim / 2) * sizeof(float2));
  w.part = off; off = align256(off + M * c->n_q * (size_t)mc * (c->head_dim + 2) * sizeof(float));
  w.plan = off; off = align256(off + attn_plan_bytes(B, c->n_kv, mc));
  w.mid = off; off = align256(off + (c->n_exp == 0 ? M * (size_t)c->inter * 2 : 0));
  const size_t nqkv = (size_t)(c->n_q + 2 * c->n_kv) * c->head_dim;
  w.split_qkv = gemm_splits((int)M, (int)nqkv, c->hidden);
  w.split_o = gemm_splits((int)M, c->hidden, (int)qd);
  w.split_down = c->n_exp == 0 ? gemm_splits((int)M, c->hidden, c->inter) : 1;
  size_t split_floats = 0;   // per row, the largest of the three split-K partial sets
  if (w.split_qkv > 1) split_floats = (size_t)w.split_qkv * nqkv;
  if (w.split_o > 1 && (size_t)w.split_o * c->hidden > split_floats) split_floats = (size_t)w.split_o * c->hidden;
  if (w.split_down > 1 && (size_t)w.split_down * c->hidden > split_floats)
    split_floats = (size_t)w.split_down * c->hidden;
  w.split = off; off = align256(off + M * split_floats * sizeof(float));
  w.moe = off;
  if (c->n_exp > 0) off = align256(off + moe_ws_bytes((int)M, c->hidden, c->n_exp, c->top_k, c->exp_inter));
  w.total = off;
  return w;
}

size_t layer_ws_bytes(const dcut_layer_cfg *c, int B, int D) {
  if (!layer_cfg_ok(c, B, D)) return (size_t)-1;
  return layer_ws(c, B, D).total;
}

}  // namespace dcut

using namespace dcut;

extern "C" int dcut_verify_layer(const dcut_layer_cfg *cfg, const dcut_layer_w *w, int B, int D,
                                 const int32_t *cu, const int32_t *packed_tok,
                                 const int32_t *packed_pos, const int32_t *packed_req,
                                 const int32_t *ctx_len, const float *x_in, const dcut_kv *kv,
                                 float *x_out, int32_t *dev_err, void *ws, size_t ws_bytes,
                                 hipStream_t stream) {
  if (!layer_cfg_ok(cfg, B, D) || !w || !kv) return DCUT_EINVAL;
  if (!cu || !packed_tok || !packed_pos || !packed_req || !ctx_len || !x_out) return DCUT_EINVAL;
  if (!kv->k || !kv->v || !kv->base || !kv->cap) return DCUT_EINVAL;
  if (!w->attn_norm || !w->w_qkv || !w->w_o || !w->mlp_norm) return DCUT_EINVAL;
  if (!x_in && !w->embed) return DCUT_EINVAL;
  if (cfg->n_exp == 0 && (!w->w_gate_up || !w->w_down)) return DCUT_EINVAL;
  if (cfg->n_exp > 0 && (!w->w_router || !w->w_exp_gate_up || !w->w_exp_down)) return DCUT_EINVAL;
  if (!layer_cfg_supported(cfg, B, D)) return DCUT_EUNSUPPORTED;
  const LayerWs L = layer_ws(cfg, B, D);
  if (!ws || ws_bytes < L.total || ((uintptr_t)ws & 255)) return DCUT_EWORKSPACE;

  char *base = (char *)ws;
  uint16_t *h = (uint16_t *)(base + L.h);
  uint16_t *q = (uint16_t *)(base + L.q);
  uint16_t *att = (uint16_t *)(base + L.attn);
  float2 *rope = (float2 *)(base + L.rope);
  float *part = (float *)(base + L.part);
  uint16_t *mid = (uint16_t *)(base + L.mid);
  float *split = (float *)(base + L.split);

  const int H = cfg->hidden, hd = cfg->head_dim, nq = cfg->n_q, nkv = cfg->n_kv;
  const int M = B * (D + 1);
  const int32_t *Kstar = cu + B;

  // attention arguments (the work order is built by norm1)
  AttnArgs at = {};
  at.q = q; at.kv_k = kv->k; at.kv_v = kv->v; at.kv_base = kv->base; at.kv_cap = kv->cap;
  at.cu = cu; at.ctx_len = ctx_len; at.B = B; at.D = D; at.n_q = nq; at.n_kv = nkv; at.head_dim = hd;
  at.chunk = attn_chunk(cfg, B); at.max_chunks = (cfg->max_ctx + at.chunk - 1) / at.chunk;
  at.part = part; at.out = att; at.dev_err = dev_err;
  at.plan = attn_plan_bytes(B, nkv, at.max_chunks) ? (int32_t *)(base + L.plan) : nullptr;

  // 1. norm1 (+ embedding gather, residual copy, RoPE table, attention work order)
  DCUT_TRY(rmsnorm_launch(DCUT_KERNEL_NORM, x_in, w->embed, packed_tok, cfg->vocab, w->attn_norm,
                          cfg->rms_eps, H, M, Kstar, x_out, h, packed_pos, hd, cfg->rope_theta,
                          rope, nullptr, dev_err, &at, stream));
  // 2. QKV + RoPE + cache append
  GemmArgs g = {};
  g.A = h; g.lda = H; g.K = H; g.M_max = M; g.m_count = Kstar;
  g.W = w->w_qkv; g.ldw = H; g.N = (nq + 2 * nkv) * hd;
  g.out_bf16 = q; g.ldo = nq * hd;
  g.packed_pos = packed_pos; g.packed_req = packed_req; g.ctx_len = ctx_len; g.rope_cs = rope;
  g.kv_k = kv->k; g.kv_v = kv->v; g.kv_base = kv->base; g.kv_cap = kv->cap;
  g.n_q = nq; g.n_kv = nkv; g.head_dim = hd; g.n_req = B;
  g.splits = L.split_qkv; g.split_part = split;
  DCUT_TRY(gemm_launch(DCUT_KERNEL_GEMM_QKV, EPI_QKV_ROPE, g, stream));
  // 3. attention
  const int waves = ((nq / nkv) * (D + 1) + 15) / 16;
  DCUT_TRY(attention_launch(at, M, packed_req, waves, stream));
  // 4. O projection + residual
  GemmArgs o = {};
  o.A = att; o.lda = nq * hd; o.K = nq * hd; o.M_max = M; o.m_count = Kstar;
  o.W = w->w_o; o.ldw = nq * hd; o.N = H;
  o.out_f32 = x_out; o.ldo = H;
  o.splits = L.split_o; o.split_part = split;
  // 5. norm2; with split-K, the residual add of the O projection is fused into it
  const bool fuse = L.split_o > 1 && H <= 8192;
  o.defer_reduce = fuse ? 1 : 0;
  DCUT_TRY(gemm_launch(DCUT_KERNEL_GEMM_O, EPI_RESID_F32, o, stream));
  if (fuse)
    DCUT_TRY(reduce_rmsnorm_launch(DCUT_KERNEL_NORM, split, L.split_o, M, H, Kstar, x_out, w->mlp_norm,
                                   cfg->rms_eps, h, stream));
  else
    DCUT_TRY(rmsnorm_launch(DCUT_KERNEL_NORM, x_out, nullptr, nullptr, 0, w->mlp_norm, cfg->rms_eps, H,
                            M, Kstar, nullptr, h, nullptr, 0, 0.0f, nullptr, nullptr, dev_err, nullptr,
                            stream));
  // 6. MLP
  if (cfg->n_exp > 0) {
    MoeArgs me = {};
    me.h = h; me.w_router = w->w_router; me.w_gate_up = w->w_exp_gate_up; me.w_down = w->w_exp_down;
    me.H = H; me.E = cfg->n_exp; me.top_k = cfg->top_k; me.inter = cfg->exp_inter; me.M_max = M;
    me.m_count = Kstar; me.x_out = x_out; me.ws = base + L.moe;
    return moe_launch(me, stream);
  }
  GemmArgs gu = {};
  gu.A = h; gu.lda = H; gu.K = H; gu.M_max = M; gu.m_count = Kstar;
  gu.W = w->w_gate_up; gu.ldw = H; gu.N = 2 * cfg->inter; gu.swiglu_inter = cfg->inter;
  gu.out_bf16 = mid; gu.ldo = cfg->inter;
  DCUT_TRY(gemm_launch(DCUT_KERNEL_GEMM_GATE_UP, EPI_SWIGLU, gu, stream));
  GemmArgs dn = {};
  dn.A = mid; dn.lda = cfg->inter; dn.K = cfg->inter; dn.M_max = M; dn.m_count = Kstar;
  dn.W = w->w_down; dn.ldw = cfg->inter; dn.N = H;
  dn.out_f32 = x_out; dn.ldo = H;
  dn.splits = L.split_down; dn.split_part = split;
  DCUT_TRY(gemm_launch(DCUT_KERNEL_GEMM_DOWN, EPI_RESID_F32, dn, stream));
  return DCUT_OK;
}
