"""Device-resident verify step: uploads a workload once and runs the library calls.

Holds every buffer the C ABI needs (weights, KV cache, step inputs, outputs,
workspaces) as torch device tensors and calls the library on torch's current
stream.  No computation happens here.
"""
from __future__ import annotations

from typing import Dict, Optional, Sequence

import numpy as np
import torch

from . import lib as L
from . import workload as wl


def _dev(a: np.ndarray, device) -> torch.Tensor:
    if a.dtype == np.uint16:
        a = a.view(np.int16)
    return torch.from_numpy(np.ascontiguousarray(a)).to(device)


class VerifyStep:
    def __init__(self, cfg: wl.Config, weights: Dict[str, np.ndarray], step: Dict[str, np.ndarray],
                 kv: Dict[str, np.ndarray], device: str = "cuda", R_max: int = 64,
                 share_weights: Optional["VerifyStep"] = None):
        self.cfg = cfg
        self.B, self.D = cfg.B, cfg.D
        self.rows = cfg.B * (cfg.D + 1)
        ly = cfg.layer
        self.ly = ly
        self.device = device
        if share_weights is not None:          # another batch size of the same model
            assert share_weights.ly == ly
            self.w = share_weights.w
        else:
            self.w = {k: _dev(v, device) for k, v in weights.items()}
        self.lw = L.layer_weights(self.w)
        self.conf = _dev(step["conf"], device)
        self.draft = _dev(step["draft"], device)
        self.ctx_len = _dev(step["ctx_len"], device)
        self.kv = {k: _dev(v, device) for k, v in kv.items()}
        self.kvd = L.kv_desc(self.kv)
        self.extra = []             # decoder layers after the first: (weights, descriptor, kv, kv descriptor)
        self.lcfg = L.layer_cfg(ly, int(kv["cap"].max()))
        self.sel = L.select_outputs(self.B, self.D, R_max, device)
        i32 = dict(dtype=torch.int32, device=device)
        self.dev_err = torch.zeros(1, **i32)
        self.x = torch.zeros(self.rows, ly.hidden, dtype=torch.float32, device=device)
        self.argmax = torch.zeros(self.rows, **i32)
        self.max_logit = torch.zeros(self.rows, dtype=torch.float32, device=device)
        self.accept_len = torch.zeros(self.B, **i32)
        self.next_tok = torch.zeros(self.B, **i32)
        self.total = torch.zeros(1, **i32)
        self.ws_layer = L.workspace(L.workspace_bytes(1, self.lcfg, self.B, self.D), device)
        self.ws_lm = L.workspace(L.workspace_bytes(2, self.lcfg, self.B, self.D), device)
        self.temperature = 0.0      # > 0: temperature sampling instead of the greedy argmax
        self.seed = 0
        self.q = None               # proposal distributions [B][D][V]: rejection-sampling verification
        self.rs_mode = L.RS_SCAN    # budget choice of step_rs with several candidates
        self.k_state = torch.zeros(1, **i32)   # history-based budget carried between steps

    def enable_rs(self, q) -> None:
        """Switch to rejection-sampling verification with proposal distributions q [B][D][V]
        (numpy or device tensor; None allocates zeros to fill later): the LM head then also
        writes logits and log-partition values."""
        V = self.ly.vocab
        if q is None:
            q = torch.zeros(self.B, self.D, V, dtype=torch.float32, device=self.device)
        self.q = q if isinstance(q, torch.Tensor) else _dev(np.asarray(q, dtype=np.float32), self.device)
        assert tuple(self.q.shape) == (self.B, self.D, V) and self.q.dtype == torch.float32
        self.logits = torch.empty(self.rows, V, dtype=torch.float32, device=self.device)
        self.lse = torch.empty(self.rows, dtype=torch.float32, device=self.device)
        self.ws_rs = L.workspace(L.workspace_bytes(4, self.lcfg, self.B, self.D), self.device)

    def set_draft(self, draft: np.ndarray) -> None:
        self.draft.copy_(torch.from_numpy(np.ascontiguousarray(draft, dtype=np.int32)))

    def set_conf(self, conf: np.ndarray) -> None:
        self.conf.copy_(torch.from_numpy(np.ascontiguousarray(conf, dtype=np.float32)))

    def select(self, budgets: Sequence[int], costs: Sequence[float]) -> None:
        L.select(self.B, self.D, self.conf, self.draft, self.ctx_len, budgets, costs, self.sel,
                 self.dev_err)

    def select_rs(self, mode: int, budgets: Sequence[int], costs: Sequence[float]) -> None:
        L.select_rs(self.B, self.D, self.conf, self.draft, self.ctx_len, mode, budgets, costs, self.sel,
                    self.dev_err, k_state=self.k_state)

    def add_layer(self, weights: Dict[str, np.ndarray], kv: Dict[str, np.ndarray]) -> None:
        """Append a decoder layer (its weights and KV cache) after the first: the
        verify pass then runs every layer in order on the residual stream."""
        w = {k: _dev(v, self.device) for k, v in weights.items()}
        kvt = {k: _dev(v, self.device) for k, v in kv.items()}
        self.extra.append((w, L.layer_weights(w), kvt, L.kv_desc(kvt)))

    def verify(self, x_in: Optional[torch.Tensor] = None) -> None:
        L.verify_layer(self.lcfg, self.lw, self.B, self.D, self.sel, self.ctx_len, self.kvd, self.x,
                       self.ws_layer, x_in=x_in, dev_err=self.dev_err)
        for _, lw, _, kvd in self.extra:
            L.verify_layer(self.lcfg, lw, self.B, self.D, self.sel, self.ctx_len, kvd, self.x,
                           self.ws_layer, x_in=self.x, dev_err=self.dev_err)

    def lm_head(self, logits: Optional[torch.Tensor] = None) -> None:
        """Target token of every kept row into `argmax`: the greedy argmax, or a
        temperature-T draw when `self.temperature` > 0 (seeded by `self.seed`)."""
        if self.temperature > 0.0:
            L.lm_head_sample(self.ly.hidden, self.ly.vocab, self.B, self.D, self.sel["cu"],
                             self.sel["packed_req"], self.sel["packed_pos"], self.x, self.w["final_norm"],
                             self.ly.rms_eps, self.w["w_lm"], self.temperature, self.seed, self.argmax,
                             self.ws_lm, max_score=self.max_logit,
                             logits=self.logits if self.q is not None else logits,
                             lse=self.lse if self.q is not None else None)
            return
        L.lm_head_argmax(self.ly.hidden, self.ly.vocab, self.B, self.D, self.sel["cu"], self.x,
                         self.w["final_norm"], self.ly.rms_eps, self.w["w_lm"], self.argmax,
                         self.ws_lm, max_logit=self.max_logit, logits=logits)

    def accept(self, ctx_inout: Optional[torch.Tensor] = None) -> None:
        L.accept(self.B, self.D, self.draft, self.sel["keep_len"], self.sel["cu"], self.argmax,
                 self.accept_len, self.next_tok, self.total, ctx_inout)

    def accept_rs(self, ctx_inout: Optional[torch.Tensor] = None) -> None:
        L.accept_rs(self.B, self.D, self.ly.vocab, self.temperature, self.seed, self.draft, self.q,
                    self.sel["keep_len"], self.sel["cu"], self.sel["packed_pos"], self.logits, self.lse,
                    self.argmax, self.accept_len, self.next_tok, self.total, self.ws_rs, ctx_inout,
                    self.dev_err)

    def step(self, budgets: Sequence[int], costs: Sequence[float]) -> None:
        self.select(budgets, costs)
        self.verify()
        self.lm_head()
        self.accept()

    def step_rs(self, budgets: Sequence[int], costs: Sequence[float]) -> None:
        """One rejection-sampling step: `rs_mode` over the candidates (the causal
        scan or the history-based budget), or the fixed budget when only one is given."""
        self.select_rs(L.RS_FIXED if len(budgets) == 1 else self.rs_mode, budgets, costs)
        self.verify()
        self.lm_head()
        self.accept_rs()

    def capture(self, fn) -> "torch.cuda.CUDAGraph":
        """Capture the library calls `fn` makes into one HIP graph (stream capture
        through torch.cuda.graph on a default-priority side stream); replay it
        with .replay().  The calls take every size from the host and K* from the
        device, so one graph per batch size serves every budget the step picks."""
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):          # one eager pass first (kernel attributes, caches)
            fn()
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            fn()
        torch.cuda.synchronize()
        return g

    def host(self, name: str) -> np.ndarray:
        src = self.sel[name] if name in self.sel else getattr(self, name)
        return src.cpu().numpy()


def force_drafts_on_device(st: VerifyStep, draft: np.ndarray, conf: np.ndarray,
                           match_u: np.ndarray) -> np.ndarray:
    """Synthetic drafter for benchmarks: z_{i,k} := the library's own greedy token at
    position k-1 when match_u < conf (depth order, full budget each pass).

    The target's greedy token at block position k-1 depends only on z_{i,0..k-1},
    so after D passes every forced depth agrees with the verify step's argmax."""
    B, D = st.B, st.D
    z = np.array(draft, dtype=np.int32, copy=True)
    full = [B * (D + 1)]
    for k in range(1, D + 1):
        st.set_draft(z)
        st.select(full, [1.0])
        st.verify()
        st.lm_head()
        g = st.argmax.cpu().numpy().reshape(B, D + 1)
        hit = match_u[:, k - 1] < conf[:, k - 1]
        z[hit, k] = g[hit, k - 1]
    st.set_draft(z)
    return z


def force_drafts_rs_on_device(st: VerifyStep, draft: np.ndarray, conf: np.ndarray, match_u: np.ndarray,
                              seed: int) -> np.ndarray:
    """Synthetic stochastic drafter for benchmarks of rejection-sampling verification.

    At depth k the proposal is q_{i,k} = c p + (1 - c) delta_w: the target's own
    distribution p at block position k-1 (the verify step's logits at the
    drafting seed's temperature), mixed with a point mass on an unrelated token
    w = draft[i][k]; c = conf[i][k-1].  The draft is the target's own draw
    at that row when match_u < c and w otherwise, a draw from q_{i,k}.  RS
    then accepts it with probability about c, as the greedy drafter's drafts
    survive with probability c.  Depth order, full budget each pass; the
    proposals land in st.q (enable_rs first).  Returns the drafts."""
    B, D, V = st.B, st.D, st.ly.vocab
    z = np.array(draft, dtype=np.int32, copy=True)
    full = [B * (D + 1)]
    keep_seed = st.seed
    st.seed = seed
    rows = torch.arange(B, device=st.device) * (D + 1)
    c = torch.from_numpy(np.ascontiguousarray(conf, dtype=np.float32)).to(st.device)
    w = torch.from_numpy(np.ascontiguousarray(draft[:, 1:], dtype=np.int64)).to(st.device)
    for k in range(1, D + 1):
        st.set_draft(z)
        st.select(full, [1.0])
        st.verify()
        st.lm_head()
        r = rows + (k - 1)
        p = torch.exp(st.logits[r] * (1.0 / st.temperature) - st.lse[r][:, None])
        ck = c[:, k - 1]
        qk = p * ck[:, None]
        qk[torch.arange(B, device=st.device), w[:, k - 1]] += 1.0 - ck
        st.q[:, k - 1].copy_(qk)
        g = st.argmax.cpu().numpy().reshape(B, D + 1)
        hit = match_u[:, k - 1] < conf[:, k - 1]
        z[hit, k] = g[hit, k - 1]
    st.set_draft(z)
    st.seed = keep_seed
    torch.cuda.synchronize()
    return z
