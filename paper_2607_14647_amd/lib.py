"""ctypes binding of libdcut.so (argument marshalling only).

Every function takes torch tensors that already live on the GPU and passes
their device pointers, sizes and torch's current HIP stream to the C ABI in
include/dcut.h.  Nothing here computes: if the library is missing, importing
the binding fails with an error that says how to build it.
"""
from __future__ import annotations

import ctypes as C
import os
from typing import Dict, Optional, Sequence

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libdcut.so")

OK, EINVAL, EUNSUPPORTED, EWORKSPACE, EHIP = 0, -1, -2, -3, -4
DERR_CONF, DERR_TOKEN, DERR_CAPACITY = 1, 2, 4
KERNELS = dict(NONE=0, SELECT=1, PACK=2, NORM=3, GEMM_QKV=4, ATTN=5, ATTN_COMBINE=6, GEMM_O=7,
               GEMM_GATE_UP=8, GEMM_DOWN=9, MOE=10, LM_HEAD=11, ARGMAX_FINAL=12, ACCEPT=13,
               RS_DECIDE=14, RS_RESIDUAL=15, RS_FINISH=16, ATTN_PLAN=17)
RS_SCAN, RS_FIXED, RS_HISTORY = 0, 1, 2

EXPORTS = ["dcut_select", "dcut_verify_layer", "dcut_lm_head_argmax", "dcut_lm_head_argmax_static",
           "dcut_lm_head_static_scratch_bytes", "dcut_accept", "dcut_lm_head_sample", "dcut_select_rs",
           "dcut_accept_rs", "dcut_workspace_bytes", "dcut_strerror", "dcut_budgets_from_ratios",
           "dcut_nearest_batch", "dcut_profile_arm", "dcut_stream_probe"]


class DcutError(RuntimeError):
    def __init__(self, status: int, what: str):
        super().__init__(f"{what}: {strerror(status)} ({status})")
        self.status = status


class LayerCfg(C.Structure):
    _fields_ = [("hidden", C.c_int), ("n_q", C.c_int), ("n_kv", C.c_int), ("head_dim", C.c_int),
                ("inter", C.c_int), ("n_exp", C.c_int), ("top_k", C.c_int), ("exp_inter", C.c_int),
                ("vocab", C.c_int), ("max_ctx", C.c_int), ("rms_eps", C.c_float),
                ("rope_theta", C.c_float)]


_WFIELDS = ["embed", "attn_norm", "w_qkv", "w_o", "mlp_norm", "w_gate_up", "w_down",
            "w_router", "w_exp_gate_up", "w_exp_down"]


class LayerW(C.Structure):
    _fields_ = [(n, C.c_void_p) for n in _WFIELDS]


class KV(C.Structure):
    _fields_ = [("k", C.c_void_p), ("v", C.c_void_p), ("base", C.c_void_p), ("cap", C.c_void_p)]


def _load() -> C.CDLL:
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with `python -m paper_2607_14647_amd.build`")
    lib = C.CDLL(LIB_PATH)
    vp, i32, sz = C.c_void_p, C.c_int, C.c_size_t
    lib.dcut_select.argtypes = [i32, i32, vp, vp, vp, i32, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp]
    lib.dcut_verify_layer.argtypes = [C.POINTER(LayerCfg), C.POINTER(LayerW), i32, i32, vp, vp, vp, vp,
                                      vp, vp, C.POINTER(KV), vp, vp, vp, sz, vp]
    lib.dcut_lm_head_argmax.argtypes = [i32, i32, i32, i32, vp, vp, vp, C.c_float, vp, vp, vp, vp, vp, sz, vp]
    lib.dcut_lm_head_argmax_static.argtypes = [i32, i32, i32, i32, vp, vp, vp, C.c_float, vp, vp, vp, vp, vp]
    lib.dcut_lm_head_static_scratch_bytes.argtypes = []
    lib.dcut_lm_head_static_scratch_bytes.restype = sz
    lib.dcut_lm_head_sample.argtypes = [i32, i32, i32, i32, vp, vp, vp, vp, vp, C.c_float, vp, C.c_float,
                                        C.c_uint64, vp, vp, vp, vp, vp, sz, vp]
    lib.dcut_accept.argtypes = [i32, i32, vp, vp, vp, vp, vp, vp, vp, vp, vp]
    lib.dcut_select_rs.argtypes = [i32, i32, vp, vp, vp, i32, i32, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp]
    lib.dcut_accept_rs.argtypes = [i32, i32, i32, C.c_float, C.c_uint64, vp, vp, vp, vp, vp, vp, vp, vp, vp,
                                   vp, vp, vp, vp, sz, vp, vp]
    lib.dcut_workspace_bytes.argtypes = [i32, C.POINTER(LayerCfg), i32, i32]
    lib.dcut_workspace_bytes.restype = sz
    lib.dcut_strerror.argtypes = [i32]
    lib.dcut_strerror.restype = C.c_char_p
    lib.dcut_budgets_from_ratios.argtypes = [i32, i32, i32, vp, vp, vp]
    lib.dcut_nearest_batch.argtypes = [i32, i32, vp]
    lib.dcut_profile_arm.argtypes = [i32, vp, vp]
    lib.dcut_stream_probe.argtypes = [vp, sz, i32, vp]
    for f in ["dcut_select", "dcut_verify_layer", "dcut_lm_head_argmax", "dcut_lm_head_argmax_static",
              "dcut_lm_head_sample", "dcut_accept",
              "dcut_select_rs", "dcut_accept_rs", "dcut_budgets_from_ratios", "dcut_nearest_batch",
              "dcut_profile_arm"]:
        getattr(lib, f).restype = i32
    return lib


_lib = _load()


def lib() -> C.CDLL:
    return _lib


def strerror(status: int) -> str:
    return _lib.dcut_strerror(int(status)).decode()


def _p(t: Optional[torch.Tensor]):
    return None if t is None else C.c_void_p(t.data_ptr())


def _stream(stream=None):
    s = torch.cuda.current_stream() if stream is None else stream
    return C.c_void_p(s.cuda_stream)


def _check(st: int, what: str) -> None:
    if st != OK:
        raise DcutError(st, what)


def layer_cfg(ly, max_ctx: int) -> LayerCfg:
    return LayerCfg(ly.hidden, ly.n_q, ly.n_kv, ly.head_dim, ly.inter, ly.n_exp, ly.top_k,
                    ly.exp_inter, ly.vocab, int(max_ctx), ly.rms_eps, ly.rope_theta)


# ------------------------------------------------------------------ host helpers

def budgets_from_ratios(B: int, D: int, ratios: Sequence[Sequence[int]]) -> list:
    R = len(ratios)
    num = (C.c_int32 * R)(*[int(r[0]) for r in ratios])
    den = (C.c_int32 * R)(*[int(r[1]) for r in ratios])
    out = (C.c_int32 * R)()
    _check(_lib.dcut_budgets_from_ratios(B, D, R, C.cast(num, C.c_void_p), C.cast(den, C.c_void_p),
                                         C.cast(out, C.c_void_p)), "dcut_budgets_from_ratios")
    return list(out)


def nearest_batch(B: int, captured: Sequence[int]) -> int:
    arr = (C.c_int32 * len(captured))(*[int(c) for c in captured])
    return int(_lib.dcut_nearest_batch(B, len(captured), C.cast(arr, C.c_void_p)))


def workspace_bytes(which: int, cfg: Optional[LayerCfg], B: int, D: int) -> int:
    return int(_lib.dcut_workspace_bytes(which, C.byref(cfg) if cfg is not None else None, B, D))


def profile_arm(kernel: str, start=None, stop=None) -> None:
    """Arm the timing hook for one kernel on this thread: `start` and `stop` carry a HIP event handle in
    `cuda_event` (a torch.cuda.Event already recorded once, or an event created directly)."""
    kid = KERNELS[kernel]
    s = C.c_void_p(start.cuda_event) if start is not None else None
    e = C.c_void_p(stop.cuda_event) if stop is not None else None
    _check(_lib.dcut_profile_arm(kid, s, e), "dcut_profile_arm")


def stream_probe(src: torch.Tensor, workgroups: int, stream=None) -> None:
    """Stream the whole of `src` (a contiguous device tensor) through LDS with
    `workgroups` workgroups of four waves: a measurement aid, not a step."""
    st = _lib.dcut_stream_probe(_p(src), src.numel() * src.element_size(), int(workgroups), _stream(stream))
    _check(st, "dcut_stream_probe")


# ------------------------------------------------------------------ the calls

def select(B: int, D: int, conf: torch.Tensor, draft: torch.Tensor, ctx_len: torch.Tensor,
           budgets: Sequence[int], costs: Sequence[float], out: Dict[str, torch.Tensor],
           dev_err: Optional[torch.Tensor] = None, stream=None) -> None:
    R = len(budgets)
    b = (C.c_int32 * max(R, 1))(*[int(x) for x in budgets])
    c = (C.c_double * max(R, 1))(*[float(x) for x in costs])
    st = _lib.dcut_select(B, D, _p(conf), _p(draft), _p(ctx_len), R, C.cast(b, C.c_void_p),
                          C.cast(c, C.c_void_p), _p(out["keep_len"]), _p(out["cu"]),
                          _p(out["packed_tok"]), _p(out["packed_pos"]), _p(out["packed_req"]),
                          _p(out["choice"]), _p(out.get("benefit")), _p(dev_err), _stream(stream))
    _check(st, "dcut_select")


def select_rs(B: int, D: int, conf: torch.Tensor, draft: torch.Tensor, ctx_len: torch.Tensor, mode: int,
              budgets: Sequence[int], costs: Sequence[float], out: Dict[str, torch.Tensor],
              dev_err: Optional[torch.Tensor] = None, k_state: Optional[torch.Tensor] = None,
              stream=None) -> None:
    R = len(budgets)
    b = (C.c_int32 * max(R, 1))(*[int(x) for x in budgets])
    c = (C.c_double * max(R, 1))(*[float(x) for x in costs])
    st = _lib.dcut_select_rs(B, D, _p(conf), _p(draft), _p(ctx_len), int(mode), R, C.cast(b, C.c_void_p),
                             C.cast(c, C.c_void_p), _p(k_state), _p(out["keep_len"]), _p(out["cu"]),
                             _p(out["packed_tok"]), _p(out["packed_pos"]), _p(out["packed_req"]),
                             _p(out["choice"]), _p(out.get("benefit")), _p(dev_err), _stream(stream))
    _check(st, "dcut_select_rs")


def select_outputs(B: int, D: int, R: int, device="cuda") -> Dict[str, torch.Tensor]:
    rows = B * (D + 1)
    i32 = dict(dtype=torch.int32, device=device)
    return dict(keep_len=torch.zeros(B, **i32), cu=torch.zeros(B + 1, **i32),
                packed_tok=torch.zeros(rows, **i32), packed_pos=torch.zeros(rows, **i32),
                packed_req=torch.zeros(rows, **i32), choice=torch.zeros(2, **i32),
                benefit=torch.zeros(R, dtype=torch.int64, device=device))


def layer_weights(w: Dict[str, torch.Tensor]) -> LayerW:
    return LayerW(*[(w[n].data_ptr() if w.get(n) is not None else None) for n in _WFIELDS])


def kv_desc(kv: Dict[str, torch.Tensor]) -> KV:
    return KV(kv["k"].data_ptr(), kv["v"].data_ptr(), kv["base"].data_ptr(), kv["cap"].data_ptr())


def verify_layer(cfg: LayerCfg, w: LayerW, B: int, D: int, sel: Dict[str, torch.Tensor],
                 ctx_len: torch.Tensor, kv: KV, x_out: torch.Tensor, ws: torch.Tensor,
                 x_in: Optional[torch.Tensor] = None, dev_err: Optional[torch.Tensor] = None,
                 stream=None) -> None:
    st = _lib.dcut_verify_layer(C.byref(cfg), C.byref(w), B, D, _p(sel["cu"]), _p(sel["packed_tok"]),
                                _p(sel["packed_pos"]), _p(sel["packed_req"]), _p(ctx_len), _p(x_in),
                                C.byref(kv), _p(x_out), _p(dev_err), _p(ws), ws.numel() * ws.element_size(),
                                _stream(stream))
    _check(st, "dcut_verify_layer")


def lm_head_argmax(H: int, V: int, B: int, D: int, cu: torch.Tensor, x: torch.Tensor,
                   final_norm: torch.Tensor, eps: float, w_lm: torch.Tensor, argmax: torch.Tensor,
                   ws: torch.Tensor, max_logit: Optional[torch.Tensor] = None,
                   logits: Optional[torch.Tensor] = None, stream=None) -> None:
    st = _lib.dcut_lm_head_argmax(H, V, B, D, _p(cu), _p(x), _p(final_norm), float(eps), _p(w_lm),
                                  _p(argmax), _p(max_logit), _p(logits), _p(ws),
                                  ws.numel() * ws.element_size(), _stream(stream))
    _check(st, "dcut_lm_head_argmax")


def lm_head_argmax_static(H: int, V: int, B: int, D: int, cu: torch.Tensor, x: torch.Tensor,
                          final_norm: torch.Tensor, eps: float, w_lm: torch.Tensor, argmax: torch.Tensor,
                          max_logit: Optional[torch.Tensor] = None, logits: Optional[torch.Tensor] = None,
                          stream=None) -> None:
    st = _lib.dcut_lm_head_argmax_static(H, V, B, D, _p(cu), _p(x), _p(final_norm), float(eps), _p(w_lm),
                                         _p(argmax), _p(max_logit), _p(logits), _stream(stream))
    _check(st, "dcut_lm_head_argmax_static")


def lm_head_static_scratch_bytes() -> int:
    return int(_lib.dcut_lm_head_static_scratch_bytes())


def lm_head_sample(H: int, V: int, B: int, D: int, cu: torch.Tensor, packed_req: torch.Tensor,
                   packed_pos: torch.Tensor, x: torch.Tensor, final_norm: torch.Tensor, eps: float,
                   w_lm: torch.Tensor, temperature: float, seed: int, token: torch.Tensor, ws: torch.Tensor,
                   max_score: Optional[torch.Tensor] = None, logits: Optional[torch.Tensor] = None,
                   lse: Optional[torch.Tensor] = None, stream=None) -> None:
    st = _lib.dcut_lm_head_sample(H, V, B, D, _p(cu), _p(packed_req), _p(packed_pos), _p(x), _p(final_norm),
                                  float(eps), _p(w_lm), float(temperature), int(seed) & 0xFFFFFFFFFFFFFFFF,
                                  _p(token), _p(max_score), _p(logits), _p(lse), _p(ws),
                                  ws.numel() * ws.element_size(), _stream(stream))
    _check(st, "dcut_lm_head_sample")


def accept(B: int, D: int, draft: torch.Tensor, keep_len: torch.Tensor, cu: torch.Tensor,
           argmax: torch.Tensor, accept_len: torch.Tensor, next_tok: torch.Tensor,
           total: torch.Tensor, ctx_len_inout: Optional[torch.Tensor] = None, stream=None) -> None:
    st = _lib.dcut_accept(B, D, _p(draft), _p(keep_len), _p(cu), _p(argmax), _p(accept_len),
                          _p(next_tok), _p(total), _p(ctx_len_inout), _stream(stream))
    _check(st, "dcut_accept")


def accept_rs(B: int, D: int, V: int, temperature: float, seed: int, draft: torch.Tensor, q: torch.Tensor,
              keep_len: torch.Tensor, cu: torch.Tensor, packed_pos: torch.Tensor, logits: torch.Tensor,
              lse: torch.Tensor, token: torch.Tensor, accept_len: torch.Tensor, next_tok: torch.Tensor,
              total: torch.Tensor, ws: torch.Tensor, ctx_len_inout: Optional[torch.Tensor] = None,
              dev_err: Optional[torch.Tensor] = None, stream=None) -> None:
    st = _lib.dcut_accept_rs(B, D, V, float(temperature), int(seed) & 0xFFFFFFFFFFFFFFFF, _p(draft), _p(q),
                             _p(keep_len), _p(cu), _p(packed_pos), _p(logits), _p(lse), _p(token),
                             _p(accept_len), _p(next_tok), _p(total), _p(ctx_len_inout), _p(ws),
                             ws.numel() * ws.element_size(), _p(dev_err), _stream(stream))
    _check(st, "dcut_accept_rs")


def workspace(nbytes: int, device="cuda") -> torch.Tensor:
    """A 256-byte aligned device scratch buffer (torch's allocator aligns to 512 bytes)."""
    t = torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device=device)
    assert t.data_ptr() % 256 == 0
    return t
