"""The C ABI without a GPU: exports, host helpers, argument validation before any launch."""
import ctypes as C
import json
import os
import re

import pytest

from paper_2607_14647_amd import lib as L
from oracle import select as osel

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "dcut.h")


def _declared():
    src = open(HEADER).read()
    return sorted(set(re.findall(r"^\w[\w\s\*]*?\b(dcut_\w+)\s*\(", src, flags=re.M)))


def test_every_declared_symbol_is_exported():
    names = _declared()
    assert set(names) == set(L.EXPORTS)
    lib = L.lib()
    for n in names:
        assert hasattr(lib, n), n


def test_enums_match_header():
    src = open(HEADER).read()
    for name, val in [("DCUT_EINVAL", L.EINVAL), ("DCUT_EWORKSPACE", L.EWORKSPACE),
                      ("DCUT_DERR_CAPACITY", L.DERR_CAPACITY)]:
        assert re.search(rf"{name}\s*=\s*{val}\b", src)
    ids = re.sub(r"/\*.*?\*/", "", re.search(r"DCUT_KERNEL_NONE = 0,([^}]*)\}", src).group(1), flags=re.S)
    names = ["NONE"] + [s.strip().replace("DCUT_KERNEL_", "") for s in ids.split(",") if s.strip()]
    assert names == list(L.KERNELS)


def test_budgets_from_ratios_match_paper_and_oracle():
    g = json.load(open(os.path.join(ROOT, "tests", "golden", "cost_table_tab3.json")))
    for bi, B in enumerate(g["B"]):
        assert L.budgets_from_ratios(B, g["D"], g["ratios"]) == g["budget_from_caption"][bi]
    for B, D, n, d in [(10, 0, 1, 4), (3, 3, 1, 3), (3, 3, 1, 5), (7, 9, 2, 3), (4096, 1, 1, 3)]:
        assert L.budgets_from_ratios(B, D, [(n, d)]) == [osel.budget_from_ratio(B, D, n, d)]
    for bad in [[(5, 4)], [(1, 0)], [(-1, 2)]]:
        with pytest.raises(L.DcutError):
            L.budgets_from_ratios(8, 15, bad)


def test_nearest_batch_rule():
    caps = [1, 8, 16, 32, 64]
    assert L.nearest_batch(20, caps) == 2
    assert L.nearest_batch(24, caps) == 3          # tie 16/32 -> larger
    assert L.nearest_batch(100, caps) == 4
    assert L.nearest_batch(0, caps) == 0
    assert L.nearest_batch(5, []) == -1


def test_workspace_sizes():
    cfg = L.LayerCfg(4096, 32, 8, 128, 14336, 0, 0, 0, 128256, 4112, 1e-5, 5e5)
    assert L.workspace_bytes(0, None, 64, 15) == 0
    assert L.workspace_bytes(3, None, 64, 15) == 0
    ws1 = L.workspace_bytes(1, cfg, 64, 15)
    assert 0 < ws1 < (1 << 31) and ws1 % 256 == 0
    # normalised rows plus, per row and 64 columns of the vocabulary, one key and one
    # (max, sum) pair of the log-partition function
    assert L.workspace_bytes(2, cfg, 64, 15) >= 1024 * 4096 * 2 + 2 * 1024 * 4 * ((cfg.vocab + 255) // 256) * 8
    odd = L.LayerCfg(2048, 32, 4, 128, 0, 128, 8, 768, 151936, 4112, 1e-5, 1e6)      # V / 128 odd
    assert L.workspace_bytes(2, odd, 128, 15) >= 2048 * 2048 * 2 + 2 * 2048 * 4 * ((151936 + 255) // 256) * 8
    # RS acceptance: two int32 per request plus one key per request and 2048-column chunk
    nch = (cfg.vocab + 2047) // 2048
    assert L.workspace_bytes(4, cfg, 64, 15) >= 64 * 8 + 64 * nch * 8
    assert L.workspace_bytes(4, None, 64, 15) == 2 ** 64 - 1
    assert L.workspace_bytes(1, cfg, 0, 15) == 2 ** 64 - 1
    bad = L.LayerCfg(4096, 32, 7, 128, 14336, 0, 0, 0, 128256, 4112, 1e-5, 5e5)
    assert L.workspace_bytes(1, bad, 64, 15) == 2 ** 64 - 1


def _sel_call(B, D, R, budgets, costs, null_out=False):
    lib = L.lib()
    b = (C.c_int32 * max(R, 1))(*budgets)
    c = (C.c_double * max(R, 1))(*costs)
    fake = C.c_void_p(0x1000)           # never dereferenced: validation fails first
    outp = None if null_out else fake
    return lib.dcut_select(B, D, fake, fake, fake, R, C.cast(b, C.c_void_p), C.cast(c, C.c_void_p),
                           outp, fake, fake, fake, fake, fake, None, None, None)


@pytest.mark.parametrize("B,D,R,budgets,costs", [
    (0, 15, 1, [1], [1.0]), (4097, 0, 1, [4097], [1.0]), (4, 64, 1, [4], [1.0]),
    (1024, 15, 1, [1024], [1.0]), (4, 15, 0, [], []), (4, 15, 65, [4] * 65, [1.0] * 65),
    (4, 15, 1, [3], [1.0]), (4, 15, 1, [65], [1.0]), (4, 15, 2, [8, 6], [1.0, 1.0]),
    (4, 15, 1, [8], [0.0]), (4, 15, 1, [8], [-1.0]), (4, 15, 1, [8], [float("nan")]),
    (4, 15, 1, [8], [float("inf")]),
])
def test_select_rejects_invalid_args(B, D, R, budgets, costs):
    assert _sel_call(B, D, R, budgets, costs) == L.EINVAL


def _sel_rs_call(mode, R, budgets, costs, k_state=None):
    lib = L.lib()
    b = (C.c_int32 * max(R, 1))(*budgets)
    c = (C.c_double * max(R, 1))(*costs)
    fake = C.c_void_p(0x1000)
    return lib.dcut_select_rs(4, 15, fake, fake, fake, mode, R, C.cast(b, C.c_void_p), C.cast(c, C.c_void_p),
                              k_state, fake, fake, fake, fake, fake, fake, None, None, None)


def test_select_rs_rejects_invalid_args():
    assert _sel_rs_call(-1, 1, [8], [1.0]) == L.EINVAL
    assert _sel_rs_call(L.RS_FIXED, 2, [8, 16], [1.0, 2.0]) == L.EINVAL    # a fixed budget is one budget
    assert _sel_rs_call(L.RS_SCAN, 1, [3], [1.0]) == L.EINVAL              # below B
    assert _sel_rs_call(L.RS_SCAN, 2, [16, 8], [1.0, 2.0]) == L.EINVAL     # decreasing
    assert _sel_rs_call(L.RS_SCAN, 1, [8], [0.0]) == L.EINVAL
    assert _sel_rs_call(L.RS_HISTORY, 2, [8, 16], [1.0, 2.0]) == L.EINVAL   # history needs its state word
    assert _sel_rs_call(3, 1, [8], [1.0]) == L.EINVAL


def test_select_rejects_null_outputs():
    assert _sel_call(4, 15, 1, [8], [1.0], null_out=True) == L.EINVAL


def test_other_entry_points_reject_invalid_args():
    lib = L.lib()
    fake = C.c_void_p(0x1000)
    assert lib.dcut_accept(0, 15, fake, fake, fake, fake, fake, fake, fake, None, None) == L.EINVAL
    assert lib.dcut_accept(4, 15, None, fake, fake, fake, fake, fake, fake, None, None) == L.EINVAL
    assert lib.dcut_lm_head_argmax(4095, 10, 4, 15, fake, fake, fake, 1e-5, fake, fake, None, None,
                                   fake, 1 << 30, None) == L.EINVAL
    assert lib.dcut_lm_head_argmax(4096, 10, 4, 15, fake, fake, fake, 1e-5, fake, fake, None, None,
                                   None, 0, None) == L.EWORKSPACE
    # temperature sampling: null request/position arrays, non-positive or infinite temperature
    smp = lambda req, pos, T, wsb, lg=None, lse=None: lib.dcut_lm_head_sample(
        4096, 10, 4, 15, fake, req, pos, fake, fake, 1e-5, fake, T, 7, fake, None, lg, lse, fake, wsb, None)
    assert smp(None, fake, 1.0, 1 << 30) == L.EINVAL
    assert smp(fake, None, 1.0, 1 << 30) == L.EINVAL
    assert smp(fake, fake, 0.0, 1 << 30) == L.EINVAL
    assert smp(fake, fake, -1.0, 1 << 30) == L.EINVAL
    assert smp(fake, fake, float("inf"), 1 << 30) == L.EINVAL
    assert smp(fake, fake, float("nan"), 1 << 30) == L.EINVAL
    assert smp(fake, fake, 1.0, 0) == L.EWORKSPACE
    cfg = L.LayerCfg(256, 4, 2, 64, 688, 0, 0, 0, 1024, 160, 1e-5, 5e5)
    w = L.LayerW(*([0x1000] * 7 + [None] * 3))
    kv = L.KV(0x1000, 0x1000, 0x1000, 0x1000)
    args = lambda c, wsb: lib.dcut_verify_layer(C.byref(c), C.byref(w), 4, 15, fake, fake, fake, fake,
                                                fake, None, C.byref(kv), fake, None, fake, wsb, None)
    assert args(cfg, 0) == L.EWORKSPACE
    bad = L.LayerCfg(256, 4, 3, 64, 688, 0, 0, 0, 1024, 160, 1e-5, 5e5)
    assert args(bad, 1 << 30) == L.EINVAL
    hd = L.LayerCfg(256, 4, 2, 96, 688, 0, 0, 0, 1024, 160, 1e-5, 5e5)
    assert args(hd, 1 << 30) == L.EUNSUPPORTED
    # RS acceptance: sizes, temperature, null pointers, then the workspace
    acc = lambda B, V, T, q, wsb: lib.dcut_accept_rs(B, 15, V, T, 3, fake, q, fake, fake, fake, fake, fake, fake,
                                                      fake, fake, fake, None, fake, wsb, None, None)
    assert acc(0, 10, 1.0, fake, 1 << 30) == L.EINVAL
    assert acc(4, 0, 1.0, fake, 1 << 30) == L.EINVAL
    assert acc(4, 10, 0.0, fake, 1 << 30) == L.EINVAL
    assert acc(4, 10, float("inf"), fake, 1 << 30) == L.EINVAL
    assert acc(4, 10, 1.0, None, 1 << 30) == L.EINVAL
    assert acc(4, 10, 1.0, fake, 0) == L.EWORKSPACE
    assert lib.dcut_profile_arm(99, None, None) == L.EINVAL
    assert lib.dcut_profile_arm(L.KERNELS["LM_HEAD"], None, None) == L.EINVAL
    assert lib.dcut_profile_arm(0, None, None) == L.OK
    assert L.strerror(L.EHIP).startswith("HIP")
    # stream probe: alignment, workgroup count, a size that does not split into whole 1 KB loads
    # per wave, and a per-wave range past what one buffer resource addresses
    sp = lib.dcut_stream_probe
    assert sp(None, 1 << 20, 4, None) == L.EINVAL
    assert sp(C.c_void_p(0x1008), 1 << 20, 4, None) == L.EINVAL
    assert sp(fake, 1 << 20, 0, None) == L.EINVAL
    assert sp(fake, 1 << 20, 65537, None) == L.EINVAL
    assert sp(fake, 0, 4, None) == L.EINVAL
    assert sp(fake, (1 << 20) + 1024, 4, None) == L.EINVAL
    assert sp(fake, 4 << 31, 1, None) == L.EUNSUPPORTED


def test_operands_past_32bit_offsets_are_rejected_before_any_launch():
    """The GEMM addresses each task's A rows and each column tile's W rows from their own
    base, so any total weight size is accepted (an LM head of H = 8192, V = 152064, 2.49 GB,
    passes validation and fails only on the fake workspace); what a single task or column
    tile spans must stay below 2 GiB, else DCUT_EUNSUPPORTED before any launch."""
    lib = L.lib()
    fake = C.c_void_p(0x1000)
    lm = lambda H, V: lib.dcut_lm_head_argmax(H, V, 4, 15, fake, fake, fake, 1e-5, fake, fake, None, None,
                                              None, 0, None)
    assert lm(8192, 152064) == L.EWORKSPACE
    assert lm(1 << 22, 1024) == L.EUNSUPPORTED         # one 256-row tile of W spans 2 GiB
    w = L.LayerW(*([0x1000] * 7 + [None] * 3))
    kv = L.KV(0x1000, 0x1000, 0x1000, 0x1000)
    call = lambda c: lib.dcut_verify_layer(C.byref(c), C.byref(w), 4, 15, fake, fake, fake, fake, fake, None,
                                           C.byref(kv), fake, None, None, 0, None)
    # a SwiGLU tile pairs gate row p with up row inter + p: inter * hidden * 2 bytes apart
    assert call(L.LayerCfg(8192, 64, 8, 128, 1 << 17, 0, 0, 0, 1024, 160, 1e-5, 5e5)) == L.EUNSUPPORTED
    assert call(L.LayerCfg(8192, 64, 8, 128, 28672, 0, 0, 0, 1024, 160, 1e-5, 5e5)) == L.EWORKSPACE
    # one request's key slab [cap][head_dim] must stay below 2 GiB
    assert call(L.LayerCfg(256, 4, 2, 128, 688, 0, 0, 0, 1024, 1 << 23, 1e-5, 5e5)) == L.EUNSUPPORTED


def test_static_lm_head_rejects_shapes_beyond_its_array():
    """dcut_lm_head_argmax_static refuses, before any launch, a shape whose scratch exceeds its
    32 MiB array (the 256-request step with V = 151936 needs far more) and validates like the
    workspace call."""
    lib = L.lib()
    fake = C.c_void_p(0x1000)
    call = lambda H, V, B, D, out=fake: lib.dcut_lm_head_argmax_static(H, V, B, D, fake, fake, fake, 1e-5, fake,
                                                                       out, None, None, None)
    assert L.lm_head_static_scratch_bytes() == 32 << 20
    assert call(4096, 151936, 256, 15) == L.EUNSUPPORTED
    assert call(4095, 1024, 4, 15) == L.EINVAL
    assert call(4096, 1024, 0, 15) == L.EINVAL
    assert call(4096, 1024, 4, 15, out=None) == L.EINVAL
