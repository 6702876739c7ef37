#!/usr/bin/env python3
"""Benchmark of the D-cut verify step on one MI355X.

A step is the whole hot path over one batch: dcut_select (scores, ranking,
cost-model budget, keep depths, packing), dcut_verify_layer (one dense 8B-class
decoder layer), dcut_lm_head_argmax and dcut_accept, on one stream with every
input already resident in HBM.  The metric is accepted tokens per second:
sum_i (a_i + 1) per step divided by the step time, at the budget K* that the
step picks from the measured cost row.

Sequence:
  1. seeded synthetic workload (default: batch 64, dense 8B-shaped layer);
  2. synthetic drafter: draft k matches the library's own greedy token at
     position k-1 with probability c_k (so acceptance follows the scores);
  3. cost row: each candidate budget K_r forced alone (R = 1), median step time;
  4. per-kernel breakdown with the library's timing hook, to find the dominant kernel;
  5. timed region: `--steps` adaptive steps (all candidates, measured costs),
     with the dominant kernel timed by HIP events inside the same region;
  6. CPU baseline: the oracle on a bounded sample of the same batch.
Prints one JSON line.

`--temperature T` samples the target's tokens (dcut_lm_head_sample); `--rs`
verifies by rejection sampling (dcut_select_rs, dcut_lm_head_sample with
logits, dcut_accept_rs) against a synthetic stochastic drafter.
"""
import argparse
import hashlib
import json
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0
PEAK_BF16_TFLOPS = 2500.0
RIDGE = PEAK_BF16_TFLOPS * 1e12 / (PEAK_HBM_GBS * 1e9)


class HookEvent:
    """A HIP event for the library's timing hook, created with hipEventDisableSystemFence:
    recording it around a launch then writes back and invalidates no cache, so timing a kernel
    inside the timed region costs the step about 1 us instead of about 6 (torch's events use the
    system-scope fence).  `cuda_event` is the raw handle that `lib.profile_arm` passes on."""
    _hip = None

    def __init__(self):
        import ctypes as C
        if HookEvent._hip is None:
            hip = C.CDLL("libamdhip64.so")
            hip.hipEventCreateWithFlags.argtypes = [C.POINTER(C.c_void_p), C.c_uint]
            hip.hipEventElapsedTime.argtypes = [C.POINTER(C.c_float), C.c_void_p, C.c_void_p]
            hip.hipEventDestroy.argtypes = [C.c_void_p]
            HookEvent._hip = hip
        e = C.c_void_p()
        rc = HookEvent._hip.hipEventCreateWithFlags(C.byref(e), 0x20000000)   # hipEventDisableSystemFence
        assert rc == 0, f"hipEventCreateWithFlags: {rc}"
        self.cuda_event = e.value

    def elapsed_time(self, end):
        """Milliseconds from this event to `end` (both recorded by a hooked launch)."""
        import ctypes as C
        f = C.c_float()
        rc = HookEvent._hip.hipEventElapsedTime(C.byref(f), C.c_void_p(self.cuda_event), C.c_void_p(end.cuda_event))
        assert rc == 0, f"hipEventElapsedTime: {rc}"
        return f.value

    def __del__(self):
        if HookEvent._hip is not None and self.cuda_event:
            HookEvent._hip.hipEventDestroy(self.cuda_event)


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def kernel_work(name, cfg, K, ctx_len):
    """Algorithmic (flops, bytes) of one launch of `name` at K kept rows."""
    ly = cfg.layer
    H, V, hd, nq, nkv = ly.hidden, ly.vocab, ly.head_dim, ly.n_q, ly.n_kv
    I = ly.inter
    nqkv = (nq + 2 * nkv) * hd
    if ly.n_exp > 0 and name in ("GEMM_GATE_UP", "GEMM_DOWN"):
        # grouped expert GEMMs over the K * top_k routed rows; every expert's weights are
        # counted (with K * top_k >> n_exp nearly all of them are touched)
        E, k, Ie = ly.n_exp, ly.top_k, ly.exp_inter
        if name == "GEMM_GATE_UP":
            return 2.0 * K * k * 2 * Ie * H, E * 2 * Ie * H * 2 + K * k * (H + Ie) * 2
        return 2.0 * K * k * H * Ie, E * H * Ie * 2 + K * k * (Ie * 2 + H * 4)
    if name == "LM_HEAD":
        return 2.0 * K * V * H, V * H * 2 + K * H * 2 + K * 8
    if name == "GEMM_GATE_UP":
        return 2.0 * K * 2 * I * H, 2 * I * H * 2 + K * H * 2 + K * I * 2
    if name == "GEMM_DOWN":
        return 2.0 * K * H * I, H * I * 2 + K * I * 2 + 2 * K * H * 4
    if name == "GEMM_QKV":
        return 2.0 * K * nqkv * H, nqkv * H * 2 + K * H * 2 + K * nqkv * 2
    if name == "GEMM_O":
        return 2.0 * K * H * nq * hd, H * nq * hd * 2 + K * nq * hd * 2 + 2 * K * H * 4
    if name == "ATTN":
        kv_bytes = float(sum(int(L) for L in ctx_len)) * nkv * hd * 2 * 2
        return 0.0, kv_bytes + K * (nq + 2 * nkv) * hd * 2
    return 0.0, 0.0


def roofline(name, cfg, K, ctx_len, us):
    fl, by = kernel_work(name, cfg, K, ctx_len)
    if fl > 0 and fl / by > RIDGE:
        ach = fl / (us * 1e-6) / 1e12
        return dict(bound="mfma", achieved=round(ach, 2), peak=PEAK_BF16_TFLOPS, unit="TFLOP/s",
                    frac=round(ach / PEAK_BF16_TFLOPS, 4), flops=fl, bytes=by)
    ach = by / (us * 1e-6) / 1e9
    return dict(bound="hbm", achieved=round(ach, 1), peak=PEAK_HBM_GBS, unit="GB/s",
                frac=round(ach / PEAK_HBM_GBS, 4), flops=fl, bytes=by)


def kernel_fraction(name, cfg, K, ctx_len, us):
    """Fraction of the roofline time max(bytes / HBM peak, flops / bf16 peak) that a
    kernel with algorithmic work reaches; None for latency-bound kernels."""
    fl, by = kernel_work(name, cfg, K, ctx_len)
    if by <= 0 or us <= 0:
        return None
    ideal_us = max(by / (PEAK_HBM_GBS * 1e9), fl / (PEAK_BF16_TFLOPS * 1e12)) * 1e6
    return dict(bound="mfma" if fl / by > RIDGE else "hbm", ideal_us=round(ideal_us, 2), us=us,
                frac=round(ideal_us / us, 4))


# launches per step of each kernel that the counter summary covers (per decoder layer
# where the kernel belongs to the layer); O and down share one kernel and one entry
COUNTED_LAUNCHES = {"LM_HEAD": (1, False), "GEMM_GATE_UP": (1, True), "GEMM_QKV": (1, True),
                    "ATTN": (1, True), "GEMM_O+DOWN": (2, True)}


def counted_step_bytes(workload, K, layers):
    """HBM bytes per step of the kernels in the committed counter summary, when it
    was taken on the current sources, the same workload and K*; else None."""
    p = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(p):
        return None
    try:
        t = json.load(open(p))
    except ValueError:
        return None
    total, kernels = 0.0, []
    for kid, (n, per_layer) in COUNTED_LAUNCHES.items():
        e = t.get(kid)
        if not e or e.get("source_hash") != source_hash() or e.get("workload") != workload or e.get("K") != K:
            return None
        total += e["bytes_per_launch"] * n * (layers if per_layer else 1)
        kernels.append(kid)
    return total, kernels


def source_hash():
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2607_14647_amd", "csrc")
    for f in sorted(os.listdir(csrc)):
        h.update(open(os.path.join(csrc, f), "rb").read())
    return h.hexdigest()[:16]


def measured_traffic(kernel, workload, K):
    """HBM bytes per launch from the committed rocprofv3 counter summary, if it
    was taken on the current kernel sources and the same workload and K*."""
    p = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(p):
        return None
    try:
        t = json.load(open(p))
    except ValueError:
        return None
    e = t.get(kernel)
    if not e or e.get("source_hash") != source_hash() or e.get("workload") != workload or e.get("K") != K:
        return None
    return e.get("bytes_per_launch")


def cpu_baseline(cfg, st, w, kv, budgets, costs, target_s=15.0):
    """The oracle on the first n requests of the batch, n sized for ~10-30 s of CPU work."""
    import numpy as np
    import threadpoolctl
    from oracle import accept as oacc
    from oracle import drafts as odr
    from oracle import layer as olay
    from oracle import lm_head as olm
    from oracle import select as osel

    info = threadpoolctl.threadpool_info()
    cores = max([d.get("num_threads", 1) for d in info] + [1])
    cpu_model = "unknown"
    try:
        cpu_model = next((l.split(":", 1)[1].strip() for l in open("/proc/cpuinfo") if l.startswith("model name")),
                         "unknown")
    except OSError:
        pass
    blas = sorted({d.get("internal_api", "?") for d in info if d.get("user_api") == "blas"})
    # the selection alone, single-threaded, median of 3
    with threadpoolctl.threadpool_limits(1):
        ts = []
        for _ in range(3):
            t0 = time.perf_counter()
            osel.select(st["conf"], st["draft"], st["ctx_len"], budgets, costs)
            ts.append(time.perf_counter() - t0)
    select_ms = 1000.0 * statistics.median(ts)
    log(f"cpu baseline: converting weights (BLAS threads {cores})")
    w64 = olay.prepare_weights(w)
    ly = cfg.layer

    def run(sample, z):
        t0 = time.perf_counter()
        sel = osel.select(st["conf"], z, st["ctx_len"], budgets, costs)
        lay = olay.verify_layer(ly, w64, kv, sel["cu"], sel["packed_tok"], sel["packed_pos"],
                                sel["packed_req"], st["ctx_len"], cfg.D, requests=sample)
        rows = np.concatenate([np.arange(sel["cu"][i], sel["cu"][i + 1]) for i in sample])
        lm = olm.lm_head_argmax(lay["x_out"][rows], w64["final_norm"], ly.rms_eps, w64["w_lm"])
        g = np.zeros(int(sel["cu"][-1]), np.int32)
        g[rows] = lm["argmax"]
        acc = oacc.accept(z, sel["keep_len"], sel["cu"], g)
        dt = time.perf_counter() - t0
        # requests whose deciding rows hold a near-tie of the top-2 logits (argmax gate 1e-2)
        gap = np.full(len(g), np.inf)
        gap[rows] = lm["gap"]
        tie = [i for i in sample if (gap[sel["cu"][i]: sel["cu"][i] + acc["accept_len"][i] + 1] <= 1e-2).any()]
        per_req = [int(acc["accept_len"][i]) + 1 for i in sample]
        return dt, int(sum(per_req)), len(rows), per_req, tie

    # drafts of the sampled requests forced by the oracle itself (not timed)
    probe = [0]
    z = odr.force_matches(ly, w64, kv, st["conf"], st["draft"], st["match_u"], st["ctx_len"], cfg.D,
                          requests=probe)
    dt1 = run(probe, z)[0]
    n = int(max(1, min(cfg.B, target_s / max(dt1, 1e-3))))
    sample = list(range(n))
    log(f"cpu baseline: one request {dt1:.2f}s -> sample of {n} requests; forcing their drafts")
    z = odr.force_matches(ly, w64, kv, st["conf"], st["draft"], st["match_u"], st["ctx_len"], cfg.D,
                          requests=sample)
    # the same pass repeated until about 10 s of CPU work have run (the whole batch may take less)
    dt, tokens, nrows, per_req, tie = run(sample, z)
    passes = 1
    while dt < 10.0:
        dt += run(sample, z)[0]
        passes += 1
    return dict(value=round(tokens * passes / dt, 2), unit="accepted tokens/s", cores=int(cores), kind="oracle",
                sample=f"requests 0..{n - 1} of the batch ({nrows} kept rows, {tokens} accepted tokens): "
                       f"full-batch selection, then the float64 layer + LM head + accept for the sample; "
                       f"{passes} passes, {dt:.1f} s", seconds=round(dt, 2),
                select_ms_1thread=round(select_ms, 2), cpu_model=cpu_model, cpu_count=os.cpu_count(),
                affinity=len(os.sched_getaffinity(0)), blas=blas,
                oracle_accepted=tokens, oracle_accepted_per_request=per_req, near_tie_requests=tie,
                sample_requests=sample, draft_rows=[z[i].tolist() for i in sample])


def parse_args():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--config", type=int, default=3)
    ap.add_argument("--seed", type=int, default=None,
                    help="one seed only (default: the greedy headline runs seeds 0-4 and reports their median; "
                         "the other modes run seed 0)")
    ap.add_argument("--cost-reps", type=int, default=20)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cold", action="store_true", help="evict the MALL between timed steps")
    ap.add_argument("--copy-bytes", type=int, default=0,
                    help="after the timed region, run a plain device-to-device copy of this many bytes "
                         "three times (reference kernel for scaling HBM byte counters)")
    ap.add_argument("--temperature", type=float, default=0.0,
                    help="target decoding: 0 = greedy (default), T > 0 = temperature-T sampling through "
                         "dcut_lm_head_sample (the paper's temperature-1 regime); drafts are forced from "
                         "the same sampled tokens")
    ap.add_argument("--sample-seed", type=int, default=1, help="seed of the sampling noise")
    ap.add_argument("--rs", action="store_true",
                    help="rejection-sampling verification (dcut_select_rs with the causal scan, "
                         "dcut_lm_head_sample with logits, dcut_accept_rs) against a synthetic stochastic "
                         "drafter; temperature 1 unless --temperature is given")
    ap.add_argument("--rs-budget", choices=("scan", "history"), default="scan",
                    help="with --rs: the causal early-stopping scan over the cost row, or the history-based "
                         "budget (the previous block's choice, carried on the device)")
    ap.add_argument("--layers", type=int, default=1,
                    help="decoder layers in the verify pass (each with its own seeded weights and KV cache); "
                         "32 is the full depth of the 8B-shaped target")
    ap.add_argument("--graph", action="store_true",
                    help="also capture the adaptive step into a HIP graph and time its replays "
                         "(reported as graph_ms_per_step beside the eager figures)")
    ap.add_argument("--cost-table", action="store_true",
                    help="run the startup cost-table protocol over captured batch sizes 1, 8, 16, 32, 64 and "
                         "the ratio buckets 25/50/75/100 %% (each entry a graph-captured step, median of 10)")
    ap.add_argument("--force-k", type=int, default=0,
                    help="time the step at this one budget instead of the cost model's choice (no cost row, "
                         "no CPU baseline); B(D+1) gives the unpruned step")
    ap.add_argument("--state", default=None,
                    help="JSON file with the forced drafts, cost row and dominant kernel of an earlier "
                         "run of the same workload; written when missing, reused when present (a "
                         "profiler run then sees only the timed adaptive steps at K*)")
    return ap.parse_args()


def main():
    args = parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py: measures one GPU only; the verify step has no multi-GPU path. "
              "Run with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch
    from paper_2607_14647_amd import lib as L
    from paper_2607_14647_amd import runner
    from paper_2607_14647_amd import workload as wl

    assert torch.cuda.is_available(), "bench.py needs an MI355X GPU"
    if args.rs and args.temperature == 0:
        args.temperature = 1.0
    greedy_headline = not (args.rs or args.temperature > 0 or args.layers > 1 or args.state or args.force_k)
    if args.seed is not None:
        seeds = [args.seed]
    else:
        seeds = [0, 1, 2, 3, 4] if greedy_headline else [0]
    cfg = wl.CONFIGS[args.config]
    ly = cfg.layer
    stream = torch.cuda.current_stream()
    flush = torch.empty(512 << 20, dtype=torch.uint8, device="cuda") if args.cold else None
    budgets = list(cfg.budgets) if not args.force_k else [int(args.force_k)]
    assert all(cfg.B <= K <= cfg.B * (cfg.D + 1) for K in budgets), "budget outside [B, B(D+1)]"

    def timed(fn, reps):
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(reps)]
        for a, b in evs:
            if flush is not None:
                flush.fill_(1)
            a.record(stream)
            fn()
            b.record(stream)
        torch.cuda.synchronize()
        return [a.elapsed_time(b) for a, b in evs]

    def setup(seed, state):
        log(f"workload cfg{cfg.cid} ({cfg.name}) seed {seed}: generating")
        t0 = time.time()
        st = wl.make_step_inputs(cfg, seed)
        w = wl.make_weights(cfg, seed)
        kv = wl.make_kv(cfg, seed, st["ctx_len"])
        log(f"generated in {time.time() - t0:.1f}s; uploading")
        vs = runner.VerifyStep(cfg, w, st, kv)
        for l in range(1, args.layers):
            vs.add_layer(wl.make_weights(cfg, seed, layer=l), wl.make_kv(cfg, seed, st["ctx_len"], layer=l))
            if l % 8 == 0 or l == args.layers - 1:
                log(f"layer {l} of {args.layers - 1} extra layers generated and uploaded")
        vs.temperature, vs.seed = float(args.temperature), int(args.sample_seed)
        torch.cuda.synchronize()
        if args.rs:
            vs.enable_rs(None)
            vs.rs_mode = L.RS_HISTORY if args.rs_budget == "history" else L.RS_SCAN
            vs.k_state.fill_(budgets[-1])
            log("stochastic drafter: proposals and drafts from the target's own distributions (D passes)")
            runner.force_drafts_rs_on_device(vs, st["draft"], st["conf"], st["match_u"], args.sample_seed + 1000)
        elif state is not None:
            vs.set_draft(np.array(state["draft"], dtype=np.int32))
            log(f"reusing forced drafts, cost row and dominant kernel from {args.state}")
        else:
            log("forcing draft matches (synthetic drafter, D passes at full budget)")
            runner.force_drafts_on_device(vs, st["draft"], st["conf"], st["match_u"])
        torch.cuda.synchronize()
        return vs, st, w, kv

    def cost_row(vs):
        """Each candidate budget forced alone (R = 1): median step time and accepted tokens."""
        run_step = vs.step_rs if args.rs else vs.step
        cost_ms, acc_per_k = [], []
        for K in budgets:
            step = lambda K=K: run_step([K], [1.0])
            timed(step, 2)
            cost_ms.append(statistics.median(timed(step, args.cost_reps)))
            acc_per_k.append(int(vs.total.item()))
        log("cost row (ms): " + ", ".join(f"{K}:{c:.3f}" for K, c in zip(budgets, cost_ms)))
        return cost_ms, acc_per_k

    names = ["SELECT", "NORM", "GEMM_QKV", "ATTN", "ATTN_COMBINE", "GEMM_O", "GEMM_GATE_UP", "GEMM_DOWN",
             "LM_HEAD", "ARGMAX_FINAL"]
    names += ["RS_DECIDE", "RS_RESIDUAL", "RS_FINISH"] if args.rs else ["ACCEPT"]

    def kernel_breakdown(fn):
        """Mean device time (us) of each kernel's last launch in a step, through the timing hook."""
        out = {}
        for nm in names:
            pairs = [(HookEvent(), HookEvent()) for _ in range(5)]
            torch.cuda.synchronize()
            for a, b in pairs:
                L.profile_arm(nm, a, b)
                fn()
            L.profile_arm("NONE")
            torch.cuda.synchronize()
            out[nm] = round(1000.0 * statistics.mean(a.elapsed_time(b) for a, b in pairs), 2)
        return out

    def stream_ceiling():
        """The HBM -> LDS stream rate of the library's stream probe (the load path of the GEMM
        and attention kernels) over a 1 GiB buffer: with two workgroups per CU (the attainable
        rate the HBM-bound kernels are compared with) and with 32 workgroups (one CU's share)."""
        cus = torch.cuda.get_device_properties(0).multi_processor_count
        buf = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
        buf.fill_(1)

        def rate(views, wg, warm):
            """GB/s over the views, one probe each, after an untimed probe of `warm`"""
            L.stream_probe(warm, wg)
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(stream)
            for v in views:
                L.stream_probe(v, wg)
            b.record(stream)
            torch.cuda.synchronize()
            return sum(v.numel() for v in views) / (a.elapsed_time(b) * 1e-3) / 1e9

        full = rate([buf] * 5, 2 * cus, buf)     # 1 GiB a pass: four times the 256 MB MALL
        # one CU's share: 32 workgroups, each pass over a 128 MB range not read since the full passes
        sl = 32 * 4 * (1 << 20)
        one = rate([buf[r * sl:(r + 1) * sl] for r in range(5)], 32, buf[5 * sl:6 * sl])
        del buf
        log(f"stream probe: {full:.0f} GB/s with {2 * cus} workgroups; {one / 32:.1f} GB/s per CU (32 workgroups)")
        return dict(stream_gbps=round(full, 1), unit="GB/s", workgroups=2 * cus, bytes=1 << 30,
                    per_cu_gbps=round(one / 32, 2), peak=PEAK_HBM_GBS, frac_of_peak=round(full / PEAK_HBM_GBS, 4),
                    kernel="dcut_stream_probe: non-temporal buffer loads into LDS, 16 B per lane, 8 KB in flight per wave")

    def timed_region(fn, dominant):
        """`--steps` steps after `--warmup`, bracketed by synchronisations; the dominant kernel of
        every step timed by events on the launch stream (the library's hook)."""
        for _ in range(args.warmup):
            fn()
        torch.cuda.synchronize()
        kev = [(HookEvent(), HookEvent()) for _ in range(args.steps)] if dominant != "NONE" else [(None, None)] * args.steps
        start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        start.record(stream)
        for s in range(args.steps):
            if flush is not None:
                flush.fill_(1)
            L.profile_arm(dominant, kev[s][0], kev[s][1])
            fn()
        stop.record(stream)
        torch.cuda.synchronize()
        L.profile_arm("NONE")
        ms = start.elapsed_time(stop) / args.steps
        if dominant == "NONE":
            return ms, None
        return ms, 1000.0 * statistics.mean(a.elapsed_time(b) for a, b in kev)

    # ------------------------------------------------------------ the first seed: the full analysis
    seed0 = seeds[0]
    state = None
    if args.state and os.path.exists(args.state):
        state = json.load(open(args.state))
        assert state["workload"] == [cfg.cid, seed0] and state["budgets"] == budgets, "state mismatch"
        assert state.get("temperature", 0.0) == args.temperature, "state mismatch (temperature)"
        assert state.get("rs", False) == args.rs, "state mismatch (rs)"
        assert state.get("layers", 1) == args.layers, "state mismatch (layers)"
    vs, st, w, kv = setup(seed0, state)
    run_step = vs.step_rs if args.rs else vs.step
    if state is not None:
        cost_ms, acc_per_k = state["cost_row_ms"], state["accepted_per_budget"]
    elif args.force_k:
        cost_ms, acc_per_k = [1.0], [0]
    else:
        log("cost row: every candidate budget alone")
        cost_ms, acc_per_k = cost_row(vs)
    adaptive = lambda: run_step(budgets, cost_ms)
    breakdown = state["kernel_us"] if state is not None else kernel_breakdown(adaptive)
    # the dominant kernel by time per step: layer kernels launch once per decoder layer
    per_layer = {"GEMM_QKV", "ATTN", "ATTN_COMBINE", "GEMM_O", "GEMM_GATE_UP", "GEMM_DOWN", "MOE"}
    dominant = max(breakdown, key=lambda k: breakdown[k] * (args.layers if k in per_layer else 1))
    if args.state and state is None:
        json.dump(dict(workload=[cfg.cid, seed0], budgets=budgets, cost_row_ms=cost_ms, temperature=args.temperature,
                       rs=args.rs, layers=args.layers,
                       accepted_per_budget=acc_per_k, kernel_us=breakdown,
                       draft=vs.host("draft").tolist()), open(args.state, "w"))
    log("kernel us: " + ", ".join(f"{k}={v}" for k, v in breakdown.items()) + f"; dominant {dominant}")

    ms_per_step, dom_us = timed_region(adaptive, dominant)
    Kstar, rstar = vs.host("choice").tolist()
    accepted = int(vs.total.item())
    assert int(vs.dev_err.item()) == 0, "device data fault"
    log(f"seed {seed0}: {ms_per_step:.4f} ms per step, K*={Kstar}, {accepted} accepted")
    accept_len0 = vs.host("accept_len")
    draft0 = vs.host("draft")
    # per-step distribution (events around each step, outside the timed region); a
    # profiler replay of saved state runs the timed steps only
    step_dist, cold = None, None
    if state is None and not args.force_k:
        # each step bracketed by events, and its selection kernel timed by the hook (the
        # paper reports the selector's p50/p95 too)
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True), HookEvent(), HookEvent())
               for _ in range(100)]
        for a, b, sa, sb in evs:
            L.profile_arm("SELECT", sa, sb)
            a.record(stream)
            adaptive()
            b.record(stream)
        L.profile_arm("NONE")
        torch.cuda.synchronize()
        per_step = sorted(a.elapsed_time(b) for a, b, _, _ in evs)
        sel_us = sorted(1000.0 * sa.elapsed_time(sb) for _, _, sa, sb in evs)
        p95 = int(0.95 * len(per_step)) - 1
        step_dist = dict(median_ms=round(statistics.median(per_step), 4), p95_ms=round(per_step[p95], 4),
                         reps=len(per_step), select_median_us=round(statistics.median(sel_us), 2),
                         select_p95_us=round(sel_us[p95], 2))
    if flush is None and state is None and not args.force_k:
        # cold cache: a 512 MB write before each step evicts the 256 MB MALL (not timed)
        fl = torch.empty(512 << 20, dtype=torch.uint8, device="cuda")
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(20)]
        for a, b in evs:
            fl.fill_(1)
            a.record(stream)
            adaptive()
            b.record(stream)
        torch.cuda.synchronize()
        cms = statistics.median(a.elapsed_time(b) for a, b in evs)
        cold = dict(median_ms=round(cms, 4), tokens_per_s=round(int(vs.total.item()) / (cms * 1e-3), 1), reps=20)
        del fl
        log(f"per step: median {step_dist['median_ms']} ms, p95 {step_dist['p95_ms']} ms; "
            f"cold median {cms:.4f} ms")
    # the unpruned step (K = B(D+1)): per-kernel time and the GEMMs' MFMA rate, where the
    # verify-layer GEMMs are compute-bound
    unpruned = None
    if greedy_headline:
        Kfull = cfg.B * (cfg.D + 1)
        full = lambda: vs.step([Kfull], [1.0])
        ums = statistics.median(timed(full, args.cost_reps))
        ub = kernel_breakdown(full)
        gemms = {}
        for nm in ("GEMM_QKV", "GEMM_O", "GEMM_GATE_UP", "GEMM_DOWN", "LM_HEAD"):
            fl_, _ = kernel_work(nm, cfg, Kfull, st["ctx_len"])
            tf = fl_ / (ub[nm] * 1e-6) / 1e12
            gemms[nm] = dict(us=ub[nm], tflops=round(tf, 1), mfma_frac=round(tf / PEAK_BF16_TFLOPS, 4))
        ufr = {k: kernel_fraction(k, cfg, Kfull, st["ctx_len"], v) for k, v in ub.items()}
        unpruned = dict(K=Kfull, ms=round(ums, 4), accepted=int(vs.total.item()), kernel_us=ub, gemm_mfma=gemms,
                        kernel_roofline={k: v for k, v in ufr.items() if v is not None})
        log("unpruned step: " + f"{ums:.4f} ms; " + ", ".join(
            f"{k} {v['us']} us {v['mfma_frac']:.3f} of peak" for k, v in gemms.items()))
    graph = None
    if args.graph:
        g = vs.capture(adaptive)
        for _ in range(args.warmup):
            g.replay()
        torch.cuda.synchronize()
        ga, gb = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        ga.record(stream)
        for _ in range(args.steps):
            g.replay()
        gb.record(stream)
        torch.cuda.synchronize()
        gms = ga.elapsed_time(gb) / args.steps
        graph = dict(ms_per_step=round(gms, 4), tokens_per_s=round(int(vs.total.item()) / (gms * 1e-3), 1))
        log(f"graph replay: {gms:.4f} ms per step")
        del g
    table = None
    if args.cost_table:
        from paper_2607_14647_amd import costtable as ct
        import dataclasses as dc
        steps, keep = {}, []
        for Bc in (1, 8, 16, 32, 64):
            c2 = dc.replace(cfg, B=Bc, budgets=tuple(Bc * m for m in range(1, cfg.D + 2)))
            st2 = wl.make_step_inputs(c2, seed0)
            kv2 = wl.make_kv(c2, seed0, st2["ctx_len"])
            v2 = runner.VerifyStep(c2, None, st2, kv2, share_weights=vs)
            runner.force_drafts_on_device(v2, st2["draft"], st2["conf"], st2["match_u"])
            graphs = {}

            def run(budgets, v2=v2, graphs=graphs):
                K = budgets[0]
                if K not in graphs:
                    graphs[K] = v2.capture(lambda: v2.step([K], [1.0]))
                graphs[K].replay()
            steps[Bc] = run
            keep.append((v2, graphs))
        log("cost table: captured batch sizes 1, 8, 16, 32, 64 x ratios 25/50/75/100 %")
        t = ct.profile(steps, cfg.D, ct.PAPER_RATIOS, time_ms=ct.event_timer(stream), reps=10, warmup=2)
        table = dict(D=t.D, ratios=t.ratios, batch=t.batch, ms=[[round(x, 4) for x in r] for r in t.ms],
                     budgets={B: t.budgets(B) for B in t.batch},
                     nearest={B: t.row(B)[0] for B in (4, 12, 24, 40, 48, 100)})
        log("cost table (ms): " + "; ".join(f"B={B}: " + ", ".join(f"{x:.3f}" for x in r)
                                             for B, r in zip(t.batch, t.ms)))
        del keep, steps
    if args.copy_bytes > 0:
        src = torch.ones(args.copy_bytes, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    del vs
    torch.cuda.empty_cache()

    # ------------------------------------------------------------ further seeds: the headline protocol
    per_seed = [dict(seed=seed0, tokens_per_s=round(accepted / (ms_per_step * 1e-3), 1),
                     ms_per_step=round(ms_per_step, 4), K_star=Kstar, accepted=accepted)]
    for sd in seeds[1:]:
        v2, st2, _, _ = setup(sd, None)
        c2, _ = cost_row(v2)
        ms2, _ = timed_region(lambda: v2.step(budgets, c2), "NONE")
        K2 = int(v2.host("choice")[0])
        acc2 = int(v2.total.item())
        assert int(v2.dev_err.item()) == 0, "device data fault"
        per_seed.append(dict(seed=sd, tokens_per_s=round(acc2 / (ms2 * 1e-3), 1), ms_per_step=round(ms2, 4),
                             K_star=K2, accepted=acc2))
        log(f"seed {sd}: {ms2:.4f} ms per step, K*={K2}, {acc2} accepted")
        del v2
        torch.cuda.empty_cache()
    med = sorted(per_seed, key=lambda r: r["tokens_per_s"])[len(per_seed) // 2]
    value = med["tokens_per_s"]

    # algorithmic bytes per step (weights, KV read, KV append, packed in/out) of the first seed
    hd, nkv = ly.head_dim, ly.n_kv
    layer_w = sum(int(w[k].size) * 2 for k in w if k not in ("embed", "w_lm", "final_norm"))
    wbytes = layer_w * args.layers + int(w["w_lm"].size) * 2 + Kstar * ly.hidden * 2
    kvbytes = (float(st["ctx_len"].astype(np.int64).sum()) * nkv * hd * 4 + Kstar * nkv * hd * 4) * args.layers
    step_bytes = wbytes + kvbytes
    workload = f"cfg{cfg.cid}"
    rl = roofline(dominant, cfg, Kstar, st["ctx_len"], dom_us)
    rl["traffic"] = measured_traffic(dominant, workload, Kstar)
    rl["kernel"] = dominant
    rl["avg_us"] = round(dom_us, 2)
    fractions = {k: kernel_fraction(k, cfg, Kstar, st["ctx_len"], v) for k, v in breakdown.items()}
    fractions = {k: v for k, v in fractions.items() if v is not None}
    # the attainable stream rate (skipped in a profiler replay of saved state, which times the step only)
    attainable = stream_ceiling() if state is None else None
    if attainable is not None and rl["bound"] == "hbm":
        rl["frac_of_attainable"] = round(rl["achieved"] / attainable["stream_gbps"], 4)
    for k, f in fractions.items():
        fl, by = kernel_work(k, cfg, Kstar, st["ctx_len"])
        if attainable is not None and f["bound"] == "hbm":
            f["frac_of_attainable"] = round(by / (f["us"] * 1e-6) / 1e9 / attainable["stream_gbps"], 4)
    counted = counted_step_bytes(workload, Kstar, args.layers) if args.temperature == 0 else None
    fixed = {}
    for rho, m in (("0.25", 4), ("0.50", 8), ("0.75", 12), ("1.00", 16)):
        K = cfg.B * m
        if K in budgets and not args.force_k:
            j = budgets.index(K)
            fixed[rho] = dict(K=K, ms=round(cost_ms[j], 4), accepted=acc_per_k[j],
                              tokens_per_s=round(acc_per_k[j] / (cost_ms[j] * 1e-3), 1))
    seed_txt = f"median over seeds {seeds[0]}-{seeds[-1]}" if len(seeds) > 1 else f"seed {seed0}"
    out = dict(
        metric="accepted tokens/s of pruned verify step (1 layer + LM head), batch 64; HBM GB/s"
        if args.layers == 1 else
        f"accepted tokens/s of pruned verify step ({args.layers} layers + LM head), batch 64; HBM GB/s",
        value=round(value, 1), unit="tokens/s", n_gpus=1, steps=args.steps, warmup=args.warmup,
        ms_per_step=med["ms_per_step"], higher_is_better=True, scaling="weak", vs_baseline=None,
        dtype="bf16", data="synthetic",
        config=dict(workload=f"cfg{cfg.cid} {cfg.name}: B={cfg.B}, D={cfg.D}, H={ly.hidden}, "
                             f"{ly.n_q}q/{ly.n_kv}kv hd{ly.head_dim}, I={ly.inter}, V={ly.vocab}, "
                             f"L~{cfg.ctx}, conf {cfg.conf_model}; {seed_txt}",
                    global_batch=cfg.B, K_star=Kstar, r_star=rstar, accepted_per_step=accepted,
                    layers=args.layers, seeds=seeds,
                    budgets=budgets, parallelism="single GPU", cache="cold" if args.cold else "warm",
                    target_decoding="greedy" if args.temperature == 0 else
                    (f"rejection sampling at temperature {args.temperature} ("
                     + ("causal scan" if args.rs_budget == "scan" else "history-based budget")
                     + f" over shifted scores; seed {args.sample_seed})" if args.rs else
                     f"temperature {args.temperature} (Gumbel-max, seed {args.sample_seed})")),
        per_seed=per_seed,
        hbm_gbps=round(step_bytes / (ms_per_step * 1e-3) / 1e9, 1),
        step_algorithmic_bytes=int(step_bytes),
        hbm_counted=None if counted is None else dict(
            gbps=round(counted[0] / (ms_per_step * 1e-3) / 1e9, 1), bytes=int(counted[0]), kernels=counted[1]),
        roofline=rl,
        attainable=attainable,
        kernel_us=breakdown,
        kernel_roofline=fractions,
        unpruned=unpruned,
        step_ms=step_dist,
        cold=cold,
        cost_row_ms=[round(c, 4) for c in cost_ms],
        accepted_per_budget=acc_per_k,
        fixed_ratio=fixed,
        source_hash=source_hash(),
    )
    if graph is not None:
        out["graph"] = graph
    if table is not None:
        out["cost_table"] = table
    if not args.no_cpu_baseline and greedy_headline and seed0 == 0:
        cb = cpu_baseline(cfg, st, w, kv, budgets, cost_ms)
        # The oracle-forced acceptance of the sampled requests against the GPU's (seed 0, K*):
        # compared on every request whose oracle-forced drafts equal the GPU-forced ones and
        # whose deciding rows clear the argmax gap (a near-tie may flip either way in bf16)
        sample = cb.pop("sample_requests")
        zrows = cb.pop("draft_rows")
        per_req = cb.pop("oracle_accepted_per_request")
        same = [j for j, i in enumerate(sample) if np.array_equal(zrows[j], draft0[i])]
        cmp = [j for j in same if sample[j] not in cb["near_tie_requests"]]
        ora = int(sum(per_req[j] for j in cmp))
        gpu = int(sum(int(accept_len0[sample[j]]) + 1 for j in cmp))
        cb["acceptance_check"] = dict(requests=len(sample), drafts_equal=len(same), compared=len(cmp),
                                      oracle_accepted=ora, gpu_accepted=gpu,
                                      gpu_accepted_all=int(sum(int(accept_len0[i]) + 1 for i in sample)))
        log(f"cpu baseline: acceptance on {len(cmp)} of {len(sample)} requests: oracle-forced {ora}, GPU {gpu}")
        assert ora == gpu, "oracle-forced acceptance differs from the GPU step"
        out["cpu_baseline"] = cb
    else:
        out["cpu_baseline"] = None
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
