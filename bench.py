"""Benchmark of the shifted-window attention hot path on one MI355X.

One step = one pass of the whole path over one synthetic batch, with the
token route fused into the attention kernels (NHWC read and written in
place):
  attention forward (O, LSE)                terra_winattn_fwd_nhwc
  attention backward (dQ, dK, dV, dTable)   terra_winattn_bwd_nhwc
Inputs are resident in HBM before timing starts.  W warm-up steps, then K
timed steps between device synchronisations; every launch is bracketed by
HIP events on the stream it runs on.  The same K steps are then run with
the unfused pipeline (route Q, K, V, dO; window-major forward and
backward; inverse route of O, dQ, dK, dV), which also gives the standalone
routing bandwidth.

The printed JSON line's `value` is the attention forward+backward
algorithmic TFLOP/s of the fused step (flops 12 n^2 hd per window and
head, divided by the full step time); per-phase figures, the roofline of
the dominant kernel, the unfused pipeline and the oracle CPU baseline ride
along.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--config NAME]
"""

import argparse
import json
import os
import platform
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import terra_synth as ts  # noqa: E402

METRIC = "Swin window-attn fwd+bwd TFLOP/s (% MFMA peak); routing GB/s (% HBM)"
PEAK_BF16_TFLOPS = 2500.0     # MI355X dense bf16 / fp16 MFMA
PEAK_F32_TFLOPS = 157.3       # MI355X fp32 matrix
PEAK_HBM_GBPS = 8000.0        # MI355X HBM3E
DEFAULT_CONFIG = "c4_bf16_128x1080_w8x16"


def window_sizes(cfg):
    mh, mw = -(-cfg.H // cfg.wh), -(-cfg.W // cfg.ww)
    rows = [min(cfg.wh, cfg.H - i * cfg.wh) for i in range(mh)]
    cols = [min(cfg.ww, cfg.W - j * cfg.ww) for j in range(mw)]
    return [r * c for r in rows for c in cols]


def algorithmic(cfg):
    """Flops and compulsory HBM bytes per launch of each phase."""
    e = 4 if cfg.dtype == "f32" else 2
    ns = np.asarray(window_sizes(cfg), np.float64)
    n2 = float((ns ** 2).sum()) * cfg.B * cfg.heads
    tok = cfg.B * cfg.H * cfg.W
    t = tok * cfg.C * e                        # one tensor
    lse = tok * cfg.heads * 4
    tab = (2 * cfg.wh - 1) * (2 * cfg.ww - 1) * cfg.heads * 4
    return {
        "fwd_flops": 4.0 * n2 * cfg.head_dim,
        "bwd_flops": 8.0 * n2 * cfg.head_dim,
        "route_bytes": 2.0 * t,                                  # read + write one tensor
        "fwd_bytes": 4.0 * t + lse + tab,                        # Q,K,V in; O, LSE out
        "bwd_bytes": 7.0 * t + lse + 2 * tab,                    # Q,K,V,dO,LSE in; dQ,dK,dV,dT out
    }


# HBM bytes per launch measured with two rocprofv3 passes (FETCH_SIZE, then
# WRITE_SIZE; FETCH_SIZE scaled by 1.9996 and WRITE_SIZE by 1.0000, the
# factors a plain copy of known size reads on the same run) on the 128x1080
# workload, for the fused kernels (backward: bwd_win_kernel + dtab_reduce).
# A figure is reported only while the kernel sources (the window kernels and
# the file holding the bias-table reduction) still have the SHA-256 prefixes
# they were measured with.
MEASURED_TRAFFIC = {
    ("c4_bf16_128x1080_w8x16", "bwd_nhwc"): dict(sources={"attn_win.hip": "ddf24dfca1bc3171", "dtab.hip": "a443188e370c52f5"},
                                                bytes=(437550.9 + 556.3) * 1024 * 1.9996 + (625295.8 + 303.6) * 1024),
    ("c4_bf16_128x1080_w8x16", "fwd_nhwc"): dict(sources={"attn_win.hip": "ddf24dfca1bc3171"},
                                                bytes=311299.1 * 1024 * 1.9996 + 224292.1 * 1024),
}


def measured_traffic(cfg_name, phase):
    import hashlib
    ent = MEASURED_TRAFFIC.get((cfg_name, phase))
    if ent is None:
        return None
    for name, prefix in ent["sources"].items():
        path = os.path.join(ROOT, "paper_2608_15211_amd", "csrc", name)
        if not hashlib.sha256(open(path, "rb").read()).hexdigest().startswith(prefix):
            return None
    return ent["bytes"]


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor() or platform.machine()


def cpu_baseline(cfg, seconds_target=8.0, repeats=3):
    """Time the fp64 oracle (as it stands) on a bounded sample of windows:
    the sample is grown until one pass costs about seconds_target, then
    timed `repeats` times; the median is reported."""
    import threadpoolctl
    from oracle import Geometry, route, attn_fwd_windows, attn_bwd_windows
    from oracle.geometry import window_slots

    g = Geometry(**cfg.geom_kwargs())
    inp = ts.make_inputs(cfg)
    slots = window_slots(g)
    rng = np.random.default_rng(1)
    t0 = time.perf_counter()
    q, k, v, do = (route(inp[n], g) for n in ("q", "k", "v", "dout"))
    t_route = (time.perf_counter() - t0) / 4.0
    info = threadpoolctl.threadpool_info()
    threads = max([i.get("num_threads", 1) for i in info] + [1])

    def one(sel):
        t0 = time.perf_counter()
        attn_fwd_windows(q, k, v, inp["table"], g, sel)
        attn_bwd_windows(q, k, v, do, inp["table"], g, sel)
        return time.perf_counter() - t0

    nsel = 256      # each pass also converts whole tensors (about 2 s on c4), so start large
    while True:
        sel = sorted(int(x) for x in rng.choice(len(slots), size=min(nsel, len(slots)), replace=False))
        dt = one(sel)
        if dt >= seconds_target * 0.6 or nsel >= len(slots):
            break
        nsel = min(len(slots), int(nsel * max(1.2, seconds_target / max(dt, 1e-3))))
    times = sorted([dt] + [one(sel) for _ in range(repeats - 1)])
    sample_time = times[len(times) // 2]
    n2 = sum(float(slots[w][2]) ** 2 for w in sel) * cfg.B * cfg.heads
    sample_flops = 12.0 * n2 * cfg.head_dim
    e = 4 if cfg.dtype == "f32" else 2
    route_gbps = 2.0 * cfg.B * cfg.H * cfg.W * cfg.C * e / t_route / 1e9
    return {
        "value": sample_flops / sample_time / 1e12,
        "unit": "TFLOP/s",
        "cores": int(threads),
        "kind": "oracle",
        "sample": "fp64 oracle fwd+bwd on %d of %d windows x %d heads, median of %d passes "
                  "(%.1f s each); route of 4 full tensors %.1f GB/s; host %s, %d logical CPUs, "
                  "%d BLAS threads" % (
                      len(sel), len(slots), cfg.heads, repeats, sample_time, route_gbps,
                      cpu_model(), os.cpu_count(), threads),
        "route_GBps": route_gbps,
    }


def time_block(cfg, args, dev, flush):
    """The whole Swin block (LayerNorm, QKV projection, attention, output
    projection, MLP; forward then backward) on the same grid, timed like the
    attention step.  Flops: the four linear layers' 24 T C^2 forward and
    48 T C^2 backward (T tokens) plus the attention's 12 n^2 hd per window
    and head."""
    import torch
    import paper_2608_15211_amd as P

    print("bench: Swin block inputs", file=sys.stderr, flush=True)
    inp = ts.make_block_inputs(cfg)
    x = torch.from_numpy(inp["x"]).to(dev).to(torch.bfloat16)
    dx2 = torch.from_numpy(inp["dx2"]).to(dev).to(torch.bfloat16)
    params = {n: torch.from_numpy(v).to(dev).to(torch.bfloat16 if n.startswith("w_") else torch.float32)
              for n, v in inp["params"].items()}
    table = torch.from_numpy(inp["table"]).to(dev)
    del inp
    saved = P.terra_block_saved_alloc(cfg, dev)
    x2 = torch.empty_like(x)
    shapes = {n: params[n].shape for n in params}
    out = (torch.empty_like(x), {n: torch.empty(shapes[n], dtype=torch.float32, device=dev) for n in params},
           torch.empty_like(table))
    ws = torch.empty(P.terra_block_bwd_workspace_bytes(cfg), dtype=torch.uint8, device=dev)
    fws = torch.empty(P.terra_block_fwd_workspace_bytes(cfg), dtype=torch.uint8, device=dev)

    def fwd():
        P.terra_block_fwd(x, params, table, cfg, saved=saved, out=x2, workspace=fws)

    def bwd():
        P.terra_block_bwd(dx2, x, params, table, cfg, saved, out=out, workspace=ws)

    for _ in range(max(2, args.warmup // 5)):
        fwd()
        bwd()
    torch.cuda.synchronize()
    tf, tb = [], []
    for _ in range(max(5, args.steps // 2)):
        flush()
        e0, e1, e2 = (torch.cuda.Event(enable_timing=True) for _ in range(3))
        e0.record()
        fwd()
        e1.record()
        bwd()
        e2.record()
        tf.append(e0)
        tb.append((e1, e2))
    torch.cuda.synchronize()
    fwd_ms = float(np.median([a.elapsed_time(b) for a, (b, _) in zip(tf, tb)]))
    bwd_ms = float(np.median([b.elapsed_time(c) for b, c in tb]))
    T, C = cfg.B * cfg.H * cfg.W, cfg.C
    alg = algorithmic(cfg)
    lin_f, lin_b = 24.0 * T * C * C, 48.0 * T * C * C
    fl_f, fl_b = lin_f + alg["fwd_flops"], lin_b + alg["bwd_flops"]
    peak = PEAK_BF16_TFLOPS
    tot = (fl_f + fl_b) / ((fwd_ms + bwd_ms) * 1e-3) / 1e12
    print("bench: Swin block timed", file=sys.stderr, flush=True)
    return {"fwd_ms": round(fwd_ms, 4), "bwd_ms": round(bwd_ms, 4),
            "step_ms": round(fwd_ms + bwd_ms, 4),
            "tflops": round(tot, 1), "frac_mfma_peak": round(tot / peak, 4),
            "fwd_tflops": round(fl_f / (fwd_ms * 1e-3) / 1e12, 1),
            "bwd_tflops": round(fl_b / (bwd_ms * 1e-3) / 1e12, 1),
            "flops_per_step": fl_f + fl_b,
            "note": "LayerNorm + QKV + attention + projection + GELU MLP (ratio 4), forward and backward; "
                    "medians of the timed steps"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=50)
    ap.add_argument("--config", default=DEFAULT_CONFIG, choices=list(ts.ALL))
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-block", action="store_true", help="skip the Swin-block timing")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the attention path has no multi-GPU leg "
              "(it would shard by windows and heads, exchanging only boundary rows); run with --gpus 1",
              file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2608_15211_amd as P

    cfg = ts.ALL[args.config]
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    tdt = {"f32": torch.float32, "bf16": torch.bfloat16, "f16": torch.float16}[cfg.dtype]
    print("bench: generating %s inputs" % cfg.name, file=sys.stderr, flush=True)
    inp = ts.make_inputs(cfg)
    x = {n: torch.from_numpy(inp[n]).to(dev).to(tdt) for n in ("q", "k", "v", "dout")}
    table = torch.from_numpy(inp["table"]).to(dev)
    del inp
    shape_w = (cfg.B, cfg.H * cfg.W, cfg.C)
    w = {n: torch.empty(shape_w, dtype=tdt, device=dev) for n in ("q", "k", "v", "dout")}
    o = torch.empty(shape_w, dtype=tdt, device=dev)
    lse = torch.empty((cfg.B, cfg.heads, cfg.H * cfg.W), dtype=torch.float32, device=dev)
    grads = (torch.empty(shape_w, dtype=tdt, device=dev), torch.empty(shape_w, dtype=tdt, device=dev),
             torch.empty(shape_w, dtype=tdt, device=dev), torch.empty_like(table))
    back = {n: torch.empty((cfg.B, cfg.H, cfg.W, cfg.C), dtype=tdt, device=dev)
            for n in ("o", "dq", "dk", "dv")}
    ws = torch.empty(max(1, P.terra_winattn_bwd_workspace_bytes(cfg, tdt)), dtype=torch.uint8, device=dev)
    # shapes on the general kernels keep O's rounding residual for the
    # backward's D (no extra sweep over the keys); None elsewhere
    uses_lo = P.terra_winattn_uses_o_lo(cfg, tdt)
    o_lo = torch.empty((cfg.B, cfg.H, cfg.W, cfg.C), dtype=tdt, device=dev) if uses_lo else None
    o_lo_w = torch.empty(shape_w, dtype=tdt, device=dev) if uses_lo else None

    fused_phases = ["fwd", "bwd"]
    unfused_phases = ["route", "fwd_wm", "bwd_wm", "unroute"]

    def rec(ev, name, fn):
        if ev is not None:
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            fn()
            b.record()
            ev[name].append((a, b))
        else:
            fn()

    def step(ev):
        rec(ev, "fwd", lambda: P.terra_winattn_fwd_nhwc(x["q"], x["k"], x["v"], table, cfg,
                                                         out=back["o"], lse=lse, o_lo=o_lo))
        rec(ev, "bwd", lambda: P.terra_winattn_bwd_nhwc(x["q"], x["k"], x["v"], back["o"], x["dout"],
                                                         lse, table, cfg, workspace=ws,
                                                         out=(back["dq"], back["dk"], back["dv"],
                                                              grads[3]), o_lo=o_lo))

    def step_unfused(ev):
        for n in ("q", "k", "v"):
            rec(ev, "route", lambda n=n: P.terra_window_route(x[n], cfg, out=w[n]))
        rec(ev, "fwd_wm", lambda: P.terra_winattn_fwd(w["q"], w["k"], w["v"], table, cfg, out=o, lse=lse,
                                                      o_lo=o_lo_w))
        rec(ev, "route", lambda: P.terra_window_route(x["dout"], cfg, out=w["dout"]))
        rec(ev, "bwd_wm", lambda: P.terra_winattn_bwd(w["q"], w["k"], w["v"], o, w["dout"], lse, table, cfg,
                                                      out=grads, workspace=ws, o_lo=o_lo_w))
        for n, t in (("o", o), ("dq", grads[0]), ("dk", grads[1]), ("dv", grads[2])):
            rec(ev, "unroute", lambda n=n, t=t: P.terra_window_unroute(t, cfg, out=back[n]))

    # Between timed steps (outside the step's events) a 1 GiB buffer is
    # overwritten and then a second 1 GiB buffer is read, so that no step
    # finds the previous one's tensors in the 256 MB last-level cache (MALL).
    # The read matters: after the write alone the cache is full of dirty
    # lines, and their write-back lands inside the next step (the 128 x 1080
    # forward measured 0.268 ms after a write-only flush, 0.217 ms after write + read
    # or a read alone, 0.218 ms with no flush).
    flush_w = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
    flush_r = torch.ones(1 << 28, dtype=torch.float32, device=dev)
    flush_sink = torch.empty((), dtype=torch.float32, device=dev)

    def flush():
        flush_w.zero_()
        torch.sum(flush_r, dim=0, out=flush_sink)

    def timed(fn, phases):
        print("bench: warm-up %d steps" % args.warmup, file=sys.stderr, flush=True)
        for _ in range(args.warmup):
            fn(None)
        torch.cuda.synchronize()
        ev = {p: [] for p in phases}
        marks = []
        torch.cuda.synchronize()
        for _ in range(args.steps):
            flush()
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            fn(ev)
            b.record()
            marks.append((a, b))
        torch.cuda.synchronize()
        print("bench: timed %d steps" % args.steps, file=sys.stderr, flush=True)
        steps_ms = [a.elapsed_time(b) for a, b in marks]
        launches = {p: [a.elapsed_time(b) for a, b in ev[p]] for p in phases}
        per_launch = {p: float(np.mean(launches[p])) for p in phases}
        per_step = {p: float(np.sum(launches[p])) / args.steps for p in phases}
        return float(np.median(steps_ms)), float(np.mean(steps_ms)), per_launch, per_step

    # The unfused pipeline (a secondary figure) is timed first: its steps
    # leave the device running rather than idle when the fused step's W
    # warm-up steps start (a fresh process needs tens of milliseconds of work
    # before clocks and translation caches settle; with 5 warm-up steps and
    # nothing before them the 128 x 1080 fused step measured 0.859 ms, with
    # 30 0.794 ms).
    ms_unf, _, pl_unf, ps_unf = timed(step_unfused, unfused_phases)
    ms_step, ms_step_mean, per_launch, per_step = timed(step, fused_phases)

    alg = algorithmic(cfg)
    attn_flops = alg["fwd_flops"] + alg["bwd_flops"]
    peak = PEAK_F32_TFLOPS if cfg.dtype == "f32" else PEAK_BF16_TFLOPS
    value = attn_flops / (ms_step * 1e-3) / 1e12
    attn_ms = per_step["fwd"] + per_step["bwd"]
    attn_tflops = attn_flops / (attn_ms * 1e-3) / 1e12
    ai = attn_flops / (alg["fwd_bytes"] + alg["bwd_bytes"])
    attainable = min(peak, ai * PEAK_HBM_GBPS / 1e3)
    route_gbps = alg["route_bytes"] / (pl_unf["route"] * 1e-3) / 1e9
    unroute_gbps = alg["route_bytes"] / (pl_unf["unroute"] * 1e-3) / 1e9

    # dominant kernel of the step (by time per step) -> roofline object: HBM
    # bound below the ridge point (peak flops / peak bandwidth), matrix-core
    # bound above it
    unit_bytes = {"fwd": alg["fwd_bytes"], "bwd": alg["bwd_bytes"]}
    unit_flops = {"fwd": alg["fwd_flops"], "bwd": alg["bwd_flops"]}
    dom = max(fused_phases, key=lambda p: per_step[p])
    traffic = measured_traffic(cfg.name, dom + "_nhwc")
    if unit_flops[dom] / unit_bytes[dom] > peak * 1e12 / (PEAK_HBM_GBPS * 1e9):
        achieved = unit_flops[dom] / (per_launch[dom] * 1e-3) / 1e12
        roofline = {"bound": "mfma", "achieved": round(achieved, 1), "peak": peak,
                    "unit": "TFLOP/s", "frac": round(achieved / peak, 4),
                    "algorithmic_flops_per_launch": unit_flops[dom]}
    else:
        achieved = unit_bytes[dom] / (per_launch[dom] * 1e-3) / 1e9
        roofline = {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBPS,
                    "unit": "GB/s", "frac": round(achieved / PEAK_HBM_GBPS, 4),
                    "algorithmic_bytes_per_launch": unit_bytes[dom]}
    roofline.update({"traffic": None if traffic is None else round(traffic),
                     "kernel": {"fwd": "terra_winattn_fwd_nhwc", "bwd": "terra_winattn_bwd_nhwc"}[dom],
                     "avg_launch_ms": round(per_launch[dom], 4)})

    line = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "ms_per_step_mean": round(ms_step_mean, 4),
        "step_statistic": "median of the timed steps; between steps, outside the step, a 1 GiB write then a 1 GiB read flush the caches",
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg.dtype,
        "data": "synthetic",
        "config": {"workload": cfg.name, "B": cfg.B, "grid": [cfg.H, cfg.W], "C": cfg.C,
                   "heads": cfg.heads, "head_dim": cfg.head_dim, "window": [cfg.wh, cfg.ww],
                   "shift": [cfg.sh, cfg.sw], "route": "fused", "parallelism": "single-gpu"},
        "roofline": roofline,
        "attn": {"fwd_ms": round(per_step["fwd"], 4), "bwd_ms": round(per_step["bwd"], 4),
                 "tflops_kernels_only": round(attn_tflops, 2),
                 "frac_mfma_peak": round(attn_tflops / peak, 4),
                 "attainable_tflops": round(attainable, 1),
                 "frac_attainable": round(attn_tflops / attainable, 4),
                 "fwd_hbm_GBps": round(alg["fwd_bytes"] / (per_launch["fwd"] * 1e-3) / 1e9, 1),
                 "bwd_hbm_GBps": round(alg["bwd_bytes"] / (per_launch["bwd"] * 1e-3) / 1e9, 1)},
        "routing": {"route_ms": round(pl_unf["route"], 4), "route_GBps": round(route_gbps, 1),
                    "route_frac_hbm": round(route_gbps / PEAK_HBM_GBPS, 4),
                    "unroute_ms": round(pl_unf["unroute"], 4),
                    "unroute_GBps": round(unroute_gbps, 1),
                    "unroute_frac_hbm": round(unroute_gbps / PEAK_HBM_GBPS, 4)},
        "unfused": {"ms_per_step": round(ms_unf, 4),
                    "value": round(attn_flops / (ms_unf * 1e-3) / 1e12, 2),
                    "fwd_ms": round(ps_unf["fwd_wm"], 4), "bwd_ms": round(ps_unf["bwd_wm"], 4),
                    "route_ms_per_step": round(ps_unf["route"] + ps_unf["unroute"], 4)},
    }
    if not args.no_block and cfg.dtype == "bf16" and cfg.C % 128 == 0 and cfg.C <= 2048:
        line["swin_block"] = time_block(cfg, args, dev, flush)
    if not args.no_cpu_baseline:
        print("bench: timing the oracle on a sample", file=sys.stderr, flush=True)
        cb = cpu_baseline(cfg)
        line["cpu_baseline"] = {k: cb[k] for k in ("value", "unit", "cores", "kind", "sample")}
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
