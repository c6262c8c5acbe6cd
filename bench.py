#!/usr/bin/env python3
"""Benchmark of the 4-direction GSPN line scan (forward + backward) on one MI355X.

One step = the forward and backward passes over one batch of the workload,
with every input already resident in HBM and every tensor pixel-major (the
layout of the C ABI's plain entry points), through the training pair
gspn_scan_fwd_train + gspn_scan_bwd_reserve (the forward leaves in a reserve
the blocked copies its backward reads; forward-only workloads use
gspn_scan_fwd).  The plain pair gspn_scan_fwd + gspn_scan_bwd and the _blocked
entry points (per-direction tensors in their scan order) are timed beside it
and reported under "plain" and "blocked".  With --norm the weights are given
as logits and the calls are the _norm pairs (gspn_scan_fwd_norm_train +
gspn_scan_bwd_norm_reserve, the plain _norm pair beside it).  Prints ONE
JSON line on stdout:
throughput in G pixel-channels per second (B*C*H*W per step), the roofline
of the dominant kernel (algorithmic bytes / average launch time, from HIP
events on the launch stream) and the CPU oracle timed on a bounded sample of
the same workload.  Diagnostics go to stderr.

    python bench.py [--steps K] [--warmup W] [--workload IDX|NAME|all] [--no-cpu-baseline]
                    [--layout pixel|blocked] [--no-blocked] [--norm] [--latent IDX|NAME|all]

Before every step, outside the timed events, reading a 1 GiB buffer evicts
the L2s and the 256 MB Infinity Cache (writing back what the previous step
left dirty), so every step reads its inputs from HBM: the small workloads
would otherwise run from cache.  Step time is then the sum of the
two calls' event times.  A device-to-device copy that moves the dominant
call's algorithmic byte count, timed the same way, gives the achievable
bandwidth; the share of the call's time it does not explain is reported as
the serialisation share.  `--workload all` prints one line per workload.

`--latent` times the latent-space sublayer of C-GSPN instead (gspn_latent_fwd:
P_down, the parameter product, the scan over the latent channels, P_up), one
step being one forward call; each stage is also timed on its own through the
public entry points (the parameter product and the scan on the sublayer's
latent grid), and the roofline is that of the slowest stage.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

import gspn_inputs as gi  # noqa: E402

HBM_PEAK_GBS = 8000.0     # MI355X HBM3E, published peak
METRIC = "GSPN scan fwd+bwd Gpix·ch/s at 1 MI355X; achieved HBM GB/s vs peak"


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def algorithmic_bytes(wl: gi.Workload) -> dict:
    """Compulsory HBM bytes: each input read once, each output written once.

    forward  : x, lam_d, u_d, w_d in; y out           s*N*[C(2+2D) + 3GD]
    backward : x, dy, lam_d, u_d, w_d in;
               dx, dlam_d, du_d, dw_d out            s*N*[C(3+4D) + 6GD]
    with N = B*H*W, D directions, s bytes per stored element.
    """
    s = 4 if wl.dtype == "f32" else 2
    N = wl.B * wl.H * wl.W
    D = wl.ndirs
    fwd = s * N * (wl.C * (2 + 2 * D) + 3 * wl.G * D)
    bwd = s * N * (wl.C * (3 + 4 * D) + 6 * wl.G * D)
    return {"fwd": fwd, "bwd": bwd if wl.backward else 0}


def to_device(a, dtype, torch):
    if dtype == "bf16":
        return torch.from_numpy(gi.to_bf16_bits(a).view(np.int16)).to("cuda").view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to("cuda")


def _cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown CPU"


CPU_SHARE = 16   # host threads that one GPU's jobs may use on a shared GPU host


def cpu_threads() -> int:
    """Threads of the CPU baseline: the cores this process may run on,
    at most CPU_SHARE."""
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    return max(1, min(n, CPU_SHARE))


def cpu_baseline(wl: gi.Workload, inputs: dict, min_seconds: float, norm: bool = False,
                 threads: int = 1, runs: int = 3) -> dict:
    """The fp64 oracle on (batch, group) units of the workload.

    `runs` runs, each over the same sample of units: all their forward passes
    (spread over `threads` threads; the oracle's C calls release the
    interpreter lock, so they run side by side), then all their backward
    passes, each phase timed on its own.  The sample is sized so that the runs
    take about `min_seconds` in all.  Reported: the median over the runs of
    the throughput (B*C*H*W of the sample over forward + backward time) and
    the medians of the two phases.
    """
    import concurrent.futures as cf

    import oracle
    cpg = wl.C // wl.G
    order = [(b, g) for g in range(wl.G) for b in range(wl.B)]
    slices = {}

    def sl(bg):
        if bg not in slices:
            b, g = bg
            s_ = oracle.slice_group(inputs, b, g, wl.G)
            s_["wn"] = oracle.normalize_w(s_["w"], wl.dirs) if norm else s_["w"]
            slices[bg] = s_
        return slices[bg]

    def fwd(bg):
        s_ = sl(bg)
        oracle.scan_fwd(s_["x"], s_["wn"], s_["lam"], s_["u"], wl.dirs)

    def bwd(bg):
        s_ = sl(bg)
        r = oracle.scan_bwd(s_["x"], s_["wn"], s_["lam"], s_["u"], s_["dy"], wl.dirs)
        if norm:
            oracle.normalize_w_bwd(s_["w"], r["dw"], wl.dirs)

    def phase(ex, fn, units):
        t0 = time.perf_counter()
        list(ex.map(fn, units))
        return time.perf_counter() - t0

    with cf.ThreadPoolExecutor(max_workers=threads) as ex:
        # size the sample: one unit per thread, timed once, sets the count
        probe = order[:threads]
        for bg in probe:
            sl(bg)
        # (the first pass also warms the oracle and the threads: time the second)
        phase(ex, fwd, probe)
        t1 = phase(ex, fwd, probe) + (phase(ex, bwd, probe) if wl.backward else 0.0)
        per_round = max(t1, 1e-6)
        rounds = max(1, int(min_seconds / runs / per_round))
        units = [order[k % len(order)] for k in range(rounds * threads)]
        for bg in units:
            sl(bg)
        # one untimed run at that size corrects the estimate (threads contend
        # for memory bandwidth more over many units than over one each)
        t_run = phase(ex, fwd, units) + (phase(ex, bwd, units) if wl.backward else 0.0)
        rounds = max(1, int(rounds * min_seconds / runs / max(t_run, 1e-6)))
        units = [order[k % len(order)] for k in range(rounds * threads)]
        for bg in units:
            sl(bg)
        tf, tb = [], []
        for _ in range(runs):
            tf.append(phase(ex, fwd, units))
            tb.append(phase(ex, bwd, units) if wl.backward else 0.0)
    pixch = len(units) * cpg * wl.H * wl.W
    rates = sorted(pixch / (f + b) / 1e9 for f, b in zip(tf, tb))
    how = "single thread" if threads == 1 else f"{threads} threads"
    med = lambda v: float(sorted(v)[len(v) // 2])     # noqa: E731
    return {"value": round(rates[len(rates) // 2], 6), "unit": "Gpix·ch/s", "cores": threads,
            "kind": "oracle",
            "fwd_s": round(med(tf), 4), "bwd_s": round(med(tb), 4), "runs": runs,
            "host_nproc": os.cpu_count(),
            "sample": f"{len(units)} (batch, group) units of {wl.name} ({wl.B * wl.G} per step; "
                      f"{len(units) * cpg} channel planes), fwd then bwd, each timed, median of "
                      f"{runs} runs, fp64, {how} ({os.cpu_count()} host CPUs, at most "
                      f"{CPU_SHARE} used: one GPU's share; {_cpu_model()}), "
                      f"{sum(tf) + sum(tb):.1f} s"}


def timed_copy(nbytes: int, reps: int, flush, torch) -> float:
    """Mean ms of a device-to-device copy that reads and writes nbytes / 2 each."""
    n = max(1, nbytes // 8)
    src = torch.ones(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    dst.copy_(src)
    ms = []
    for _ in range(reps):
        flush()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        dst.copy_(src)
        e1.record()
        torch.cuda.synchronize()
        ms.append(e0.elapsed_time(e1))
    del src, dst
    return float(np.mean(ms))


def run_workload(wl: gi.Workload, args, torch, gspn) -> dict:
    log(f"workload {wl}")
    t0 = time.perf_counter()
    inputs = gi.make_inputs(wl, with_dy=wl.backward)
    if args.norm:
        # the weights as logits: the calls form the row-stochastic weights
        inputs["w"] = gi.make_logits(wl)
    log(f"inputs generated in {time.perf_counter() - t0:.1f} s")
    stream = torch.cuda.current_stream()
    scrub = (torch.ones(args.flush_mib * (1 << 20) // 4, dtype=torch.float32, device="cuda")
             if args.flush_mib > 0 else None)
    train = main_is_train(wl, args, gspn)
    main = time_step(wl, inputs, args, torch, gspn, args.layout, scrub, stream, train=train)
    others = []
    if not args.no_blocked:
        if train:
            others.append(time_step(wl, inputs, args, torch, gspn, gspn.PIXEL, scrub, stream))
    if not args.norm and not args.no_blocked:
        others.append(time_step(wl, inputs, args, torch, gspn,
                                gspn.BLOCKED if args.layout == gspn.PIXEL else gspn.PIXEL, scrub,
                                stream))
    return summarize(wl, inputs, args, torch, main, others, scrub)


def main_is_train(wl, args, gspn) -> bool:
    """The headline step runs the training pair (with --norm, the one that
    takes logits): pixel-major, a backward pass, and not turned off with
    --plain."""
    return wl.backward and args.layout == gspn.PIXEL and not args.plain


def time_step(wl, inputs, args, torch, gspn, layout, scrub, stream, train=False) -> dict:
    """Event times of K steps with the per-direction tensors in `layout`
    (with `train`, through the training pair and its reserve)."""
    host = gi.inputs_line_major(inputs, wl.dirs) if layout == gspn.BLOCKED else inputs
    dev = {k: to_device(v, wl.dtype, torch) for k, v in host.items()}
    x, w, lam, u = dev["x"], dev["w"], dev["lam"], dev["u"]
    kw = {} if args.norm else {"layout": layout}
    fwd_call = gspn.scan_fwd_norm if args.norm else gspn.scan_fwd
    bwd_call = gspn.scan_bwd_norm if args.norm else gspn.scan_bwd
    if train:
        # the reserve, like the workspace, is taken once: a training loop keeps it
        nrs = gspn.reserve_size(dev["x"], dev["w"], wl.dirs, norm=args.norm)
        rsv = torch.empty(max(nrs, 1), dtype=torch.uint8, device="cuda")
        log(f"training pair: reserve {nrs} bytes")
        fwd_train = gspn.scan_fwd_norm_train if args.norm else gspn.scan_fwd_train
        bwd_reserve = gspn.scan_bwd_norm_reserve if args.norm else gspn.scan_bwd_reserve

        def fwd_call(x, w, lam, u, dirs, y, stream, workspace):
            fwd_train(x, w, lam, u, dirs, y=y, reserve=rsv, stream=stream, workspace=workspace)

        def bwd_call(x, w, lam, u, dy, dirs, out, stream, workspace):
            bwd_reserve(x, w, lam, u, dy, rsv, dirs, out=out, stream=stream, workspace=workspace)
        kw = {}
    y = torch.empty_like(x)
    if wl.backward:
        dy = dev["dy"]
        grads = (torch.empty_like(x), torch.empty_like(w), torch.empty_like(lam),
                 torch.empty_like(u))
    # the calls' workspace, taken once (a caller that keeps it allocates nothing per call)
    ops = ((gspn.OP_FWD_NORM_TRAIN, gspn.OP_BWD_NORM_RESERVE) if args.norm and train else
           (gspn.OP_FWD_NORM, gspn.OP_BWD_NORM) if args.norm else
           (gspn.OP_FWD_TRAIN, gspn.OP_BWD_RESERVE) if train else
           (gspn.OP_FWD, gspn.OP_BWD) if layout == gspn.PIXEL else
           (gspn.OP_FWD_BLOCKED, gspn.OP_BWD_BLOCKED))
    nws = max(gspn.workspace_size(op, x, w, wl.dirs) for op in ops)
    ws = torch.empty(max(nws, 1), dtype=torch.uint8, device="cuda")
    log(f"layout {layout}: workspace {nws} bytes")

    def flush():
        # read, not write: the caches end up holding clean lines, so the timed
        # calls do not pay for writing back the flush's own data
        if scrub is not None:
            scrub.sum()

    def step(ev=None):
        flush()
        if ev is not None:
            ev[0].record(stream)
        fwd_call(x, w, lam, u, wl.dirs, y=y, stream=stream, workspace=ws, **kw)
        if ev is not None:
            ev[1].record(stream)
        if wl.backward:
            bwd_call(x, w, lam, u, dy, wl.dirs, out=grads, stream=stream, workspace=ws, **kw)
        if ev is not None:
            ev[2].record(stream)

    if args.copy_calibration > 0:
        n = args.copy_calibration * (1 << 20) // 4
        src = torch.ones(n, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        log(f"copy calibration: {n * 4} bytes read, {n * 4} bytes written")
        del src, dst

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    events = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(args.steps):
        step(events[k])
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0

    fwd_ms = float(np.mean([e[0].elapsed_time(e[1]) for e in events]))
    bwd_ms = float(np.mean([e[1].elapsed_time(e[2]) for e in events])) if wl.backward else 0.0
    fwd_med = float(np.median([e[0].elapsed_time(e[1]) for e in events]))
    bwd_med = (float(np.median([e[1].elapsed_time(e[2]) for e in events]))
               if wl.backward else 0.0)
    # with flushing, the step is the two calls (the flush between steps is not
    # part of it); without, the wall clock over the K steps
    ms_per_step = fwd_ms + bwd_ms if scrub is not None else elapsed * 1e3 / args.steps
    del dev, x, w, lam, u, y, ws
    if wl.backward:
        del dy, grads
    name = "train" if train else "plain" if layout == gspn.PIXEL else layout
    return {"layout": layout, "name": name, "fwd_ms": fwd_ms, "bwd_ms": bwd_ms, "fwd_median_ms": fwd_med,
            "bwd_median_ms": bwd_med, "ms_per_step": ms_per_step}


def summarize(wl, inputs, args, torch, main, others, scrub) -> dict:
    fwd_ms, bwd_ms, ms_per_step = main["fwd_ms"], main["bwd_ms"], main["ms_per_step"]

    def flush():
        if scrub is not None:
            scrub.sum()

    pixch = wl.pixels_channels
    value = pixch / (ms_per_step * 1e-3) / 1e9
    nbytes = algorithmic_bytes(wl)
    step_gbs = (nbytes["fwd"] + nbytes["bwd"]) / (ms_per_step * 1e-3) / 1e9
    log(f"fwd {fwd_ms:.4f} ms  bwd {bwd_ms:.4f} ms  step {ms_per_step:.4f} ms  "
        f"{value:.2f} Gpix.ch/s  step algorithmic {step_gbs:.0f} GB/s "
        f"({step_gbs / HBM_PEAK_GBS:.1%} of peak)")

    train = main["name"] == "train"
    fwd_name, bwd_name = call_names(args.norm, train, wl.backward)
    if bwd_ms > fwd_ms:
        dom, call, dom_ms, dom_bytes = bwd_name, "bwd", bwd_ms, nbytes["bwd"]
    else:
        dom, call, dom_ms, dom_bytes = fwd_name, "fwd", fwd_ms, nbytes["fwd"]
    achieved = dom_bytes / (dom_ms * 1e-3) / 1e9
    # measured HBM bytes of the same call (FETCH_SIZE + WRITE_SIZE counters, scaled by a
    # plain copy), kept in profiles/ for the current kernel sources only
    from paper_2606_00746_amd import profiling
    tag = ("logits-" if args.norm else "") + ("pair" if train else args.layout)
    traffic = profiling.load_traffic(
        os.path.join(ROOT, "profiles", f"traffic_{wl.name}-{tag}.txt"), call)
    roofline = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS,
                "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                "traffic": traffic,
                "kernel": dom, "avg_ms": round(dom_ms, 5), "algorithmic_bytes": dom_bytes}

    # the achievable-bandwidth ceiling for the same bytes, and how much of the
    # call's time it leaves unexplained
    copy_ms = timed_copy(dom_bytes, 10, flush, torch)
    probe = {"bytes": dom_bytes, "ms": round(copy_ms, 5),
             "gbs": round(dom_bytes / (copy_ms * 1e-3) / 1e9, 1),
             "serialisation_share": round(1.0 - copy_ms / dom_ms, 4)}
    if traffic:
        # the same with the bytes the call actually moves
        probe["serialisation_share_measured_bytes"] = round(
            1.0 - copy_ms * traffic / dom_bytes / dom_ms, 4)

    out = {
        "metric": METRIC,
        "value": round(value, 3),
        "unit": "Gpix·ch/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": wl.name, "B": wl.B, "C": wl.C, "G": wl.G, "H": wl.H, "W": wl.W,
                   "directions": wl.ndirs, "pass": "fwd+bwd" if wl.backward else "fwd",
                   "storage": wl.dtype, "weights": "logits" if args.norm else "normalized",
                   "layout": ("pixel-major [D][B][C][H][W] / [D][B][G][3][H][W]"
                              if args.layout == "pixel" else "blocked line-major"),
                   "calls": " + ".join(c for c in (fwd_name, bwd_name) if c),
                   "parallelism": "single GPU"},
        "fwd_ms": round(fwd_ms, 5),
        "bwd_ms": round(bwd_ms, 5),
        "fwd_median_ms": round(main["fwd_median_ms"], 5),
        "bwd_median_ms": round(main["bwd_median_ms"], 5),
        "cache_flush_mib": args.flush_mib,
        "step_hbm_gbs_algorithmic": round(step_gbs, 1),
        "step_hbm_frac": round(step_gbs / HBM_PEAK_GBS, 4),
        "roofline": roofline,
        "copy_probe": probe,
    }
    for other in others:
        o_ms = other["ms_per_step"]
        out[other["name"]] = {
            "value": round(pixch / (o_ms * 1e-3) / 1e9, 3), "ms_per_step": round(o_ms, 5),
            "fwd_ms": round(other["fwd_ms"], 5), "bwd_ms": round(other["bwd_ms"], 5),
            "step_hbm_frac": round((nbytes["fwd"] + nbytes["bwd"]) / (o_ms * 1e-3) / 1e9
                                   / HBM_PEAK_GBS, 4)}
        log(f"{other['name']}: fwd {other['fwd_ms']:.4f} ms  bwd {other['bwd_ms']:.4f} ms"
            f"  step {o_ms:.4f} ms")
    if not args.no_cpu_baseline:
        # the oracle on every core this process may use, up to the 16 that
        # are one GPU's share of the host (the reported baseline), and on one
        # thread beside it
        nthr = cpu_threads()
        log(f"timing the CPU oracle on {nthr} threads ...")
        out["cpu_baseline"] = cpu_baseline(wl, inputs, args.cpu_seconds, args.norm,
                                           threads=nthr)
        log("timing the CPU oracle on one thread ...")
        out["cpu_baseline_single_thread"] = cpu_baseline(wl, inputs, args.cpu_seconds / 2,
                                                         args.norm)
    return out


def call_names(norm: bool, train: bool, backward: bool):
    """The entry points of the headline step: (forward, backward or None)."""
    if train:
        pair = (("gspn_scan_fwd_norm_train", "gspn_scan_bwd_norm_reserve") if norm else
                ("gspn_scan_fwd_train", "gspn_scan_bwd_reserve"))
    else:
        pair = (("gspn_scan_fwd_norm", "gspn_scan_bwd_norm") if norm else
                ("gspn_scan_fwd", "gspn_scan_bwd"))
    return pair[0], (pair[1] if backward else None)


LATENT_METRIC = ("C-GSPN latent sublayer fwd Gpix·ch/s (input pixel-channels) at 1 MI355X; "
                 "achieved HBM GB/s vs peak")


# Sublayer latency of the paper's A100 measurement at batch 32 (Sec. 6, the
# latency tables over resolutions), by token grid: context, not a target.
PAPER_A100_SUBLAYER_MS = {37: 0.088, 74: 0.18, 111: 0.299, 147: 0.46, 185: 0.646}


def latent_grid(lw: gi.LatentWorkload) -> tuple:
    """The grid of the sublayer's latent tensors: gspn_latent_fwd pads sides
    that are not multiples of 8 up to whole 8-line blocks (above 16 pixels,
    up to 256)."""
    up8 = lambda v: (v + 7) // 8 * 8
    pad = ((lw.H % 8 or lw.W % 8) and max(lw.H, lw.W) > 16 and up8(lw.H) <= 256
           and up8(lw.W) <= 256)
    return (up8(lw.H), up8(lw.W)) if pad else (lw.H, lw.W)


def latent_stage_bytes(lw: gi.LatentWorkload) -> dict:
    """Compulsory HBM bytes of the sublayer's stages (bf16): every input read
    once, every output written once, on the image's own grid (a padded
    latent grid's extra pixels count as overhead, not as work)."""
    HW, D = lw.H * lw.W, lw.ndirs
    x, xc = lw.B * lw.C * HW * 2, lw.B * lw.Cc * HW * 2
    scan = algorithmic_bytes(gi.Workload("latent-scan", lw.B, lw.Cc, lw.Cc, lw.H, lw.W, "bf16",
                                         lw.dirs, False, "sigmoid", 1.0, 0))["fwd"]
    return {"down": x + xc + lw.Cc * lw.C * 2,
            "params": xc + 5 * D * xc + 5 * D * lw.Cc * lw.Cc * 2,
            "scan": scan,
            "up": xc + x + lw.C * lw.Cc * 2}


def latent_cpu_baseline(lw: gi.LatentWorkload, inp: dict, min_seconds: float) -> dict:
    """The fp64 oracle on single images of the workload, until about
    `min_seconds` have passed."""
    import oracle
    done = 0
    t0 = time.perf_counter()
    while time.perf_counter() - t0 < min_seconds and done < 4 * lw.B:
        b = done % lw.B
        oracle.latent_fwd(inp["x"][b:b + 1], inp["p_down"], inp["l_u"], inp["l_lam"],
                          inp["l_w"], inp["p_up"], lw.dirs, storage="bf16")
        done += 1
    dt = time.perf_counter() - t0
    return {"value": round(done * lw.C * lw.H * lw.W / dt / 1e9, 6), "unit": "Gpix·ch/s",
            "cores": 1, "kind": "oracle",
            "sample": f"{done} images of {lw.name} ({lw.B} per step; fp64 with bf16 storage "
                      f"points, numpy matmuls + C scan, single thread, {_cpu_model()}), "
                      f"{dt:.1f} s"}


def run_latent(lw: gi.LatentWorkload, args, torch, gspn) -> dict:
    log(f"latent workload {lw}")
    inp = gi.make_latent_inputs(lw)
    dev = {k: to_device(v, "bf16", torch) for k, v in inp.items()}
    stream = torch.cuda.current_stream()
    scrub = (torch.ones(args.flush_mib * (1 << 20) // 4, dtype=torch.float32, device="cuda")
             if args.flush_mib > 0 else None)
    D, HW = lw.ndirs, lw.H * lw.W
    Hp, Wp = latent_grid(lw)
    kw = dict(dtype=torch.bfloat16, device="cuda")
    y = torch.empty_like(dev["x"])
    xc = torch.empty((lw.B, lw.Cc, lw.H, lw.W), **kw)
    yc = torch.empty_like(xc)
    # the parameter product and the scan on the latent grid, as the sublayer
    # runs them (its padding holds x_c = 0)
    xcp = torch.zeros((lw.B, lw.Cc, Hp, Wp), **kw)
    ycp = torch.empty_like(xcp)
    prm = (torch.empty((D, lw.B, lw.Cc, Hp * Wp), **kw),
           torch.empty((D, lw.B, lw.Cc, Hp * Wp), **kw),
           torch.empty((D, lw.B, lw.Cc, 3, Hp * Wp), **kw))

    def flush():
        if scrub is not None:
            scrub.sum()

    calls = {
        "sublayer": lambda: gspn.latent_fwd(dev["x"], dev["p_down"], dev["l_u"], dev["l_lam"],
                                            dev["l_w"], dev["p_up"], lw.dirs, y=y,
                                            stream=stream),
        "down": lambda: gspn.project(dev["p_down"], dev["x"], y=xc, stream=stream),
        "params": lambda: gspn.latent_params(xcp, dev["l_u"], dev["l_lam"], dev["l_w"], lw.dirs,
                                             out=prm, stream=stream),
        "scan": lambda: gspn.scan_fwd(xcp, prm[2], prm[1], prm[0], lw.dirs, y=ycp,
                                      stream=stream, layout=gspn.BLOCKED),
        "up": lambda: gspn.project(dev["p_up"], yc, y=y, stream=stream),
    }

    def timed(fn, reps):
        ms = []
        for _ in range(reps):
            flush()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            fn()
            e1.record(stream)
            torch.cuda.synchronize()
            ms.append(e0.elapsed_time(e1))
        return float(np.mean(ms))

    for k, fn in calls.items():
        for _ in range(max(1, args.warmup)):
            fn()
        if k == "down":
            xcp[:, :, :lw.H, :lw.W] = xc
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ms_step = timed(calls["sublayer"], args.steps)
    log(f"sublayer {ms_step:.4f} ms over {args.steps} steps ({time.perf_counter() - t0:.1f} s)")
    stage_ms = {k: timed(fn, args.steps) for k, fn in calls.items() if k != "sublayer"}
    nbytes = latent_stage_bytes(lw)
    stages = {k: {"ms": round(v, 5), "algorithmic_bytes": nbytes[k],
                  "hbm_frac": round(nbytes[k] / (v * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)}
              for k, v in stage_ms.items()}
    log("stages: " + ", ".join(f"{k} {v['ms']:.4f} ms ({v['hbm_frac']:.1%})"
                               for k, v in stages.items()))
    dom = max(stage_ms, key=stage_ms.get)
    achieved = nbytes[dom] / (stage_ms[dom] * 1e-3) / 1e9
    total = sum(nbytes.values())
    out = {
        "metric": LATENT_METRIC,
        "value": round(lw.B * lw.C * HW / (ms_step * 1e-3) / 1e9, 3),
        "unit": "Gpix·ch/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": lw.name, "B": lw.B, "C": lw.C, "Cc": lw.Cc, "H": lw.H,
                   "W": lw.W, "latent_grid": [Hp, Wp], "directions": D, "pass": "fwd",
                   "storage": "bf16",
                   "parallelism": "single GPU"},
        "cache_flush_mib": args.flush_mib,
        "step_hbm_gbs_algorithmic": round(total / (ms_step * 1e-3) / 1e9, 1),
        "step_hbm_frac": round(total / (ms_step * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
        "stages": stages,
        "roofline": {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": None,
                     "kernel": dom, "avg_ms": round(stage_ms[dom], 5),
                     "algorithmic_bytes": nbytes[dom]},
    }
    if lw.B == 32 and lw.H == lw.W and lw.H in PAPER_A100_SUBLAYER_MS:
        out["paper_context"] = {"a100_sublayer_ms": PAPER_A100_SUBLAYER_MS[lw.H],
                                "note": "A100, the paper's own sublayer latency at this grid "
                                        "and batch; other hardware, not vs_baseline"}
    if not args.no_cpu_baseline:
        log("timing the CPU oracle ...")
        out["cpu_baseline"] = latent_cpu_baseline(lw, inp, args.cpu_seconds)
    return out


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="3",
                    help="index or name of the workload, or 'all' (one line each)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--layout", default="pixel", choices=("pixel", "blocked"),
                    help="layout of the per-direction tensors of the reported step")
    ap.add_argument("--plain", action="store_true",
                    help="time the plain pair gspn_scan_fwd + gspn_scan_bwd as the headline")
    ap.add_argument("--no-blocked", action="store_true",
                    help="time only the headline pair (no plain or blocked entries beside it)")
    ap.add_argument("--norm", action="store_true",
                    help="weights given as logits: time the _norm training pair (and the "
                         "plain gspn_scan_fwd_norm / gspn_scan_bwd_norm beside it)")
    ap.add_argument("--latent", default=None,
                    help="time the latent sublayer instead: index or name of the latent "
                         "workload, or 'all'")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="approximate CPU time of the oracle baseline")
    ap.add_argument("--flush-mib", type=int, default=1024,
                    help="MiB read before every step, outside the timed events (0: none; "
                         "the step is then timed by the wall clock over all K steps)")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="before the timed region, copy MIB MiB device to device once (a plain "
                         "copy kernel of known traffic, the reference for HBM byte counters)")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the scan needs no communication, and each GPU "
              "of a data-parallel job runs this kernel on its own batch shard. Run with --gpus 1.",
              file=sys.stderr)
        return 2

    import torch
    import paper_2606_00746_amd as gspn

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 1
    gspn.load()

    if args.latent is not None:
        key = args.latent
        lws = (list(gi.LATENT_WORKLOADS) if key == "all"
               else [gi.latent_workload(int(key) if key.isdigit() else key)])
        for lw in lws:
            print(json.dumps(run_latent(lw, args, torch, gspn)), flush=True)
            torch.cuda.empty_cache()
        return 0

    key = args.workload
    if key == "all":
        wls = list(gi.WORKLOADS)
    else:
        wls = [gi.workload(int(key) if key.isdigit() else key)]
    for wl in wls:
        print(json.dumps(run_workload(wl, args, torch, gspn)), flush=True)
        torch.cuda.empty_cache()
    return 0


if __name__ == "__main__":
    sys.exit(main())
