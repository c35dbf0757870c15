#!/usr/bin/env python3
"""Benchmark: multi-level RoIAlign forward + backward on one MI355X.

One step is one pass of the whole hot path over one batch of synthetic input:
  roi_extract_plan   FPN level of every RoI, level/image/cell-bucketed launch order,
                     tile -> RoI lists
  roi_align_fwd      gather-average into [K, C, 7, 7]
  roi_align_bwd      (default, --bwd gather) every 8x8 x 64-channel tile of the fp32
                     gradient pyramid sums its RoIs and is written once, clearing included;
                     (--bwd scatter) roi_extract_zero_grad, then per-RoI fp32 atomics.
The other backward algorithm is timed separately and reported under extra.other_bwd.

Default workload: the FPN box head (batch 2, 800x1344 images, P2-P5 with C=256 fp32,
512 RoIs per image, 7x7, sampling ratio 2, aligned), inputs resident in HBM before
timing starts.  Prints one JSON line.

  python bench.py [--steps K] [--warmup W] [--workload 2] [--layout cl|nchw]
  python bench.py --calibrate-copy      # plain copy kernel for the counter scale
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "RoIAlign fwd+bwd RoIs/sec and achieved HBM GB/s vs peak, FPN Mask R-CNN shapes"
HBM_PEAK_GBS = 8000.0
PROFILE_DIR = os.path.join(ROOT, "profiles")


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", type=int, default=2, choices=[1, 2, 3, 4, 5])
    ap.add_argument("--head", default="box", choices=["box", "mask"])
    ap.add_argument("--feat-dtype", default=None, choices=[None, "f32", "bf16"])
    ap.add_argument("--layout", default="cl", choices=["cl", "nchw"])
    ap.add_argument("--no-plan", action="store_true", help="RoIs in index order (no sort)")
    ap.add_argument("--bwd", default="gather", choices=["gather", "scatter"],
                    help="backward algorithm of the timed step (the other is timed apart)")
    ap.add_argument("--alt-steps", type=int, default=50,
                    help="steps timed with the other backward algorithm (0: skip)")
    ap.add_argument("--cold-reps", type=int, default=10,
                    help="extra steps each preceded by a 1 GiB cache flush (reported apart)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-copy-ceiling", dest="copy_ceiling", action="store_false",
                    help="skip the 1 GiB copy that measures the practical HBM ceiling")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="oracle work timed for the CPU baseline (seconds)")
    ap.add_argument("--calibrate-copy", action="store_true")
    ap.add_argument("--op", default="align",
                    choices=["align", "pool", "heads", "deform", "nms", "select"],
                    help="align: RoIAlign (the benchmark); pool: RoI max pooling on the same "
                         "workload (plan, roi_pool_fwd, roi_pool_bwd with clearing); heads: "
                         "box and mask heads on one pyramid (workload 2: the batch-2 box and "
                         "mask RoIs; workload 5: both heads of the batch-16 step), one fused "
                         "backward, timed against two separate backward calls; deform: "
                         "modulated deformable RoI pooling on the workload (offsets "
                         "N(0, 0.3^2), modulation U(0, 1), gamma 0.1); nms: greedy NMS of "
                         "two images of 4096 scored proposals in one call (IoU 0.7); "
                         "select: per-image proposal selection of a batch of 16 images x "
                         "2000 proposals in one call (greedy NMS at IoU 0.7 keeping up to "
                         "1000 per image; Soft-NMS linear and Gaussian timed beside it)")
    return ap.parse_args()


ALL_SOURCES = ("common.hpp", "internal.hpp", "gather.hpp", "plan.hip", "fwd.hip", "bwd.hip",
               "pool.hip", "deform.hip", "nms.hip", "select.hip", "api.hip")
# the sources a kernel's code comes from (its device code and the shared headers)
KERNEL_SOURCES = {"fwd": ("common.hpp", "internal.hpp", "fwd.hip"),
                  "bwd_gather": ("common.hpp", "internal.hpp", "gather.hpp", "bwd.hip"),
                  "bwd_scatter": ("common.hpp", "internal.hpp", "gather.hpp", "bwd.hip")}


def kernel_source_hash(kernel: str = None) -> str:
    """Hash of the sources of `kernel` (a KERNEL_SOURCES key), or of every source."""
    h = hashlib.sha256()
    for name in KERNEL_SOURCES[kernel] if kernel else ALL_SOURCES:
        with open(os.path.join(ROOT, "paper_1906_07155_amd", "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def stored_traffic(kernel: str, workload: str):  # kernel: fwd | bwd_gather | bwd_scatter
    """Bytes per launch between the L2 and memory (rocprofv3 FETCH_SIZE + WRITE_SIZE,
    scaled by a plain copy) from a committed counter summary, if it was taken on the
    current sources of that kernel (else None)."""
    path = os.path.join(PROFILE_DIR, "traffic_%s_%s.txt" % (kernel, workload))
    if not os.path.exists(path):
        return None
    vals = {}
    with open(path) as f:
        for line in f:
            if ":" in line and not line.startswith("#"):
                k, v = line.split(":", 1)
                vals[k.strip()] = v.strip()
    if vals.get("kernel_source_hash") != kernel_source_hash(kernel):
        return None
    try:
        return float(vals["bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def time_two_passes(step, names, nsteps, stream):
    """Step time and per-call durations over `nsteps` steps of `step(ev)`.

    An event recorded between two kernels on the stream leaves the GPU idle for about
    5 us, so the step time comes from a pass with events only at its two ends, and the
    per-call durations from a second pass of as many steps in which `step` records
    ev[j] before call j and ev[len(names)] after the last.  Returns (ms per step,
    {name: ms per call}, ms per step of the pass with events)."""
    import torch

    def ev():
        return torch.cuda.Event(enable_timing=True)

    torch.cuda.synchronize()
    t0, t1 = ev(), ev()
    t0.record(stream)
    for _ in range(nsteps):
        step(None)
    t1.record(stream)
    torch.cuda.synchronize()
    ms = t0.elapsed_time(t1) / nsteps
    evs = [[ev() for _ in range(len(names) + 1)] for _ in range(nsteps)]
    t0, t1 = ev(), ev()
    t0.record(stream)
    for i in range(nsteps):
        step(evs[i])
    t1.record(stream)
    torch.cuda.synchronize()
    per = {n: float(np.mean([evs[i][j].elapsed_time(evs[i][j + 1]) for i in range(nsteps)]))
           for j, n in enumerate(names)}
    return ms, per, t0.elapsed_time(t1) / nsteps


def calibrate_copy():
    import torch
    n = 256 * 1024 * 1024          # 1 GiB of float32
    src = torch.ones(n, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(5):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes_read": n * 4, "copy_bytes_written": n * 4, "reps": 5}))


def main():
    args = parse()
    if args.gpus != 1:
        print("bench.py: this build runs on one GPU only (the operator shards by image with no "
              "exchange; see the design notes). --gpus %d is not supported." % args.gpus,
              file=sys.stderr)
        sys.exit(2)
    if args.calibrate_copy:
        calibrate_copy()
        return
    if args.op == "pool":
        main_pool(args)
        return
    if args.op == "heads":
        main_heads(args)
        return
    if args.op == "deform":
        main_deform(args)
        return
    if args.op == "nms":
        main_nms(args)
        return
    if args.op == "select":
        main_select(args)
        return

    import torch

    import paper_1906_07155_amd as rex
    from paper_1906_07155_amd import accounting, workloads

    dev = torch.device("cuda:0")
    wl = workloads.config(args.workload, head=args.head, feat_dtype=args.feat_dtype)
    feats_np = wl.features()
    rois_np = wl.rois()
    K = rois_np.shape[0]
    C = wl.channels
    bf16 = wl.feat_dtype == "bf16"

    def to_dev(a, dt, layout):
        if dt == "bf16":
            t = torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(dev).view(torch.bfloat16)
        else:
            t = torch.from_numpy(a).to(dev)
        return t.contiguous(memory_format=torch.channels_last) if layout == "cl" else t

    feats = [to_dev(f, wl.feat_dtype, args.layout) for f in feats_np]
    rois = torch.from_numpy(rois_np).to(dev)
    odt = torch.bfloat16 if wl.out_dtype == "bf16" else torch.float32
    out = torch.empty((K, C) + tuple(wl.out_hw), dtype=odt, device=dev)
    backward = wl.backward
    if backward:
        gout = to_dev(wl.grad(), wl.grad_dtype, "nchw")
        grads = [torch.empty(f.shape, dtype=torch.float32, device=dev) for f in feats]
        if args.layout == "cl":
            grads = [g.contiguous(memory_format=torch.channels_last) for g in grads]
    L = len(feats)
    levels = torch.empty(K, dtype=torch.int32, device=dev)
    ws = torch.empty(rex.workspace_size(feats, wl.scales, K), dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream()
    S, aligned, out_hw = wl.sampling_ratio, wl.aligned, wl.out_hw
    plan_ws = None if args.no_plan else ws

    def names_for(algo):
        if not backward:
            return ["plan", "fwd"]
        return ["plan", "fwd", "bwd"] if algo == "gather" else ["plan", "fwd", "zero", "bwd"]

    def step(algo, ev=None):
        j = 0

        def mark():
            nonlocal j
            if ev is not None:
                ev[j].record(stream)
            j += 1

        mark()
        rex.plan(feats, wl.scales, rois, wl.finest_scale, levels_out=levels, workspace=ws)
        mark()
        rex.roi_align_fwd(feats, wl.scales, rois, levels, out_hw, S, aligned, out=out,
                          workspace=plan_ws)
        mark()
        if backward:
            if algo == "scatter":
                rex.zero_grad(grads, wl.scales)
                mark()
                rex.roi_align_bwd(gout, rois, levels, out_hw, S, aligned, grads, wl.scales,
                                  zero_init=False, workspace=plan_ws, algorithm="scatter")
            else:
                rex.roi_align_bwd(gout, rois, levels, out_hw, S, aligned, grads, wl.scales,
                                  zero_init=True, workspace=ws, algorithm="gather")
            mark()

    def timed(algo, nsteps):
        return time_two_passes(lambda ev: step(algo, ev), names_for(algo), nsteps, stream)

    algo = args.bwd
    names = names_for(algo)
    for _ in range(args.warmup):
        step(algo)
    torch.cuda.synchronize()
    ms_per_step, per_kernel, ms_with_events = timed(algo, args.steps)

    alt = None
    if backward and args.alt_steps > 0:
        other = "scatter" if algo == "gather" else "gather"
        for _ in range(5):
            step(other)
        alt_ms, alt_per, _ = timed(other, args.alt_steps)
        alt = {"bwd": other, "ms_per_step": round(alt_ms, 5),
               "kernel_ms": {n: round(v, 5) for n, v in alt_per.items()}}

    # NCHW levels: the same step with the pyramid converted to channels-last first and
    # the gradients converted back (torch copies), for callers choosing between them
    via_cl = None
    if args.layout == "nchw" and backward:
        cl_feats = [f.contiguous(memory_format=torch.channels_last) for f in feats]
        cl_grads = [torch.empty(f.shape, dtype=torch.float32, device=dev).contiguous(
            memory_format=torch.channels_last) for f in feats]

        def step_cl(ev=None):
            if ev is not None:
                ev[0].record(stream)
            for d, f in zip(cl_feats, feats):
                d.copy_(f)
            if ev is not None:
                ev[1].record(stream)
            rex.plan(cl_feats, wl.scales, rois, wl.finest_scale, levels_out=levels, workspace=ws)
            rex.roi_align_fwd(cl_feats, wl.scales, rois, levels, out_hw, S, aligned, out=out,
                              workspace=ws)
            rex.roi_align_bwd(gout, rois, levels, out_hw, S, aligned, cl_grads, wl.scales,
                              zero_init=True, workspace=ws, algorithm="gather")
            if ev is not None:
                ev[2].record(stream)
            for d, g in zip(grads, cl_grads):
                d.copy_(g)
            if ev is not None:
                ev[3].record(stream)

        for _ in range(3):
            step_cl()
        vms, vper, _ = time_two_passes(step_cl, ["to_channels_last", "plan_fwd_bwd",
                                                 "grads_to_nchw"], max(3, args.steps // 2), stream)
        via_cl = {"ms_per_step": round(vms, 5), "kernel_ms": {n: round(v, 5) for n, v in vper.items()}}
        del cl_feats, cl_grads

    # cold: each step after a 1 GiB write that evicts L2 and the 256 MB MALL
    cold = None
    if args.cold_reps > 0:
        flush = torch.empty(256 * 1024 * 1024, dtype=torch.float32, device=dev)
        nev = len(names) + 1
        cts = {n: [] for n in names}
        csteps = []
        for _ in range(args.cold_reps):
            flush.zero_()
            ev = [torch.cuda.Event(enable_timing=True) for _ in range(nev)]
            step(algo, ev)
            torch.cuda.synchronize()
            for j, n in enumerate(names):
                cts[n].append(ev[j].elapsed_time(ev[j + 1]))
            csteps.append(ev[0].elapsed_time(ev[-1]))
        cold = {"ms_per_step": float(np.median(csteps)),
                "kernel_ms": {n: float(np.median(v)) for n, v in cts.items()}}
        del flush

    # measured ceiling: a plain 1 GiB device-to-device copy (torch's copy kernel)
    copy_gbs = None
    if args.copy_ceiling:
        n = 256 * 1024 * 1024
        src = torch.ones(n, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        c0 = torch.cuda.Event(enable_timing=True)
        c1 = torch.cuda.Event(enable_timing=True)
        c0.record(stream)
        for _ in range(10):
            dst.copy_(src)
        c1.record(stream)
        torch.cuda.synchronize()
        copy_gbs = round(2 * 4 * n * 10 / (c0.elapsed_time(c1) * 1e-3) / 1e9, 1)
        del src, dst

    # algorithmic bytes
    lv_np = levels.cpu().numpy()
    s_feat = 2 if bf16 else 4
    s_out = 2 if wl.out_dtype == "bf16" else 4
    s_gout = 2 if wl.grad_dtype == "bf16" else 4
    by = accounting.count(rois_np, lv_np, wl.level_hw, wl.scales, wl.n_images, C, out_hw, S,
                          aligned, s_feat, s_out, s_gout)
    # bytes each kernel must move: the gather backward reads the upstream gradient once
    # and writes every gradient element once (the clearing is part of it); the scatter
    # backward does one fp32 read-modify-write per distinct (pixel, channel) of each RoI
    gather_bytes = by.out_bytes // s_out * s_gout + by.zero + 24 * K
    alg = {"plan": 24 * K + 4 * K * 3, "fwd": by.e_fwd}
    if backward:
        alg.update({"zero": by.zero, "bwd": gather_bytes if algo == "gather" else by.e_bwd})
    gbs = {n: alg[n] / (per_kernel[n] * 1e-3) / 1e9 for n in names}
    dominant = max(["fwd", "bwd"] if backward else ["fwd"], key=lambda n: per_kernel[n])
    wname = wl.tag + ("_nchw" if args.layout == "nchw" else "")
    kname = {"fwd": "fwd", "bwd": "bwd_" + algo}[dominant]
    traffic = stored_traffic(kname, wname)
    roofline = {"bound": "hbm", "achieved": round(gbs[dominant], 1), "peak": HBM_PEAK_GBS,
                "unit": "GB/s", "frac": round(gbs[dominant] / HBM_PEAK_GBS, 4),
                "traffic": traffic, "kernel": "roi_align_" + kname,
                "bytes_per_launch": alg[dominant],
                "bytes_model": ("bytes the kernel must move: for the gather backward the "
                                "upstream gradient read once and every gradient element "
                                "written once; for the forward E_fwd (each RoI's distinct "
                                "footprint read once per channel plus the output)"),
                "launch_ms": round(per_kernel[dominant], 5)}
    if traffic is not None:
        roofline["traffic_kind"] = ("L2 egress: rocprofv3 FETCH_SIZE + WRITE_SIZE per launch, "
                                    "scaled by a plain copy; hits in the 256 MB MALL are not "
                                    "seen by these counters")
    if dominant == "bwd":
        # the same kernel against the effective-byte model of the workload (E_bwd: the
        # upstream gradient plus one fp32 read-modify-write per distinct (pixel, channel)
        # of every RoI, the traffic of a scatter with atomics).  The gather performs no
        # read-modify-write (it accumulates in registers and writes each element once),
        # so E_bwd is not a bound for it and this fraction can exceed 1.
        roofline["frac_effective"] = round(by.e_bwd / (per_kernel["bwd"] * 1e-3) / 1e9
                                           / HBM_PEAK_GBS, 4)
        roofline["effective_bytes_per_launch"] = by.e_bwd

    step_bytes = sum(alg[n] for n in names)
    extra = {
        "kernel_ms": {n: round(v, 5) for n, v in per_kernel.items()},
        "kernel_GBps_effective": {n: round(v, 1) for n, v in gbs.items()},
        "step_GBps_effective": round(step_bytes / (ms_per_step * 1e-3) / 1e9, 1),
        "ms_per_step_with_kernel_events": round(ms_with_events, 5),
        "copy_GBps_measured": copy_gbs,
        "bytes": {"E_fwd": by.e_fwd, "E_bwd": by.e_bwd, "U_fwd": by.u_fwd, "U_bwd": by.u_bwd,
                  "T_fwd": by.t_fwd, "zero_fill": by.zero,
                  "footprint_px": by.footprint_px, "union_px": by.union_px},
        "fwd_bwd_GBps_effective": (
            round((by.e_fwd + by.e_bwd) / ((per_kernel["fwd"] + per_kernel["bwd"]) * 1e-3) / 1e9,
                  1) if backward else None),
        # the same against the 8 TB/s peak: effective bytes (E_fwd + E_bwd, the backward
        # counted as the read-modify-write of a scatter), the measure the >= 50% target of
        # the box-head workload is stated in; roofline.frac above uses the bytes the
        # gather backward must move instead (upstream gradient read once, pyramid written
        # once), which is stricter
        "fwd_bwd_frac_effective": (
            round((by.e_fwd + by.e_bwd) / ((per_kernel["fwd"] + per_kernel["bwd"]) * 1e-3) / 1e9
                  / HBM_PEAK_GBS, 4) if backward else None),
        "bwd_algorithm": algo if backward else None,
        "other_bwd": alt,
        "cold": cold,
        "layout": args.layout,
        "nchw_via_channels_last": via_cl,
        "plan": not args.no_plan,
        "kernel_source_hash": kernel_source_hash(),
        "kernel_source_hashes": {k: kernel_source_hash(k) for k in KERNEL_SOURCES},
    }

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(wl, feats_np, rois_np, lv_np, args.cpu_seconds)

    # cold step (each step after a 1 GiB write that evicts L2 and the MALL), with the
    # headline measure of the effective-byte model: (E_fwd + E_bwd) over the forward and
    # backward times, the plan included in the forward, zero-fill not counted
    cold_line = None
    if cold is not None:
        ck = cold["kernel_ms"]
        t_fb = ck["plan"] + ck["fwd"] + (ck["bwd"] if backward else 0.0)
        cold_line = {
            "ms_per_step": round(cold["ms_per_step"], 5),
            "value": round(K / (cold["ms_per_step"] * 1e-3), 1), "unit": "RoIs/s",
            "kernel_ms": {n: round(v, 5) for n, v in ck.items()},
            "frac_effective_fwd_bwd": round((by.e_fwd + (by.e_bwd if backward else 0))
                                            / (t_fb * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
            "reps": args.cold_reps}
    warm_fb = per_kernel["plan"] + per_kernel["fwd"] + (per_kernel["bwd"] if backward else 0.0)
    warm_line = {
        "ms_per_step": round(ms_per_step, 5), "value": round(K / (ms_per_step * 1e-3), 1),
        "unit": "RoIs/s",
        "frac_effective_fwd_bwd": round((by.e_fwd + (by.e_bwd if backward else 0))
                                        / (warm_fb * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)}

    result = {
        "metric": METRIC,
        "value": round(K / (ms_per_step * 1e-3), 1),
        "unit": "RoIs/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if bf16 else "f32",
        "data": "synthetic (seeded normal features, log-uniform RoIs; no COCO)",
        "config": {"workload": wl.name, "num_rois": K, "channels": C,
                   "levels": [list(x) for x in wl.level_hw], "out": list(out_hw),
                   "sampling_ratio": S, "aligned": aligned, "layout": args.layout,
                   "backward": backward},
        "roofline": roofline,
        "cpu_baseline": cpu,
        "warm": warm_line,
        "cold": cold_line,
        "extra": extra,
    }
    print(json.dumps(result), flush=True)


def main_pool(args):
    """RoI max pooling on a workload's pyramid and RoIs: one step is roi_extract_plan,
    roi_pool_fwd and roi_pool_bwd (with the plan's tile lists the backward is the tile
    gather, which writes every gradient element once; otherwise clearing and fp32
    atomics)."""
    import torch

    import oracle
    import paper_1906_07155_amd as rex
    from paper_1906_07155_amd import accounting, workloads

    dev = torch.device("cuda:0")
    wl = workloads.config(args.workload, head=args.head, feat_dtype=args.feat_dtype)
    feats_np, rois_np = wl.features(), wl.rois()
    K, C = rois_np.shape[0], wl.channels
    bf16 = wl.feat_dtype == "bf16"

    def to_dev(a, dt):
        if dt == "bf16":
            t = torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(dev).view(torch.bfloat16)
        else:
            t = torch.from_numpy(a).to(dev)
        return t.contiguous(memory_format=torch.channels_last)

    feats = [to_dev(f, wl.feat_dtype) for f in feats_np]
    rois = torch.from_numpy(rois_np).to(dev)
    odt = torch.bfloat16 if wl.out_dtype == "bf16" else torch.float32
    out = torch.empty((K, C) + tuple(wl.out_hw), dtype=odt, device=dev)
    am = torch.empty((K, C) + tuple(wl.out_hw), dtype=torch.int32, device=dev)
    gout = torch.from_numpy(np.ascontiguousarray(wl.grad()).view(
        np.int16 if wl.grad_dtype == "bf16" else np.float32)).to(dev)
    if wl.grad_dtype == "bf16":
        gout = gout.view(torch.bfloat16)
    grads = [torch.empty(f.shape, dtype=torch.float32, device=dev).contiguous(
        memory_format=torch.channels_last) for f in feats]
    levels = torch.empty(K, dtype=torch.int32, device=dev)
    ws = torch.empty(rex.workspace_size(feats, wl.scales, K), dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream()
    names = ["plan", "fwd", "bwd"]

    def step(ev=None):
        if ev is not None:
            ev[0].record(stream)
        rex.plan(feats, wl.scales, rois, wl.finest_scale, levels_out=levels, workspace=ws)
        if ev is not None:
            ev[1].record(stream)
        rex.roi_pool_fwd(feats, wl.scales, rois, levels, wl.out_hw, out=out, argmax=am,
                         workspace=ws)
        if ev is not None:
            ev[2].record(stream)
        rex.roi_pool_bwd(gout, am, rois, levels, grads, wl.scales, zero_init=True, workspace=ws)
        if ev is not None:
            ev[3].record(stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    ms_per_step, per, ms_with_events = time_two_passes(step, names, args.steps, stream)
    lv_np = levels.cpu().numpy()
    by = accounting.count_pool(rois_np, lv_np, wl.level_hw, wl.scales, wl.n_images, C, wl.out_hw,
                               2 if bf16 else 4, 2 if wl.out_dtype == "bf16" else 4,
                               2 if wl.grad_dtype == "bf16" else 4)
    # the library takes the tile gather for 7x7 bins when the plan holds tile lists (it
    # does here); other grids take the clearing and the atomics
    bwd_alg = "gather" if tuple(wl.out_hw) == (7, 7) else "scatter"
    alg = {"plan": 24 * K + 12 * K, "fwd": by.e_fwd,
           "bwd": by.g_bwd if bwd_alg == "gather" else by.e_bwd + by.zero}
    gbs = {n: alg[n] / (per[n] * 1e-3) / 1e9 for n in names}
    dominant = max(["fwd", "bwd"], key=lambda n: per[n])
    roofline = {"bound": "hbm", "achieved": round(gbs[dominant], 1), "peak": HBM_PEAK_GBS,
                "unit": "GB/s", "frac": round(gbs[dominant] / HBM_PEAK_GBS, 4), "traffic": None,
                "kernel": "roi_pool_" + dominant, "bytes_per_launch": alg[dominant],
                "launch_ms": round(per[dominant], 5)}
    cpu = None
    if not args.no_cpu_baseline:
        lib = oracle.load()
        f64 = [(workloads.bf16_bits_to_f32(f) if bf16 else f).astype(np.float64) for f in feats_np]
        g64 = np.random.default_rng(0).standard_normal((K, C) + tuple(wl.out_hw))
        elapsed, passes = 0.0, 0
        while elapsed < args.cpu_seconds:
            c0 = time.perf_counter()
            _, am_ref = oracle.roi_pool_fwd(f64, wl.scales, rois_np, lv_np, *wl.out_hw, lib=lib)
            oracle.roi_pool_bwd(g64, am_ref, [f.shape for f in f64], rois_np, lv_np, lib=lib)
            elapsed += time.perf_counter() - c0
            passes += 1
        cpu = {"value": round(K * passes / elapsed, 1), "unit": "RoIs/s",
               "cores": oracle.num_threads(lib), "kind": "oracle",
               "sample": "all %d RoIs (all %d channels), fwd+bwd, %d passes in %.1f s wall" % (
                   K, C, passes, elapsed)}
    result = {
        "metric": "RoI max pooling fwd+bwd RoIs/sec and achieved HBM GB/s vs peak, FPN shapes",
        "value": round(K / (ms_per_step * 1e-3), 1), "unit": "RoIs/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16" if bf16 else "f32",
        "data": "synthetic (seeded normal features, log-uniform RoIs; no COCO)",
        "config": {"workload": wl.name + ", RoI max pooling", "num_rois": K, "channels": C,
                   "levels": [list(x) for x in wl.level_hw], "out": list(wl.out_hw),
                   "layout": "cl", "backward": True},
        "roofline": roofline, "cpu_baseline": cpu,
        "extra": {"kernel_ms": {n: round(v, 5) for n, v in per.items()},
                  "ms_per_step_with_kernel_events": round(ms_with_events, 5),
                  "kernel_GBps_effective": {n: round(v, 1) for n, v in gbs.items()},
                  "bytes": {"E_fwd": by.e_fwd, "E_bwd": by.e_bwd, "G_bwd": by.g_bwd,
                            "zero_fill": by.zero, "box_px": by.box_px},
                  "bwd_algorithm": bwd_alg,
                  "kernel_source_hash": kernel_source_hash()},
    }
    print(json.dumps(result), flush=True)


def main_heads(args):
    """Box (7x7) and mask (14x14) heads on one pyramid: one step is a plan per head,
    roi_align_fwd_multi (both heads' forwards in one launch) and roi_align_bwd_multi
    (both heads in one pass over the gradient pyramid).  The same step with one
    roi_align_fwd and one roi_align_bwd call per head is timed too."""
    import torch

    import paper_1906_07155_amd as rex
    from paper_1906_07155_amd import accounting, workloads

    if args.workload == 5:
        wb, wm = workloads.config(5, head="box"), workloads.config(5, head="mask")
    elif args.workload == 2:
        wb, wm = workloads.config(2), workloads.config(3)
    else:
        raise SystemExit("--op heads takes workload 2 or 5")
    dev = torch.device("cuda:0")
    bf16 = wb.feat_dtype == "bf16"

    def to_dev(a, dt, cl=True):
        if dt == "bf16":
            t = torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(dev).view(torch.bfloat16)
        else:
            t = torch.from_numpy(np.ascontiguousarray(a)).to(dev)
        return t.contiguous(memory_format=torch.channels_last) if cl else t

    feats_np = wb.features()
    feats = [to_dev(f, wb.feat_dtype) for f in feats_np]
    grads = [torch.empty(f.shape, dtype=torch.float32, device=dev).contiguous(
        memory_format=torch.channels_last) for f in feats]
    odt = torch.bfloat16 if wb.out_dtype == "bf16" else torch.float32
    heads = []
    for w in (wb, wm):
        r_np = w.rois()
        K = r_np.shape[0]
        heads.append({
            "wl": w, "rois_np": r_np, "rois": torch.from_numpy(r_np).to(dev),
            "levels": torch.empty(K, dtype=torch.int32, device=dev),
            "ws": torch.empty(rex.workspace_size(feats, wb.scales, K), dtype=torch.uint8,
                              device=dev),
            "out": torch.empty((K, wb.channels) + tuple(w.out_hw), dtype=odt, device=dev),
            "gout": to_dev(w.grad(), w.grad_dtype, cl=False)})
    stream = torch.cuda.current_stream()

    fwd_heads = [{"rois": h["rois"], "roi_levels": h["levels"], "out_size": h["wl"].out_hw,
                  "sampling_ratio": h["wl"].sampling_ratio, "aligned": h["wl"].aligned,
                  "workspace": h["ws"], "out": h["out"]} for h in heads]

    def step(fused, ev=None):
        if ev is not None:
            ev[0].record(stream)
        for h in heads:
            rex.plan(feats, wb.scales, h["rois"], wb.finest_scale, levels_out=h["levels"],
                     workspace=h["ws"])
        if ev is not None:
            ev[1].record(stream)
        if fused:
            rex.roi_align_fwd_multi(feats, wb.scales, fwd_heads, out_dtype=odt)
        else:
            for h in heads:
                w = h["wl"]
                rex.roi_align_fwd(feats, wb.scales, h["rois"], h["levels"], w.out_hw,
                                  w.sampling_ratio, w.aligned, out=h["out"], workspace=h["ws"])
        if ev is not None:
            ev[2].record(stream)
        if fused:
            rex.roi_align_bwd_multi(
                [{"grad_out": h["gout"], "rois": h["rois"], "roi_levels": h["levels"],
                  "out_size": h["wl"].out_hw, "workspace": h["ws"]} for h in heads],
                grads, wb.scales, zero_init=True)
        else:
            for i, h in enumerate(heads):
                w = h["wl"]
                rex.roi_align_bwd(h["gout"], h["rois"], h["levels"], w.out_hw, w.sampling_ratio,
                                  w.aligned, grads, wb.scales, zero_init=(i == 0),
                                  workspace=h["ws"])
        if ev is not None:
            ev[3].record(stream)

    def timed(fused, n):
        for _ in range(max(1, args.warmup)):
            step(fused)
        ms, per, _ = time_two_passes(lambda ev: step(fused, ev), ["plan", "fwd", "bwd"], n,
                                     stream)
        return ms, per["plan"], per["fwd"], per["bwd"]

    ms, ms_plan, ms_fwd, ms_bwd = timed(True, args.steps)
    alt = timed(False, max(1, args.alt_steps)) if args.alt_steps > 0 else None
    Ktot = sum(h["rois_np"].shape[0] for h in heads)
    s_g = 2 if wb.grad_dtype == "bf16" else 4
    by = accounting.count(heads[0]["rois_np"], heads[0]["levels"].cpu().numpy(),
                          wb.level_hw, wb.scales, wb.n_images, wb.channels, (7, 7), 2, True,
                          2 if bf16 else 4, 2 if wb.out_dtype == "bf16" else 4, s_g)
    # the fused backward must read both upstream gradients and write every gradient once
    gout_bytes = sum(h["gout"].numel() * s_g for h in heads)
    bwd_bytes = gout_bytes + by.zero + 24 * Ktot
    gbs = bwd_bytes / (ms_bwd * 1e-3) / 1e9
    result = {
        "metric": "RoIAlign box+mask heads fwd+bwd RoIs/sec and achieved HBM GB/s vs peak, FPN shapes",
        "value": round(Ktot / (ms * 1e-3), 1), "unit": "RoIs/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms, 5), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16" if bf16 else "f32",
        "data": "synthetic (seeded normal features, log-uniform RoIs; no COCO)",
        "config": {"workload": "%s + %s on one pyramid" % (wb.name, wm.name),
                   "num_rois": [h["rois_np"].shape[0] for h in heads], "channels": wb.channels,
                   "levels": [list(x) for x in wb.level_hw], "out": [[7, 7], [14, 14]],
                   "layout": "cl", "backward": True},
        "roofline": {"bound": "hbm", "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": round(gbs / HBM_PEAK_GBS, 4), "traffic": None,
                     "kernel": "roi_align_bwd_multi", "bytes_per_launch": bwd_bytes,
                     "launch_ms": round(ms_bwd, 5)},
        "cpu_baseline": None,
        "extra": {"ms_plans": round(ms_plan, 5), "ms_fused_fwd": round(ms_fwd, 5),
                  "ms_fused_bwd": round(ms_bwd, 5),
                  "separate_fwd_and_bwd": None if alt is None else {
                      "ms_per_step": round(alt[0], 5), "ms_plans": round(alt[1], 5),
                      "ms_fwd": round(alt[2], 5), "ms_bwd": round(alt[3], 5)},
                  "kernel_source_hash": kernel_source_hash()},
    }
    print(json.dumps(result), flush=True)


def main_deform(args):
    """Modulated deformable RoI pooling: one step is roi_extract_plan,
    deform_roi_pool_fwd and deform_roi_pool_bwd (clearing included)."""
    import torch

    import oracle
    import paper_1906_07155_amd as rex
    from paper_1906_07155_amd import accounting, workloads

    dev = torch.device("cuda:0")
    wl = workloads.config(args.workload, head=args.head, feat_dtype=args.feat_dtype)
    feats_np, rois_np = wl.features(), wl.rois()
    K, C = rois_np.shape[0], wl.channels
    PH, PW = wl.out_hw
    bf16 = wl.feat_dtype == "bf16"
    gamma = 0.1
    rng = np.random.default_rng(workloads.BASE_SEED + 50)
    off_np = (rng.standard_normal((K, 2, PH, PW)) * 0.3).astype(np.float32)
    m_np = rng.uniform(0.0, 1.0, (K, PH, PW)).astype(np.float32)

    def to_dev(a, dt, cl=True):
        if dt == "bf16":
            t = torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(dev).view(torch.bfloat16)
        else:
            t = torch.from_numpy(np.ascontiguousarray(a)).to(dev)
        return t.contiguous(memory_format=torch.channels_last) if cl else t

    feats = [to_dev(f, wl.feat_dtype) for f in feats_np]
    rois = torch.from_numpy(rois_np).to(dev)
    off = torch.from_numpy(off_np).to(dev)
    msk = torch.from_numpy(m_np).to(dev)
    odt = torch.bfloat16 if wl.out_dtype == "bf16" else torch.float32
    out = torch.empty((K, C, PH, PW), dtype=odt, device=dev)
    gout = to_dev(wl.grad() if wl.backward else
                  np.random.default_rng(1).standard_normal((K, C, PH, PW), dtype=np.float32),
                  wl.grad_dtype, cl=False)
    grads = [torch.empty(f.shape, dtype=torch.float32, device=dev).contiguous(
        memory_format=torch.channels_last) for f in feats]
    goff = torch.empty_like(off)
    gmsk = torch.empty_like(msk)
    levels = torch.empty(K, dtype=torch.int32, device=dev)
    ws = torch.empty(rex.workspace_size(feats, wl.scales, K), dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream()
    names = ["plan", "fwd", "bwd"]

    def step(ev=None):
        if ev is not None:
            ev[0].record(stream)
        rex.plan(feats, wl.scales, rois, wl.finest_scale, levels_out=levels, workspace=ws)
        if ev is not None:
            ev[1].record(stream)
        rex.deform_roi_pool_fwd(feats, wl.scales, rois, levels, wl.out_hw, off, msk, gamma,
                                wl.sampling_ratio, wl.aligned, out=out, workspace=ws)
        if ev is not None:
            ev[2].record(stream)
        rex.deform_roi_pool_bwd(gout, feats, rois, levels, off, msk, grads, wl.scales, gamma,
                                wl.sampling_ratio, wl.aligned, zero_init=True, grad_offset=goff,
                                grad_mask=gmsk, workspace=ws)
        if ev is not None:
            ev[3].record(stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    ms_per_step, per, ms_with_events = time_two_passes(step, names, args.steps, stream)
    lv_np = levels.cpu().numpy()
    fp = accounting.deform_footprint(rois_np, lv_np, wl.level_hw, wl.scales, wl.n_images,
                                     wl.out_hw, wl.sampling_ratio, wl.aligned, off_np, gamma)
    s_f, s_o = (2 if bf16 else 4), (2 if wl.out_dtype == "bf16" else 4)
    s_g = 2 if wl.grad_dtype == "bf16" else 4
    elems = K * C * PH * PW
    side = K * PH * PW * 3 * 4                       # offsets and modulation
    zero = sum(wl.n_images * C * H * W * 4 for (H, W) in wl.level_hw)
    # the library takes the tile gather for 7x7 grids with 1-2 samples per axis when the
    # plan holds tile lists (it does here): the upstream gradient read by the gather and
    # by the per-RoI pass, the features read once, every gradient element written once;
    # otherwise one fp32 read-modify-write per footprint pixel and channel plus clearing
    bwd_alg = ("gather" if tuple(wl.out_hw) == (7, 7) and 1 <= wl.sampling_ratio <= 2
               else "atomic")
    alg = {"plan": 36 * K, "fwd": fp * C * s_f + elems * s_o + side + 24 * K,
           "bwd": (2 * elems * s_g + fp * C * s_f + 2 * side + zero + 24 * K
                   if bwd_alg == "gather" else
                   elems * s_g + fp * C * (s_f + 8) + 2 * side + zero + 24 * K)}
    gbs = {n: alg[n] / (per[n] * 1e-3) / 1e9 for n in names}
    dominant = max(["fwd", "bwd"], key=lambda n: per[n])
    cpu = None
    if not args.no_cpu_baseline:
        lib = oracle.load()
        f64 = [(workloads.bf16_bits_to_f32(f) if bf16 else f).astype(np.float64) for f in feats_np]
        g64 = np.random.default_rng(0).standard_normal((K, C, PH, PW))
        n = min(K, 64)
        sub = np.sort(np.random.default_rng(0).choice(K, n, replace=False))
        elapsed, passes = 0.0, 0
        while elapsed < args.cpu_seconds:
            c0 = time.perf_counter()
            oracle.deform_roi_pool_fwd(f64, wl.scales, rois_np[sub], lv_np[sub], PH, PW,
                                       wl.sampling_ratio, wl.aligned, off_np[sub], m_np[sub],
                                       gamma, lib=lib)
            oracle.deform_roi_pool_bwd(g64[sub], f64, wl.scales, rois_np[sub], lv_np[sub], PH, PW,
                                       wl.sampling_ratio, wl.aligned, off_np[sub], m_np[sub],
                                       gamma, lib=lib)
            elapsed += time.perf_counter() - c0
            passes += 1
        cpu = {"value": round(n * passes / elapsed, 1), "unit": "RoIs/s",
               "cores": oracle.num_threads(lib), "kind": "oracle",
               "sample": "%d of %d RoIs (all %d channels), fwd+bwd, %d passes in %.1f s wall" % (
                   n, K, C, passes, elapsed)}
    result = {
        "metric": "modulated deformable RoI pooling fwd+bwd RoIs/sec and achieved HBM GB/s vs "
                  "peak, FPN shapes",
        "value": round(K / (ms_per_step * 1e-3), 1), "unit": "RoIs/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16" if bf16 else "f32",
        "data": "synthetic (seeded normal features, log-uniform RoIs, normal offsets; no COCO)",
        "config": {"workload": wl.name + ", modulated deformable RoI pooling", "num_rois": K,
                   "channels": C, "out": [PH, PW], "gamma": gamma, "layout": "cl",
                   "backward": True},
        "roofline": {"bound": "hbm", "achieved": round(gbs[dominant], 1), "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": round(gbs[dominant] / HBM_PEAK_GBS, 4),
                     "traffic": None, "kernel": "deform_roi_pool_" + dominant,
                     "bytes_per_launch": alg[dominant], "launch_ms": round(per[dominant], 5)},
        "cpu_baseline": cpu,
        "extra": {"kernel_ms": {n: round(v, 5) for n, v in per.items()},
                  "ms_per_step_with_kernel_events": round(ms_with_events, 5),
                  "kernel_GBps_effective": {n: round(v, 1) for n, v in gbs.items()},
                  "footprint_px": fp, "bwd_algorithm": bwd_alg,
                  "kernel_source_hash": kernel_source_hash()},
    }
    print(json.dumps(result), flush=True)


def main_nms(args):
    """Greedy NMS of RPN-like proposals: two images of 4096 scored boxes (centres uniform
    in a 1333 x 800 image, sides log-uniform in [8, 600] px), the image as the category,
    IoU threshold 0.7, every kept box returned.  One step is one box_nms call."""
    import torch

    import oracle
    import paper_1906_07155_amd as rex
    from paper_1906_07155_amd import workloads

    dev = torch.device("cuda:0")
    rng = np.random.default_rng(workloads.BASE_SEED + 60)
    per, n_img = 4096, 2
    boxes = []
    for _ in range(n_img):
        cx, cy = rng.uniform(0, 1333, per), rng.uniform(0, 800, per)
        w = np.exp(rng.uniform(np.log(8), np.log(600), per))
        h = np.exp(rng.uniform(np.log(8), np.log(600), per))
        boxes.append(np.stack([cx - w / 2, cy - h / 2, cx + w / 2, cy + h / 2], 1))
    boxes_np = np.concatenate(boxes).astype(np.float32)
    scores_np = rng.uniform(0, 1, n_img * per).astype(np.float32)
    cats_np = np.repeat(np.arange(n_img, dtype=np.int32), per)
    N = boxes_np.shape[0]
    b = torch.from_numpy(boxes_np).to(dev)
    sc = torch.from_numpy(scores_np).to(dev)
    ct = torch.from_numpy(cats_np).to(dev)
    keep, nk = rex.box_nms(b, sc, 0.7, ct)
    import ctypes
    n = ctypes.c_size_t(0)
    rex.lib().box_nms_workspace_size(N, ctypes.byref(n))
    ws = torch.empty(n.value, dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream()
    for _ in range(args.warmup):
        rex.box_nms(b, sc, 0.7, ct, workspace=ws, keep=keep, num_keep=nk)
    torch.cuda.synchronize()
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    t0.record(stream)
    for _ in range(args.steps):
        rex.box_nms(b, sc, 0.7, ct, workspace=ws, keep=keep, num_keep=nk)
    t1.record(stream)
    torch.cuda.synchronize()
    ms = t0.elapsed_time(t1) / args.steps
    kept = int(nk.item())
    # pairwise overlap tests of the upper triangle (every pair, also across categories),
    # about 16 fp32 operations each: the arithmetic the mask kernel must do
    pairs = N * (N - 1) // 2
    flops = pairs * 16
    achieved = flops / (ms * 1e-3) / 1e12
    cpu = None
    if not args.no_cpu_baseline:
        lib = oracle.load()
        elapsed, passes = 0.0, 0
        while elapsed < args.cpu_seconds:
            c0 = time.perf_counter()
            oracle.nms(boxes_np, scores_np, 0.7, cats_np, lib=lib)
            elapsed += time.perf_counter() - c0
            passes += 1
        cpu = {"value": round(N * passes / elapsed, 1), "unit": "boxes/s", "cores": 1,
               "kind": "oracle", "sample": "all %d boxes, %d passes in %.1f s wall" % (
                   N, passes, elapsed)}
    result = {
        "metric": "greedy NMS boxes/sec (proposal selection before the RoI extraction)",
        "value": round(N / (ms * 1e-3), 1), "unit": "boxes/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms, 5), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "f32",
        "data": "synthetic (uniform centres, log-uniform sizes, uniform scores; no COCO)",
        "config": {"workload": "NMS of 2 x 4096 proposals, IoU 0.7, image as category",
                   "num_boxes": N, "kept": kept},
        "roofline": {"bound": "alu", "achieved": round(achieved, 3), "peak": 157.3,
                     "unit": "TFLOP/s", "frac": round(achieved / 157.3, 5), "traffic": None,
                     "kernel": "box_nms (sort + overlap masks + scan)", "flops_per_launch": flops,
                     "launch_ms": round(ms, 5)},
        "cpu_baseline": cpu,
        "extra": {"kernel_source_hash": kernel_source_hash()},
    }
    print(json.dumps(result), flush=True)


def select_pair_tests(scores, cats, keep, num_keep, n_categories):
    """Box pairs the greedy selection tests: per category, each block of 64 candidates
    (rank order) against the boxes kept before it, plus the pairs inside the block."""
    total = 0
    for c in range(n_categories):
        idx = np.flatnonzero(cats == c)
        u = scores[idx].view(np.uint32).astype(np.uint64)
        asc = np.where(u & 0x80000000, (~u) & 0xFFFFFFFF, u | 0x80000000)
        order = idx[np.lexsort((idx, (~asc) & 0xFFFFFFFF))]
        pos = {int(i): r for r, i in enumerate(order)}
        kept_pos = np.sort([pos[int(i)] for i in keep[c, :num_keep[c]]])
        for b0 in range(0, len(order), 64):
            nb = min(64, len(order) - b0)
            total += nb * int(np.searchsorted(kept_pos, b0)) + nb * (nb - 1) // 2
            if np.searchsorted(kept_pos, b0 + nb) >= len(kept_pos) and \
                    len(kept_pos) == keep.shape[1]:
                break
    return total


def main_select(args):
    """Per-image proposal selection of a training batch: 16 images x 2000 scored
    proposals (synthetic RPN output: uniform centres, log-uniform sides, 30% jittered
    duplicates) in one box_nms_batched call, greedy NMS at IoU 0.7 keeping up to 1000
    per image (the RPN's post-NMS count); Soft-NMS (linear at 0.3, Gaussian sigma 0.5,
    score threshold 0.05, 100 per image) timed beside it.  One step is one call."""
    import torch

    import oracle
    import paper_1906_07155_amd as rex
    from paper_1906_07155_amd import workloads

    dev = torch.device("cuda:0")
    rng = np.random.default_rng(workloads.BASE_SEED + 70)
    n_img, per = 16, 2000
    boxes_np, scores_np, cats_np = workloads.draw_proposals(rng, n_img, per)
    perm = rng.permutation(boxes_np.shape[0])        # images interleaved in the input
    boxes_np, scores_np, cats_np = boxes_np[perm], scores_np[perm], cats_np[perm]
    N = boxes_np.shape[0]
    b = torch.from_numpy(boxes_np).to(dev)
    sc = torch.from_numpy(scores_np).to(dev)
    ct = torch.from_numpy(cats_np).to(dev)
    stream = torch.cuda.current_stream()
    cfgs = {"hard": dict(method="hard", iou_threshold=0.7, max_keep=1000),
            "linear": dict(method="linear", iou_threshold=0.3, score_threshold=0.05,
                           max_keep=100),
            "gaussian": dict(method="gaussian", sigma=0.5, score_threshold=0.05, max_keep=100)}

    def timed(cfg, steps):
        out = rex.box_nms_batched(b, sc, ct, n_img, **cfg)
        for _ in range(args.warmup):
            rex.box_nms_batched(b, sc, ct, n_img, keep=out[0], kept_scores=out[1],
                                num_keep=out[2], **cfg)
        torch.cuda.synchronize()
        t0 = torch.cuda.Event(enable_timing=True)
        t1 = torch.cuda.Event(enable_timing=True)
        t0.record(stream)
        for _ in range(steps):
            rex.box_nms_batched(b, sc, ct, n_img, keep=out[0], kept_scores=out[1],
                                num_keep=out[2], **cfg)
        t1.record(stream)
        torch.cuda.synchronize()
        return t0.elapsed_time(t1) / steps, [o.cpu().numpy() for o in out]

    ms, (keep, ks, nk) = timed(cfgs["hard"], args.steps)
    soft = {}
    for name in ("linear", "gaussian"):
        m, (k2, s2, n2) = timed(cfgs[name], max(1, args.steps // 4))
        soft[name] = {"ms_per_call": round(m, 5), "boxes_per_s": round(N / (m * 1e-3), 1),
                      "kept_per_image": int(n2.mean())}
    pairs = select_pair_tests(scores_np, cats_np, keep, nk, n_img)
    flops = pairs * 16          # about 16 fp32 operations per IoU test
    achieved = flops / (ms * 1e-3) / 1e12
    cpu = None
    if not args.no_cpu_baseline:
        lib = oracle.load()
        elapsed, passes = 0.0, 0
        while elapsed < args.cpu_seconds:
            c0 = time.perf_counter()
            oracle.nms_batched(boxes_np, scores_np, cats_np, n_img, "hard", 0.7, max_keep=1000,
                               lib=lib)
            elapsed += time.perf_counter() - c0
            passes += 1
        cpu = {"value": round(N * passes / elapsed, 1), "unit": "boxes/s", "cores": 1,
               "kind": "oracle", "sample": "all %d boxes (greedy, IoU 0.7), %d passes in %.1f s "
               "wall" % (N, passes, elapsed)}
    result = {
        "metric": "per-image proposal selection boxes/sec (greedy NMS, batch of 16 images)",
        "value": round(N / (ms * 1e-3), 1), "unit": "boxes/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms, 5), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "f32",
        "data": "synthetic (uniform centres, log-uniform sizes, jittered duplicates, uniform "
                "scores; no COCO)",
        "config": {"workload": "16 images x 2000 proposals, greedy NMS IoU 0.7, up to 1000 "
                               "per image", "num_boxes": N, "kept_per_image": int(nk.mean())},
        "roofline": {"bound": "alu", "achieved": round(achieved, 4), "peak": 157.3,
                     "unit": "TFLOP/s", "frac": round(achieved / 157.3, 6), "traffic": None,
                     "kernel": "box_nms_batched (5 launches)", "flops_per_launch": flops,
                     "iou_tests": pairs, "launch_ms": round(ms, 5)},
        "cpu_baseline": cpu,
        "extra": {"soft_nms": soft, "kernel_source_hash": kernel_source_hash()},
    }
    print(json.dumps(result), flush=True)


def cpu_baseline(wl, feats_np, rois_np, lv_np, target_s):
    """The CPU oracle (parity mode, as it stands) on a bounded sample of the same RoIs:
    the sample grows until one pass takes about a second (or covers every RoI), then
    whole passes repeat until `target_s` seconds of oracle work have been timed."""
    import oracle
    from paper_1906_07155_amd import workloads
    lib = oracle.load()
    if wl.feat_dtype == "bf16":
        f64 = [workloads.bf16_bits_to_f32(f).astype(np.float64) for f in feats_np]
    else:
        f64 = [f.astype(np.float64) for f in feats_np]
    shapes = [f.shape for f in f64]
    rng = np.random.default_rng(0)
    K = rois_np.shape[0]

    def one_pass(sub, g):
        t0 = time.perf_counter()
        oracle.roi_align_fwd(f64, wl.scales, rois_np[sub], lv_np[sub], *wl.out_hw,
                             wl.sampling_ratio, wl.aligned, "parity", lib=lib)
        if wl.backward:
            oracle.roi_align_bwd(g, shapes, wl.scales, rois_np[sub], lv_np[sub], *wl.out_hw,
                                 wl.sampling_ratio, wl.aligned, "parity", lib=lib)
        return time.perf_counter() - t0

    n = min(K, 32)
    while True:
        sub = np.sort(rng.choice(K, n, replace=False))
        g = rng.standard_normal((n, wl.channels) + tuple(wl.out_hw)) if wl.backward else None
        el = one_pass(sub, g)
        if el >= 1.0 or n >= K:
            break
        n = min(K, n * 4)
    elapsed, passes = el, 1
    while elapsed < target_s:
        elapsed += one_pass(sub, g)
        passes += 1
    return {"value": round(n * passes / elapsed, 1), "unit": "RoIs/s",
            "cores": oracle.num_threads(lib), "kind": "oracle",
            "sample": "%d of %d RoIs (all %d channels), %s, %d passes in %.1f s wall" % (
                n, K, wl.channels, "fwd+bwd" if wl.backward else "fwd", passes, elapsed)}


if __name__ == "__main__":
    main()
