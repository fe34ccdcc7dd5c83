#!/usr/bin/env python3
"""Benchmark of row-centric CNN training (LR-CNN) on one MI355X.

One step = lrcnn_forward_rows + lrcnn_backward_rows over one batch of the
workload (Algorithm 1's FP and BP over all row bands: forward, band
recompute, input gradients, weight gradients). Inputs are synthetic N(0, 1)
tensors with the paper's shapes (ImageNet is not available), resident in HBM
before timing starts. Prints one JSON line.

Default workload: the largest single-GPU one, ResNet-50 conv trunk,
bfloat16 storage with float32 accumulation, batch 8, 3x2400x3600, 32 row
bands of 75 rows, two-phase sharing. The timed step is captured once in a
HIP graph and replayed (--eager launches every kernel from the host
instead). Also reported: peak activation bytes of the row-centric step
against the layer-wise baseline (same kernels, every feature map kept), the
layer-wise step's speed, the overlapping-recompute mode's speed (halo
overhead), the finer-backward and hybrid-depth variants, a roofline line for
the dominant kernel, the CPU oracle's speed on a bounded sample, and compact
lines (speed, roofline, memory ratio) for the 224x224 workloads.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK = {"f32": ("mfma", 157.3, "TFLOP/s"), "bf16": ("mfma", 2500.0, "TFLOP/s")}
HBM_GBS = 8000.0  # MI355X HBM3E


def kernel_roofline(entry, dts):
    """Roofline of one kernel name from the library's profile aggregate
    (launches, ms, FLOPs, algorithmic bytes, roofline ms). The bound is the
    one that dominates its launches' algorithmic work: matrix-core time
    (FLOPs at the dtype's dense peak) or HBM time (bytes at 8 TB/s);
    `achieved` is FLOP/s or bytes/s against that bound's peak. Also given:
    the matrix-core fraction, and the fraction of the launches' roofline
    time (per launch the larger of the two) that the measured time
    reaches."""
    n, ms, fl, by, rf = entry
    _, pk, unit = PEAK[dts]
    t_mfma = fl / (pk * 1e12)
    t_hbm = by / (HBM_GBS * 1e9)
    tflops = fl / (ms * 1e-3) / 1e12
    if t_hbm > t_mfma:
        achieved, peak, unit, bound = by / (ms * 1e-3) / 1e9, HBM_GBS, "GB/s", "hbm"
    else:
        achieved, peak, bound = tflops, pk, "mfma"
    return {"bound": bound, "achieved": round(achieved, 2), "peak": peak, "unit": unit,
            "frac": round(achieved / peak, 4), "avg_launch_ms": round(ms / n, 4),
            "algorithmic_bytes_per_launch": round(by / n), "flops_per_launch": round(fl / n),
            "tflops": round(tflops, 2), "mfma_frac": round(tflops / pk, 4),
            "roofline_time_frac": round(rf / ms, 4) if ms > 0 else None}


def parse():
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", type=int, default=5, help="workload id 1..5")
    ap.add_argument("--extra-configs", default="2,3",
                    help="comma-separated workload ids measured in compact form after "
                         "the main line (empty: none)")
    ap.add_argument("--mode", default="carry",
                    choices=["carry", "balanced", "paper2ps", "recompute"])
    ap.add_argument("--bands", type=int, default=0, help="override the band count")
    ap.add_argument("--bp-refine", type=int, default=0,
                    help="backward bands per forward band (finer BP partition; 0: the "
                         "workload's step preset)")
    ap.add_argument("--batch", type=int, default=0, help="override the batch")
    ap.add_argument("--hybrid-from", type=int, default=None,
                    help="hybrid depth: first node run layer-wise (-1: the planner's "
                         "smallest-workspace checkpoint; 0: all row-centric; default: the "
                         "workload's step preset)")
    ap.add_argument("--plain", action="store_true",
                    help="ignore the workload's step preset (even bands, no refinement, "
                         "no hybrid depth)")
    ap.add_argument("--no-extras", action="store_true",
                    help="skip the layer-wise / recompute comparison runs")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-images", type=int, default=16)
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--eager", action="store_true",
                    help="launch every kernel from the host in the timed region "
                         "(default: the step is captured once in a HIP graph and replayed)")
    ap.add_argument("--max-batch", action="store_true",
                    help="largest-batch study instead of the throughput line: the "
                         "largest layer-wise and row-centric batches that fit the free "
                         "device memory (planner search), each confirmed by one step")
    ap.add_argument("--sweep-bands", default="",
                    help="band-count study instead of the throughput line: comma-separated "
                         "N values; for each, the CARRY and RECOMPUTE steps' speed, peak "
                         "activation bytes, shared rows and halo rows (use with --batch)")
    ap.add_argument("--train-steps", type=int, default=0,
                    help="full-training study instead of the throughput line: this many "
                         "SGD steps (classifier head, softmax cross-entropy, update) of the "
                         "row-centric and the layer-wise step from the same initial values "
                         "on one synthetic labelled batch; prints both loss curves")
    ap.add_argument("--lr", type=float, default=1e-5)
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="run one plain device copy of this many MiB first (a "
                         "known-size reference for hardware byte counters)")
    return ap.parse_args()


KERNEL_SOURCES = ("kernels.hpp", "kdev.hpp", "kconv.hpp", "kernels.hip", "conv_f32_fwd.hip",
                  "conv_f32_dgrad.hip", "conv_bf16_fwd.hip", "conv_bf16_dgrad.hip",
                  "wgrad.hip")


def kernel_source_hash():
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        with open(os.path.join(ROOT, "paper_2401_11471_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def policy_of(L, mode):
    return {"balanced": L.BALANCED, "paper2ps": L.PAPER_2PS}.get(mode, L.EVEN)


def cpu_baseline(cfg_id, n_img, seconds):
    """Column oracle (float64, numpy/BLAS) FP+BP on a bounded sample of the
    workload, one image at a time, stopping once `seconds` have passed (at
    least one piece); weight gradients are summed. Images of more than 448
    rows are taken in strips of 1/8 of their rows (a strip is an image of
    its own, zero-padded at its edges, and costs 1/8 of an image's work), so
    that the sample stays within the time; images/s counts the rows done."""
    import numpy as np
    import threadpoolctl
    from oracle import column as OC
    from workloads import config_inputs, BF16
    nodes, inp = config_inputs(cfg_id, batch=n_img)
    bf = inp.dtype == BF16
    H = inp.x.shape[1]
    strip = H if H <= 448 else H // 8
    info = threadpoolctl.threadpool_info()
    cores = max([i.get("num_threads", 1) for i in info] or [1])
    t0 = time.perf_counter()
    rows = 0
    pieces = 0
    while rows < n_img * H and (pieces == 0 or time.perf_counter() - t0 < seconds):
        img, r0 = divmod(rows, H)
        x = inp.x[img:img + 1, r0:r0 + strip]
        acts, am = OC.forward(nodes, x, inp.weights, inp.scales, inp.shifts, bf16=bf)
        g = np.zeros(acts[-1].shape) + 1.0
        OC.backward(nodes, acts, am, inp.weights, inp.scales, g, bf16=bf, want_dx=False)
        rows += x.shape[1]
        pieces += 1
    dt = time.perf_counter() - t0
    images = rows / H
    what = (f"{pieces} image(s)" if strip == H else
            f"{pieces} strip(s) of {strip} of the {H} rows ({images:.3f} images)")
    return {"value": round(images / dt, 5), "unit": "images/s", "cores": int(cores),
            "cpu": cpu_model(), "kind": "oracle",
            "sample": f"{what} of the same workload, float64 column FP+BP "
                      f"(numpy/BLAS), {dt:.1f} s"}


def timed_steps(torch, step, steps, warmup, eager, profile=None):
    """ms per step over `steps` steps between two events on the current
    stream. By default the step is captured once in a HIP graph (after a
    warm-up run on a side stream, as capture requires) and replayed, so the
    host's per-launch cost is not in the timed region; the library's
    per-launch events, when `profile` switches them on, are captured into
    the graph and hold the last replay's times. Returns (ms, profiled steps,
    graph)."""
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    # an idle gap before each timed phase, so that a kernel trace of the
    # run can tell the phases apart
    torch.cuda.synchronize()
    time.sleep(0.1)
    if eager:
        for _ in range(warmup):
            step()
        torch.cuda.synchronize()
        if profile:
            profile(True)
        e0.record()
        for _ in range(steps):
            step()
        e1.record()
        torch.cuda.synchronize()
        if profile:
            profile(False)
        return e0.elapsed_time(e1) / steps, steps, None
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        step()
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    if profile:
        profile(True)
    with torch.cuda.graph(graph):
        step()
    if profile:
        profile(False)
    for _ in range(warmup):
        graph.replay()
    torch.cuda.synchronize()
    e0.record()
    for _ in range(steps):
        graph.replay()
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / steps, 1, graph


def compact_workload(args, cid):
    """Compact measurement of another workload: the default row-centric step
    (graph replay; dominant-kernel roofline from an eager pass with the
    library's per-launch events), the layer-wise step, and the variants that
    trade speed for memory (peak-minimising band placement, the hybrid depth
    at the planner's checkpoint, finer backward bands), each with its peak
    activation bytes against the layer-wise step's."""
    import torch
    from paper_2401_11471_amd import lrcnn as L
    from paper_2401_11471_amd.device import DeviceModel
    from workloads import CONFIGS, config_inputs, BF16

    c = dict(CONFIGS[cid])
    nodes, inp = config_inputs(cid)
    B, H, W, Cin = inp.x.shape
    dts = "bf16" if inp.dtype == BF16 else "f32"
    dm = DeviceModel.from_inputs(nodes, inp)
    preset = c.get("step", {})
    base = L.lrcnn_plan(nodes, B, Cin, H, W, inp.dtype, L.CARRY, c["bands"], **preset)
    out_shape = (B,) + base.node_shape(len(nodes) - 1)
    dy = dm.to_device(inp.grad(out_shape))

    def run(plan, layerwise=False, profile=False):
        info = plan.info()
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
        torch.cuda.reset_peak_memory_stats()
        b0 = torch.cuda.memory_allocated()
        ws = dm.workspace(info["layerwise_workspace_bytes" if layerwise else
                               "workspace_bytes"])
        y = dm.empty(out_shape)

        def step():
            if layerwise:
                L.lrcnn_layerwise_reference_gpu(plan, dm.x, dm.w, dm.sc, dm.sf, dy, y, dm.dw,
                                                None, ws)
            else:
                L.lrcnn_forward_rows(plan, dm.x, dm.w, dm.sc, dm.sf, y, ws)
                L.lrcnn_backward_rows(plan, dm.x, dm.w, dm.sc, dm.sf, dy, dm.dw, None, ws)
        step()
        torch.cuda.synchronize()
        peak = torch.cuda.max_memory_allocated() - b0
        ms, _, g = timed_steps(torch, step, args.steps, args.warmup, False)
        del g
        prof = None
        if profile:
            _, ps, _ = timed_steps(torch, step, args.steps, 0, True, L.lrcnn_debug_profile)
            prof = (L.lrcnn_debug_profile_collect(roofline=True), ps)
        del ws, y
        return ms, int(peak), prof

    ms, peak, (kern, ps) = run(base, profile=True)
    dom_name, dom = max(kern.items(), key=lambda kv: kv[1][2])
    roof = kernel_roofline(dom, dts)
    roof.update({"kernel": dom_name, "launches_per_step": dom[0] // ps})
    lw_ms, lw_peak, _ = run(base, layerwise=True)
    res = {"value": round(B * 1000.0 / ms, 3), "unit": "images/s", "ms_per_step": round(ms, 3),
           "dtype": dts,
           "config": {"workload": c["name"], "net": c["net"], "batch": B,
                      "input": [Cin, H, W], "bands": c["bands"], "mode": "carry",
                      "policy": ["even", "balanced"][preset.get("policy", 0)],
                      "bp_bands": base.info()["bp_bands"],
                      "hybrid_from": base.info()["hybrid_from"]},
           "roofline": roof,
           "peak_act_bytes": peak,
           "layerwise": {"images_per_s": round(B * 1000.0 / lw_ms, 3),
                         "ms_per_step": round(lw_ms, 3), "peak_act_bytes": lw_peak},
           "mem_ratio_layerwise_over_rows": round(lw_peak / peak, 3)}
    variants = {}
    for label, kw in (("plain", dict()),
                      ("balanced", dict(policy=L.BALANCED)),
                      ("hybrid", dict(hybrid_from=L.HYBRID_AUTO)),
                      ("balanced_hybrid", dict(policy=L.BALANCED, hybrid_from=L.HYBRID_AUTO)),
                      ("finer_bp", dict(bp_refine=2)),
                      ("finer_bp_hybrid", dict(bp_refine=2, hybrid_from=L.HYBRID_AUTO))):
        plan = L.lrcnn_plan(nodes, B, Cin, H, W, inp.dtype, L.CARRY, c["bands"], **kw)
        info = plan.info()
        v_ms, v_peak, _ = run(plan)
        variants[label] = {"images_per_s": round(B * 1000.0 / v_ms, 3),
                           "ms_per_step": round(v_ms, 3), "peak_act_bytes": v_peak,
                           "mem_ratio_layerwise_over_rows": round(lw_peak / v_peak, 3),
                           "bp_bands": info["bp_bands"], "hybrid_from": info["hybrid_from"],
                           "flops_over_layerwise": round(info["flops_rows"] /
                                                         info["flops_layerwise"], 3)}
        print(f"workload {cid} {label}: {variants[label]['images_per_s']} img/s, ratio "
              f"{variants[label]['mem_ratio_layerwise_over_rows']}", file=sys.stderr,
              flush=True)
    res["variants"] = variants
    ok = {k: v for k, v in variants.items() if v["mem_ratio_layerwise_over_rows"] >= 3.0}
    if res["mem_ratio_layerwise_over_rows"] >= 3.0:
        ok["step"] = {"images_per_s": res["value"]}
    res["fastest_with_3x_memory_cut"] = (max(ok, key=lambda k: ok[k]["images_per_s"])
                                         if ok else None)
    del dm, dy
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return res


def max_batch_study(args):
    """Largest batch of the layer-wise baseline and of the row-centric step
    that fit in the device's free memory: found by the planner's search
    (lrcnn_max_batch over the exact workspace plus every other buffer of the
    step), then confirmed by allocating every buffer and running one step.
    Inputs are N(0, 1) drawn on the device (the confirmation measures
    capacity and time, not values)."""
    import torch
    from paper_2401_11471_amd import lrcnn as L
    from workloads import CONFIGS, config_inputs, BF16

    c = dict(CONFIGS[args.config])
    nb = args.bands or c["bands"]
    mode = L.RECOMPUTE if args.mode == "recompute" else L.CARRY
    policy = policy_of(L, args.mode)
    nodes, inp = config_inputs(args.config, batch=1)
    _, H, W, Cin = inp.x.shape
    tdt = torch.bfloat16 if inp.dtype == BF16 else torch.float32
    free, total = torch.cuda.mem_get_info()
    # the allocator rounds every buffer up to whole 2 MiB blocks: leave a
    # margin for that and for the runtime's own allocations
    budget = free - (2 << 30)
    out = {"metric": "largest training batch that fits one MI355X (FP+BP)",
           "unit": "images", "n_gpus": 1, "config": {"workload": c["name"], "bands": nb,
           "mode": args.mode}, "device_total_bytes": total, "device_free_bytes": free,
           "budget_bytes": budget}
    gen = torch.Generator(device="cuda")
    for label, lw in (("layerwise", True), ("row_centric", False)):
        B = L.lrcnn_max_batch(nodes, Cin, H, W, budget, inp.dtype, mode, nb, policy,
                              bp_refine=args.bp_refine, layerwise=lw)
        plan = L.lrcnn_plan(nodes, B, Cin, H, W, inp.dtype, mode, nb, policy,
                            bp_refine=args.bp_refine)
        info = plan.info()
        print(f"max-batch {label}: B={B}, planned step bytes {plan.step_bytes(lw)}; "
              "allocating and running one step", file=sys.stderr, flush=True)
        torch.cuda.empty_cache()
        torch.cuda.reset_peak_memory_stats()
        base = torch.cuda.memory_allocated()
        gen.manual_seed(args.config)
        x = torch.empty((B, H, W, Cin), device="cuda", dtype=tdt)
        for i in range(B):
            x[i].normal_(generator=gen)
        w = [None] + [None if wv is None else torch.from_numpy(wv).to("cuda", tdt)
                      for wv in inp.weights]
        sc = [None] + [None if v is None else torch.from_numpy(v).cuda() for v in inp.scales]
        sf = [None] + [None if v is None else torch.from_numpy(v).cuda() for v in inp.shifts]
        dw = [None if t is None else torch.empty(t.shape, device="cuda") for t in w]
        oshape = (B,) + plan.node_shape(len(nodes) - 1)
        dy = torch.empty(oshape, device="cuda", dtype=tdt).normal_(generator=gen)
        y = torch.empty(oshape, device="cuda", dtype=tdt)
        ws = torch.empty(info["layerwise_workspace_bytes" if lw else "workspace_bytes"],
                         device="cuda", dtype=torch.uint8)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record()
        if lw:
            L.lrcnn_layerwise_reference_gpu(plan, x, w, sc, sf, dy, y, dw, None, ws)
        else:
            L.lrcnn_forward_rows(plan, x, w, sc, sf, y, ws)
            L.lrcnn_backward_rows(plan, x, w, sc, sf, dy, dw, None, ws)
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1)
        # per image: a float32 copy of the whole output would not fit
        finite = all(bool(torch.isfinite(y[i].float().sum()).item()) for i in range(B)) and \
            all(t is None or bool(torch.isfinite(t.sum()).item()) for t in dw)
        out[label] = {"batch": B, "planned_step_bytes": plan.step_bytes(lw),
                      "peak_allocated_bytes": int(torch.cuda.max_memory_allocated() - base),
                      "step_ms": round(ms, 1), "images_per_s": round(B * 1000.0 / ms, 3),
                      "outputs_finite": finite}
        print(f"max-batch {label}: step {ms:.0f} ms", file=sys.stderr, flush=True)
        del x, w, sc, sf, dw, dy, y, ws, plan
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
    out["batch_ratio_rows_over_layerwise"] = round(
        out["row_centric"]["batch"] / out["layerwise"]["batch"], 3)
    print(json.dumps(out), flush=True)


def band_sweep(args):
    """Row granularity study (the paper's N sweep, Section V): for every band
    count N, the row-centric step in both modes -- images/s, peak activation
    bytes (allocator peak of workspace + y), the rows kept between bands
    (two-phase sharing) and the rows computed twice (overlapping partition)
    -- against the layer-wise step of the same batch."""
    import torch
    from paper_2401_11471_amd import lrcnn as L
    from paper_2401_11471_amd.device import DeviceModel
    from workloads import CONFIGS, config_inputs, BF16

    c = dict(CONFIGS[args.config])
    if args.batch:
        c["batch"] = args.batch
    nodes, inp = config_inputs(args.config, batch=c["batch"])
    B, H, W, Cin = inp.x.shape
    dm = DeviceModel.from_inputs(nodes, inp)
    p1 = L.lrcnn_plan(nodes, B, Cin, H, W, inp.dtype, L.CARRY, 1)
    out_shape = (B,) + p1.node_shape(len(nodes) - 1)
    dy = dm.to_device(inp.grad(out_shape))

    def run(make_step, ws_bytes):
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
        torch.cuda.reset_peak_memory_stats()
        base = torch.cuda.memory_allocated()
        ws = dm.workspace(ws_bytes)
        y = dm.empty(out_shape)
        step = make_step(ws, y)
        step()
        torch.cuda.synchronize()
        peak = torch.cuda.max_memory_allocated() - base
        ms, _, g = timed_steps(torch, step, args.steps, args.warmup, args.eager)
        del g, ws, y
        return ms, int(peak)

    def rc_step(plan):
        return lambda ws, y: (lambda: (
            L.lrcnn_forward_rows(plan, dm.x, dm.w, dm.sc, dm.sf, y, ws),
            L.lrcnn_backward_rows(plan, dm.x, dm.w, dm.sc, dm.sf, dy, dm.dw, None, ws)))

    lw_ms, lw_peak = run(lambda ws, y: (lambda: L.lrcnn_layerwise_reference_gpu(
        p1, dm.x, dm.w, dm.sc, dm.sf, dy, y, dm.dw, None, ws)),
        p1.info()["layerwise_workspace_bytes"])
    res = []
    for nb in [int(v) for v in args.sweep_bands.split(",") if v.strip()]:
        ent = {"n_bands": nb}
        for mode, key in ((L.CARRY, "carry"), (L.RECOMPUTE, "recompute")):
            try:
                plan = L.lrcnn_plan(nodes, B, Cin, H, W, inp.dtype, mode, nb)
            except L.LrcnnError as ex:
                ent[key] = {"error": str(ex)[:120]}
                continue
            info = plan.info()
            ms, peak = run(rc_step(plan), info["workspace_bytes"])
            ent[key] = {"images_per_s": round(B * 1000.0 / ms, 3), "ms_per_step": round(ms, 3),
                        "peak_act_bytes": peak,
                        "mem_ratio_layerwise_over_rows": round(lw_peak / peak, 3),
                        "flops_over_layerwise": round(info["flops_rows"] /
                                                      info["flops_layerwise"], 3),
                        "shared_rows": info["shared_rows"], "halo_rows": info["halo_rows"],
                        "strip_bytes": info["strip_bytes"]}
        print(f"sweep N={nb}: " + ", ".join(
            f"{k} {v.get('images_per_s')} img/s {v.get('peak_act_bytes')} B"
            for k, v in ent.items() if isinstance(v, dict)), file=sys.stderr, flush=True)
        res.append(ent)
    out = {"metric": "row granularity study: training images/s and peak activation bytes vs N",
           "n_gpus": 1, "dtype": "bf16" if inp.dtype == BF16 else "f32",
           "config": {"workload": c["name"], "net": c["net"], "batch": B,
                      "input": [Cin, H, W]},
           "steps": args.steps, "warmup": args.warmup,
           "layerwise": {"images_per_s": round(B * 1000.0 / lw_ms, 3),
                         "ms_per_step": round(lw_ms, 3), "peak_act_bytes": lw_peak},
           "sweep": res}
    print(json.dumps(out), flush=True)


def train_study(args):
    """Loss curves of full training steps (Algorithm 1 with its fully
    connected head, loss and update): row-centric against layer-wise, same
    initial parameters, one synthetic batch with random labels (10 classes);
    also the time of a full row-centric training step."""
    import numpy as np
    import torch
    from paper_2401_11471_amd import lrcnn as L
    from paper_2401_11471_amd.device import DeviceModel
    from paper_2401_11471_amd.train import Trainer
    from workloads import CONFIGS, config_inputs, BF16

    c = dict(CONFIGS[args.config])
    if args.batch:
        c["batch"] = args.batch
    nb = args.bands or c["bands"]
    nodes, inp = config_inputs(args.config, batch=c["batch"])
    B, H, W, Cin = inp.x.shape
    g = np.random.default_rng(args.config)
    labels = g.integers(0, 10, B)
    out = {"metric": "training loss per SGD step (classifier head, softmax cross-entropy)",
           "n_gpus": 1, "dtype": "bf16" if inp.dtype == BF16 else "f32",
           "config": {"workload": c["name"], "net": c["net"], "batch": B, "bands": nb,
                      "classes": 10, "lr": args.lr},
           "data": "synthetic N(0,1) inputs, random labels"}
    for key, lw in (("row_centric", False), ("layerwise", True)):
        plan = L.lrcnn_plan(nodes, B, Cin, H, W, inp.dtype, L.CARRY, nb)
        oh, ow, oc = plan.node_shape(len(nodes) - 1)
        k = oh * ow * oc
        gh = np.random.default_rng(7)
        fw = (gh.standard_normal((10, k)) / np.sqrt(k)).astype(np.float32)
        fb = np.zeros(10, np.float32)
        dm = DeviceModel.from_inputs(nodes, inp)
        tr = Trainer(plan, dm, fw, fb, labels, layerwise=lw)
        losses = []
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(args.train_steps):
            losses.append(tr.step(args.lr).clone())
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / args.train_steps
        out[key] = {"losses": [round(float(v.item()), 6) for v in losses],
                    "ms_per_step": round(ms, 3), "images_per_s": round(B * 1000.0 / ms, 3)}
        print(f"train {key}: loss {losses[0].item():.4f} -> {losses[-1].item():.4f}, "
              f"{ms:.2f} ms/step", file=sys.stderr, flush=True)
        del tr, dm
        torch.cuda.empty_cache()
    a, b = np.array(out["row_centric"]["losses"]), np.array(out["layerwise"]["losses"])
    out["max_rel_loss_difference"] = float(np.max(np.abs(a - b) / np.abs(b)))
    print(json.dumps(out), flush=True)


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py: the library runs on one GPU only; --gpus {args.gpus} "
              f"(WORLD_SIZE={world}) is not supported. Multi-GPU sharding is a "
              "design note, not an implemented path.", file=sys.stderr)
        sys.exit(2)

    if args.max_batch:
        max_batch_study(args)
        return
    if args.sweep_bands:
        band_sweep(args)
        return
    if args.train_steps:
        train_study(args)
        return

    import torch
    from paper_2401_11471_amd import lrcnn as L
    from paper_2401_11471_amd.device import DeviceModel
    from workloads import CONFIGS, config_inputs, BF16

    c = dict(CONFIGS[args.config])
    if args.batch:
        c["batch"] = args.batch
    nb = args.bands or c["bands"]
    mode = L.RECOMPUTE if args.mode == "recompute" else L.CARRY
    preset = {} if args.plain or mode == L.RECOMPUTE else c.get("step", {})
    policy = policy_of(L, args.mode) if args.mode != "carry" else preset.get("policy", L.EVEN)
    args.bp_refine = args.bp_refine or preset.get("bp_refine", 1)
    if args.hybrid_from is None:
        args.hybrid_from = preset.get("hybrid_from", 0)
    nodes, inp = config_inputs(args.config, batch=c["batch"])
    B, H, W, Cin = inp.x.shape
    dts = "bf16" if inp.dtype == BF16 else "f32"

    plan = L.lrcnn_plan(nodes, B, Cin, H, W, inp.dtype, mode, nb, policy,
                        bp_refine=args.bp_refine, hybrid_from=args.hybrid_from)
    info = plan.info()
    dm = DeviceModel.from_inputs(nodes, inp)
    out_shape = (B,) + plan.node_shape(len(nodes) - 1)
    dy = dm.to_device(inp.grad(out_shape))
    torch.cuda.synchronize()

    # --- peak activation bytes: everything the step allocates beyond the
    # parameters, their gradients, the input and dL/dy
    def measure(fn_alloc, fn_step):
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
        torch.cuda.reset_peak_memory_stats()
        base = torch.cuda.memory_allocated()
        bufs = fn_alloc()
        fn_step(bufs)
        torch.cuda.synchronize()
        return torch.cuda.max_memory_allocated() - base, bufs

    def rc_alloc():
        return dict(ws=dm.workspace(info["workspace_bytes"]), y=dm.empty(out_shape))

    def rc_step(b):
        L.lrcnn_forward_rows(plan, dm.x, dm.w, dm.sc, dm.sf, b["y"], b["ws"])
        L.lrcnn_backward_rows(plan, dm.x, dm.w, dm.sc, dm.sf, dy, dm.dw, None, b["ws"])

    peak_rc, bufs = measure(rc_alloc, rc_step)
    if args.copy_calibration_mib:
        n = args.copy_calibration_mib << 18  # float32 elements
        csrc = torch.ones(n, device="cuda")
        cdst = torch.empty_like(csrc)
        torch.cuda.synchronize()
        cdst.copy_(csrc)
        torch.cuda.synchronize()
        del csrc, cdst

    # --- timed region
    ms, psteps, graph = timed_steps(torch, lambda: rc_step(bufs), args.steps, args.warmup,
                                    args.eager, L.lrcnn_debug_profile if args.eager else None)
    del graph
    value = B * 1000.0 / ms
    # the comparison runs of a long step time fewer steps (a few seconds each)
    xsteps = max(3, min(args.steps, int(4000.0 / max(ms, 1e-3))))
    xwarm = min(args.warmup, 2)
    if not args.eager:
        # HIP cannot time events recorded inside a graph, so the per-kernel
        # durations come from an eager pass of the same steps with the
        # library's events attached to every matrix-core dispatch
        _, psteps, _ = timed_steps(torch, lambda: rc_step(bufs), args.steps, 0, True,
                                   L.lrcnn_debug_profile)
    kern = L.lrcnn_debug_profile_collect(roofline=True)
    # the same eager steps with the weight gradients on the caller's stream:
    # every kernel then has the GPU to itself (the default schedule overlaps
    # each weight gradient with an input gradient, and their event times
    # include that sharing)
    L.lrcnn_debug_serial_wgrad(True)
    try:
        ms_serial, psteps_s, _ = timed_steps(torch, lambda: rc_step(bufs), args.steps, 1, True,
                                             L.lrcnn_debug_profile)
    finally:
        L.lrcnn_debug_serial_wgrad(False)
    kern_serial = L.lrcnn_debug_profile_collect(roofline=True)

    # dominant kernel: the largest share of the algorithmic FLOPs (the
    # weight gradient at the ResNet-50 workloads, whose event times in the
    # default schedule include sharing the GPU with an input gradient; the
    # serial pass above times it alone)
    dom_name, dom = max(kern.items(), key=lambda kv: kv[1][2])
    dom_n = dom[0]
    peak = PEAK[dts][1]
    traffic = None
    tpath = os.path.join(ROOT, "profiles", "traffic.json")
    if os.path.exists(tpath):
        try:
            t = json.load(open(tpath))
            ent = t.get(f"cfg{args.config}:{args.mode}:{nb}:{dom_name}")
            if ent and ent.get("source_hash") == kernel_source_hash():
                traffic = ent["bytes_per_launch"]
        except (ValueError, KeyError):
            traffic = None
    roofline = kernel_roofline(dom, dts)
    roofline.update({
        "traffic": traffic, "kernel": dom_name, "launches_per_step": dom_n // psteps,
        "timing": ("HIP events attached to every matrix-core dispatch "
                   "(hipExtLaunchKernelGGL) " +
                   ("in the timed region" if args.eager else
                    "in an eager pass of the same steps after the timed graph replays"))})
    if dom_name in kern_serial:
        alone = kernel_roofline(kern_serial[dom_name], dts)
        alone.update({"step_ms": round(ms_serial, 3),
                      "timing": "eager steps with the weight gradients on the caller's "
                                "stream (no kernel overlaps another)"})
        roofline["alone"] = alone
    all_mfma_ms = sum(v[1] for k, v in kern.items() if "reduce" not in k) / psteps
    all_mfma_fl = sum(v[2] for v in kern.values()) / psteps

    out = {
        "metric": "training images/sec (FP+BP) + peak activation bytes vs layer-wise, 1 MI355X",
        "value": round(value, 3), "unit": "images/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 3),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": dts, "data": "synthetic N(0,1), paper's shapes (ImageNet not available)",
        "config": {"workload": c["name"], "net": c["net"], "batch": B,
                   "input": [Cin, H, W], "bands": nb, "bp_bands": info["bp_bands"],
                   "mode": args.mode, "policy": ["even", "balanced", "explicit",
                                                 "paper2ps"][policy],
                   "dx": False, "hybrid_from": info["hybrid_from"],
                   "launch": "host" if args.eager else "hip-graph"},
        "roofline": roofline,
        "tflops_algorithmic": round(info["flops_rows"] / (ms * 1e-3) / 1e12, 2),
        # the whole step against the matrix-core peak: all of the method's
        # FLOPs (FP, recompute, both gradients), and the useful work of the
        # layer-wise step, 3 tau (the recompute's share made visible)
        "step_roofline": {
            "frac_algorithmic": round(info["flops_rows"] / (ms * 1e-3) / 1e12 / peak, 4),
            "tflops_useful_3tau": round(3 * info["flops_tau"] / (ms * 1e-3) / 1e12, 2),
            "frac_useful_3tau": round(3 * info["flops_tau"] / (ms * 1e-3) / 1e12 / peak, 4)},
        "mfma_kernels": {"ms_per_step": round(all_mfma_ms, 3),
                         "tflops": round(all_mfma_fl / (all_mfma_ms * 1e-3) / 1e12, 2),
                         "per_kernel": {k: {"launches": v[0] // psteps,
                                            "ms": round(v[1] / psteps, 3),
                                            "tflops": round(v[2] / max(v[1], 1e-9) / 1e9, 2)}
                                        for k, v in sorted(kern.items())},
                         "alone_ms_per_step": {k: round(v[1] / psteps_s, 3)
                                               for k, v in sorted(kern_serial.items())}},
        "peak_act_bytes": int(peak_rc),
        "analytic": {k: info[k] for k in ("workspace_bytes", "layerwise_workspace_bytes",
                                          "strip_bytes", "band_cache_bytes",
                                          "fp_window_bytes", "delta_bytes",
                                          "partial_bytes", "omega_bytes", "flops_tau",
                                          "flops_rows", "shared_rows", "halo_rows")},
    }
    # largest batch the planner fits in the whole device memory (host-side
    # search; `--max-batch` confirms it by running)
    total = torch.cuda.mem_get_info()[1]
    out["planned_max_batch"] = {
        "budget_bytes": int(total),
        "layerwise": L.lrcnn_max_batch(nodes, Cin, H, W, total, inp.dtype, mode, nb, policy,
                                       bp_refine=args.bp_refine, layerwise=True),
        "row_centric": L.lrcnn_max_batch(nodes, Cin, H, W, total, inp.dtype, mode, nb,
                                         policy, bp_refine=args.bp_refine,
                                         hybrid_from=args.hybrid_from)}
    del bufs
    torch.cuda.synchronize()
    torch.cuda.empty_cache()

    if not args.no_extras:
        # layer-wise baseline: same kernels, every feature map kept, no recompute
        def lw_alloc():
            return dict(ws=dm.workspace(info["layerwise_workspace_bytes"]),
                        y=dm.empty(out_shape))

        def lw_step(b):
            L.lrcnn_layerwise_reference_gpu(plan, dm.x, dm.w, dm.sc, dm.sf, dy, b["y"],
                                            dm.dw, None, b["ws"])
        try:
            peak_lw, lb = measure(lw_alloc, lw_step)
            lw_ms, _, g_ = timed_steps(torch, lambda: lw_step(lb), xsteps, xwarm,
                                       args.eager)
            del g_
            out["layerwise"] = {"images_per_s": round(B * 1000.0 / lw_ms, 3),
                                "ms_per_step": round(lw_ms, 3),
                                "peak_act_bytes": int(peak_lw)}
            out["mem_ratio_layerwise_over_rows"] = round(peak_lw / peak_rc, 3)
            del lb
        except (RuntimeError, L.LrcnnError) as ex:
            out["layerwise"] = {"error": str(ex)[:200]}
        torch.cuda.empty_cache()
        if mode == L.CARRY and args.bp_refine == 1:
            # the same forward bands with each backward band split in two
            # (Section III-C): smaller backward windows, more launches
            fplan = L.lrcnn_plan(nodes, B, Cin, H, W, inp.dtype, mode, nb, policy, bp_refine=2)
            finfo = fplan.info()

            def f_alloc():
                return dict(ws=dm.workspace(finfo["workspace_bytes"]), y=dm.empty(out_shape))

            def f_step(b):
                L.lrcnn_forward_rows(fplan, dm.x, dm.w, dm.sc, dm.sf, b["y"], b["ws"])
                L.lrcnn_backward_rows(fplan, dm.x, dm.w, dm.sc, dm.sf, dy, dm.dw, None, b["ws"])
            peak_f, fb = measure(f_alloc, f_step)
            f_ms, _, g_ = timed_steps(torch, lambda: f_step(fb), xsteps, xwarm,
                                      args.eager)
            del g_
            ent = {"bp_bands": finfo["bp_bands"], "images_per_s": round(B * 1000.0 / f_ms, 3),
                   "ms_per_step": round(f_ms, 3), "peak_act_bytes": int(peak_f)}
            if "peak_act_bytes" in out.get("layerwise", {}):
                ent["mem_ratio_layerwise_over_rows"] = round(
                    out["layerwise"]["peak_act_bytes"] / peak_f, 3)
            out["finer_backward_bands"] = ent
            del fb
            torch.cuda.empty_cache()
        if args.hybrid_from == 0:
            # hybrid depth (2PS-H / OverL-H) at the planner's checkpoint
            hplan = L.lrcnn_plan(nodes, B, Cin, H, W, inp.dtype, mode, nb, policy,
                                 bp_refine=args.bp_refine, hybrid_from=L.HYBRID_AUTO)
            hinfo = hplan.info()
            if hinfo["hybrid_from"]:
                def h_alloc():
                    return dict(ws=dm.workspace(hinfo["workspace_bytes"]), y=dm.empty(out_shape))

                def h_step(b):
                    L.lrcnn_forward_rows(hplan, dm.x, dm.w, dm.sc, dm.sf, b["y"], b["ws"])
                    L.lrcnn_backward_rows(hplan, dm.x, dm.w, dm.sc, dm.sf, dy, dm.dw, None,
                                          b["ws"])
                peak_h, hb = measure(h_alloc, h_step)
                h_ms, _, g_ = timed_steps(torch, lambda: h_step(hb), xsteps, xwarm,
                                          args.eager)
                del g_
                ent = {"hybrid_from": hinfo["hybrid_from"],
                       "images_per_s": round(B * 1000.0 / h_ms, 3),
                       "ms_per_step": round(h_ms, 3), "peak_act_bytes": int(peak_h),
                       "flops_over_layerwise": round(hinfo["flops_rows"] /
                                                     hinfo["flops_layerwise"], 3)}
                if "peak_act_bytes" in out.get("layerwise", {}):
                    ent["mem_ratio_layerwise_over_rows"] = round(
                        out["layerwise"]["peak_act_bytes"] / peak_h, 3)
                out["hybrid_depth"] = ent
                del hb
                torch.cuda.empty_cache()
            # the earliest checkpoint whose workspace stays 3.5x below the
            # layer-wise step's: the speed the paper's >= 3x memory target
            # leaves room for (deep layers run on whole maps)
            lw_ws = info["layerwise_workspace_bytes"]
            cut, cplan = 0, None
            for k in range(2, len(nodes)):
                try:
                    q = L.lrcnn_plan(nodes, B, Cin, H, W, inp.dtype, mode, nb, policy,
                                     bp_refine=args.bp_refine, hybrid_from=k)
                except L.LrcnnError:
                    continue
                if q.info()["workspace_bytes"] * 3.5 <= lw_ws:
                    cut, cplan = k, q
                    break
            if cut and cut != hinfo["hybrid_from"]:
                cinfo = cplan.info()

                def c_alloc():
                    return dict(ws=dm.workspace(cinfo["workspace_bytes"]), y=dm.empty(out_shape))

                def c_step(b):
                    L.lrcnn_forward_rows(cplan, dm.x, dm.w, dm.sc, dm.sf, b["y"], b["ws"])
                    L.lrcnn_backward_rows(cplan, dm.x, dm.w, dm.sc, dm.sf, dy, dm.dw, None,
                                          b["ws"])
                peak_c, cb = measure(c_alloc, c_step)
                c_ms, _, g_ = timed_steps(torch, lambda: c_step(cb), xsteps, xwarm,
                                          args.eager)
                del g_
                ent = {"hybrid_from": cut, "images_per_s": round(B * 1000.0 / c_ms, 3),
                       "ms_per_step": round(c_ms, 3), "peak_act_bytes": int(peak_c),
                       "flops_over_layerwise": round(cinfo["flops_rows"] /
                                                     cinfo["flops_layerwise"], 3)}
                if "peak_act_bytes" in out.get("layerwise", {}):
                    ent["mem_ratio_layerwise_over_rows"] = round(
                        out["layerwise"]["peak_act_bytes"] / peak_c, 3)
                out["hybrid_within_3x"] = ent
                del cb
                torch.cuda.empty_cache()
        if mode == L.CARRY:
            rplan = L.lrcnn_plan(nodes, B, Cin, H, W, inp.dtype, L.RECOMPUTE, nb,
                                 bp_refine=args.bp_refine)
            rinfo = rplan.info()
            rws = dm.workspace(rinfo["workspace_bytes"])
            ry = dm.empty(out_shape)

            def rstep():
                L.lrcnn_forward_rows(rplan, dm.x, dm.w, dm.sc, dm.sf, ry, rws)
                L.lrcnn_backward_rows(rplan, dm.x, dm.w, dm.sc, dm.sf, dy, dm.dw, None, rws)
            r_ms, _, g_ = timed_steps(torch, rstep, xsteps, xwarm, args.eager)
            del g_
            out["recompute"] = {"images_per_s": round(B * 1000.0 / r_ms, 3),
                                "ms_per_step": round(r_ms, 3),
                                "time_over_carry": round(r_ms / ms, 3),
                                "flops_over_4tau": round(rinfo["flops_rows"] /
                                                         (4 * rinfo["flops_tau"]), 3),
                                "workspace_bytes": rinfo["workspace_bytes"]}
            del rws, ry

    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(args.config, min(args.cpu_images, B),
                                           args.cpu_seconds)
    extra = [int(v) for v in args.extra_configs.split(",") if v.strip()]
    if extra and not args.no_extras:
        del dm, dy
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
        out["other_workloads"] = {}
        for cid in extra:
            if cid == args.config:
                continue
            r = compact_workload(args, cid)
            out["other_workloads"][r["config"]["workload"]] = r
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
