#!/usr/bin/env python3
"""The paper's scene experiments, measured on one MI355X.

    python experiments.py adaptability [--workloads W,...] [--reps R] [--out FILE]
    python experiments.py ablation [--fixed PLAN;PLAN...] [--reps R] [--out FILE]
    python experiments.py acc64 [--workloads W,...] [--fixed PLAN;PLAN...] [--reps R] [--out FILE]
    python experiments.py net [--nets vgg16,alexnet,resnet50] [--batch B] [--layout L] [--reps R] [--out FILE]
    python experiments.py datavalues [--workloads W] [--layers L,...] [--reps R] [--rounds N] [--out FILE]

adaptability -- Sec. 5.1: the channel-scale scenes (5.1.1), the batch sweep
    (5.1.2), the filter-size sweep (5.1.3) and the padding/stride sweep
    (5.1.4).  Per scene: fp32 TFLOPS of the C-ABI call with the selector's
    plan, and the hardware efficiency the paper uses (runtime performance /
    theoretical peak; here the 157.3 TFLOPS fp32 MFMA peak).  Group averages
    follow the paper's groupings.
ablation -- Sec. 5.3, Table 2: one fixed work-group mapping for every scene
    (by default the 128x128 tile, a 2-D wave grid sharing both operands like
    TB(8,8), and the one-wave 32x64 tile, like TB(1,1)), against the per-shape
    selector, on the batch-sweep scenes (B in {64, 128, 256}, IC = OC from 16 to
    1024); average efficiency per B, and the tile the selector picked per scene
    (the analogue of Fig. 14's best-grained map).
acc64 -- the fp64-accumulating entry point (the paper's own numerics: fp32
    data, fp64 arithmetic, Sec. 4.1.1 / Alg. 2) against the fp32 one, per
    layer: TFLOPS and % of each path's MFMA peak (fp64 78.6, fp32 157.3),
    with the selector's plan and any fixed acc64 tile plans given.
net -- whole convolution stacks of the real networks (Sec. 5.2) through the
    native executor: VGG-16 and AlexNet feature extractors and the ResNet-50
    trunk, with ReLU and residual additions fused into the convolutions and
    max pooling between blocks.  Per network: forward time run eagerly and
    replayed from a HIP graph, convolution TFLOPS over the whole forward, and
    the activation arena against keeping every activation.
datavalues -- the same layers, plans and instruction streams on different
    data values: the benchmark's (uniform x, He-normal w), small integers in
    {-2..2} and zeros, timed in interleaved rounds (3 warm-up calls and R
    timed calls per data set and round, in that order).  The MFMA work and the
    cycles it takes do not depend on the values; the power it draws does, and
    with it the clock the chip holds under load.
Inputs are the seeded synthetic tensors of ``workloads`` (HWCN, resident on
the GPU before timing).  Each scene is warmed up for ~100 ms, then timed over
R calls with HIP events on the calling stream.  One JSON line per scene and
one summary line are printed (and written to --out).  Correctness of every
scene at full size is checked by tests/test_parity_layers_gpu.py.
"""
from __future__ import annotations

import argparse
import collections
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_TFLOPS = 157.3
PEAK64_TFLOPS = 78.6


def _time_plan(mg3m, torch, L, xd, wd, yd, plan, reps, ws_cache, acc64=False):
    """Mean microseconds per call of one plan (None = the selector)."""
    args = (L.N, L.C, L.H, L.W, L.K, L.R, L.S, L.stride, L.pad, "HWCN")
    need = 0 if acc64 else mg3m.conv2d_fwd_f32_workspace_bytes(*args, plan)
    if need > ws_cache["bytes"]:
        ws_cache["t"] = None
        torch.cuda.empty_cache()
        ws_cache["t"] = torch.empty((need + 3) // 4, dtype=torch.float32, device="cuda")
        ws_cache["bytes"] = need

    def call():
        if acc64:
            mg3m.conv2d_fwd_f32_acc64(xd, wd, yd, L.N, L.C, L.H, L.W, L.K, L.R, L.S, L.stride,
                                      L.stride, L.pad, L.pad, "HWCN", plan)
        elif plan is None:
            mg3m.conv2d_fwd_f32(xd, wd, yd, *args)
        else:
            ws = ws_cache["t"] if need else None
            mg3m.conv2d_fwd_f32_ex(xd, wd, yd, *args, ws, need, plan)

    call()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        call()
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) * 1e3 / reps


def run_scenes(workload_names, plans, reps, emit, acc64_plans=None):
    """Time every scene of the workloads with the selector and the given
    fixed plans; emit one record per scene.  acc64_plans: also time the
    fp64-accumulating entry point with its selector (None in the list) and
    these fixed plans, keyed "acc64:<plan>"."""
    import torch

    import workloads
    from paper_2307_04941_amd import mg3m

    mg3m.load_library()
    torch.cuda.set_device(0)
    records = []
    ws_cache = {"t": None, "bytes": 0}
    for wl in workload_names:
        for i, L in enumerate(workloads.workload(wl)):
            _, x, w = workloads.layer_tensors(wl, i, "HWCN")
            xd, wd = torch.from_numpy(x).cuda(), torch.from_numpy(w).cuda()
            Ho, Wo = mg3m.conv2d_out_dims(L.H, L.W, L.R, L.S, L.stride, L.pad)
            yd = torch.empty((Ho, Wo, L.K, L.N), dtype=torch.float32, device="cuda")
            flops = 2.0 * L.N * L.K * L.C * L.R * L.S * Ho * Wo
            t_end = time.perf_counter() + 0.1          # clocks up before timing
            while time.perf_counter() < t_end:
                mg3m.conv2d_fwd_f32(xd, wd, yd, L.N, L.C, L.H, L.W, L.K, L.R, L.S,
                                    L.stride, L.pad, "HWCN")
                torch.cuda.synchronize()
            info = mg3m.conv2d_fwd_f32_plan_info(L.N, L.C, L.H, L.W, L.K, L.R, L.S,
                                                 L.stride, L.pad, "HWCN")
            rec = {"workload": wl, "scene": L.name, "N": L.N, "C": L.C, "K": L.K, "H": L.H,
                   "R": L.R, "stride": L.stride, "pad": L.pad, "gflop": flops / 1e9,
                   "selector_plan": f"tile={info['mt']}x{info['nt']}x{info['kt']},"
                                    f"dp={info['dp_tiles']},tail={info['tail_tiles']}x{info['split']}"}
            for plan in [None] + list(plans):
                us = _time_plan(mg3m, torch, L, xd, wd, yd, plan, reps, ws_cache)
                key = plan or "selector"
                rec[key] = {"us": round(us, 2), "tflops": round(flops / us / 1e6, 2),
                            "pct_peak": round(100 * flops / us / 1e6 / PEAK_TFLOPS, 2)}
            if acc64_plans is not None:
                info = mg3m.conv2d_fwd_f32_acc64_plan_string(L.N, L.C, L.H, L.W, L.K, L.R, L.S,
                                                             L.stride, L.stride, L.pad, L.pad, "HWCN")
                rec["acc64_selector_plan"] = info.split(",")[1]
                for plan in acc64_plans:
                    us = _time_plan(mg3m, torch, L, xd, wd, yd, plan, reps, ws_cache, acc64=True)
                    rec["acc64:" + (plan or "selector")] = {
                        "us": round(us, 2), "tflops": round(flops / us / 1e6, 2),
                        "pct_peak64": round(100 * flops / us / 1e6 / PEAK64_TFLOPS, 2)}
            records.append(rec)
            emit(rec)
            del xd, wd, yd
            torch.cuda.empty_cache()
    return records


def run_nets(names, batch, layout, reps, emit):
    import torch

    import workloads
    import workloads.nets as nets
    from paper_2307_04941_amd import mg3m

    mg3m.load_library()
    torch.cuda.set_device(0)
    recs = []
    for name in names:
        N = batch.get(name, 64)
        layers = nets.filters(nets.NETS[name](), layout, seed=1)
        shape = (N, 3, 224, 224)
        flops, shapes = nets.conv_flops(layers, shape)
        net = mg3m.Net(layers, shape, layout)
        kept = sum(4 * n * c * h * w for n, c, h, w in shapes[1:-1])
        x = workloads.uniform((N, 3, 224, 224), 7)
        if layout == "HWCN":
            x = x.transpose(2, 3, 1, 0).copy()
        xd = torch.from_numpy(x).cuda()
        y = torch.empty(net.shape(net.n_layers), dtype=torch.float32, device="cuda")
        s = torch.cuda.Stream()
        res = {}
        with torch.cuda.stream(s):
            for mode in ("eager", "graph"):
                t_end = time.perf_counter() + 0.2
                while time.perf_counter() < t_end:
                    net.forward(xd, out=y, graph=mode == "graph", stream=s)
                    s.synchronize()
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record(s)
                for _ in range(reps):
                    net.forward(xd, out=y, graph=mode == "graph", stream=s)
                e1.record(s)
                s.synchronize()
                ms = e0.elapsed_time(e1) / reps
                res[mode] = {"ms": round(ms, 3), "conv_tflops": round(flops / ms / 1e9, 2),
                             "pct_peak": round(100 * flops / ms / 1e9 / PEAK_TFLOPS, 2)}
        arena, ws = net.memory()
        rec = {"net": name, "layout": layout, "N": N, "layers": len(layers),
               "convs": sum(1 for d in layers if d["op"] == "conv"), "conv_gflop": round(flops / 1e9, 2),
               "arena_mib": round(arena / 2**20, 1), "kept_mib": round(kept / 2**20, 1),
               "workspace_mib": round(ws / 2**20, 1), **res}
        recs.append(rec)
        emit(rec)
        net.close()
        del xd, y
        torch.cuda.empty_cache()
    return recs


def run_datavalues(workload, layer_names, reps, rounds, emit):
    import numpy as np
    import torch

    import workloads
    from paper_2307_04941_amd import mg3m

    mg3m.load_library()
    Ls = workloads.workload(workload)
    ws = torch.empty(1 << 28, dtype=torch.float32, device="cuda")
    for i, L in enumerate(Ls):
        if layer_names and L.name not in layer_names:
            continue
        Ho, Wo = mg3m.conv2d_out_dims(L.H, L.W, L.R, L.S, L.stride, L.pad)
        sx, sw = workloads.seeds(workload, i)
        xu, wu = workloads.make_tensors(L, sx, sw, "HWCN")
        xi, wi = workloads.make_tensors(L, sx, sw, "HWCN", "int")
        sets = {"uniform": (xu, wu), "int": (xi, wi), "zeros": (np.zeros_like(xu), np.zeros_like(wu))}
        dev = {k: (torch.from_numpy(a).cuda(), torch.from_numpy(b).cuda()) for k, (a, b) in sets.items()}
        y = torch.empty((Ho, Wo, L.K, L.N), dtype=torch.float32, device="cuda")
        args = (L.N, L.C, L.H, L.W, L.K, L.R, L.S, L.stride, L.pad, "HWCN")
        flops = 2.0 * L.N * L.K * L.C * L.R * L.S * Ho * Wo
        us = {k: [] for k in dev}
        for _ in range(rounds):
            for k, (xd, wd) in dev.items():
                for _ in range(3):
                    mg3m.conv2d_fwd_f32_ex(xd, wd, y, *args, ws, ws.numel() * 4, None)
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record()
                for _ in range(reps):
                    mg3m.conv2d_fwd_f32_ex(xd, wd, y, *args, ws, ws.numel() * 4, None)
                e1.record()
                torch.cuda.synchronize()
                us[k].append(e0.elapsed_time(e1) * 1e3 / reps)
        emit({"workload": workload, "layer": L.name, "plan": mg3m.conv2d_fwd_f32_plan_string(*args),
              "us_min": {k: round(min(v), 2) for k, v in us.items()},
              "tflops": {k: round(flops / min(v) / 1e6, 2) for k, v in us.items()}})
        del dev, y


def _mean(v):
    return round(sum(v) / len(v), 2) if v else None


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("mode", choices=["adaptability", "ablation", "acc64", "net", "datavalues"])
    ap.add_argument("--layers", default=None, help="datavalues: layer names, comma-separated (default: all)")
    ap.add_argument("--rounds", type=int, default=3, help="datavalues: interleaved rounds")
    ap.add_argument("--nets", default="vgg16,alexnet,resnet50")
    ap.add_argument("--batch", default="vgg16=64,alexnet=128,resnet50=64",
                    help="net: batch per network, name=N,...")
    ap.add_argument("--layout", default="HWCN")
    ap.add_argument("--workloads", default=None)
    ap.add_argument("--fixed", default=None,
                    help="ablation / acc64: fixed plans separated by ';' (ablation default: "
                         "tile=128x128,split=1;tile=32x64,split=1; acc64 default: none)")
    ap.add_argument("--reps", type=int, default=10)
    ap.add_argument("--out", default=None)
    a = ap.parse_args()

    out = open(a.out, "w") if a.out else None

    def emit(obj):
        line = json.dumps(obj)
        print(line, flush=True)
        if out:
            out.write(line + "\n")
            out.flush()

    if a.mode == "datavalues":
        run_datavalues(a.workloads or "vgg16_n64", a.layers.split(",") if a.layers else None, a.reps, a.rounds,
                       emit)
    elif a.mode == "net":
        batch = {k: int(v) for k, v in (kv.split("=") for kv in a.batch.split(","))}
        run_nets(a.nets.split(","), batch, a.layout, a.reps, emit)
    elif a.mode == "adaptability":
        names = (a.workloads.split(",") if a.workloads else
                 ["channel_scenes_n128", "batch_sweep", "filter_sweep_n128", "padstride_sweep_n128"])
        recs = run_scenes(names, [], a.reps, emit)
        groups = collections.defaultdict(list)
        for r in recs:
            pct = r["selector"]["pct_peak"]
            if r["workload"] == "channel_scenes_n128":
                groups["channels_" + r["scene"].split("_")[0]].append(pct)
            elif r["workload"] == "batch_sweep":
                groups[f"batch_B{r['N']}"].append(pct)
            elif r["workload"] == "filter_sweep_n128":
                groups[f"filter_{r['R']}x{r['R']}"].append(pct)
            elif r["workload"] == "padstride_sweep_n128":
                groups[f"pad{r['pad']}_stride{r['stride']}"].append(pct)
            else:
                groups[r["workload"]].append(pct)
        emit({"summary": "adaptability", "metric": "mean % of the fp32 MFMA peak per group",
              "groups": {g: _mean(v) for g, v in groups.items()},
              "max_pct_peak": max(r["selector"]["pct_peak"] for r in recs)})
    elif a.mode == "acc64":
        fixed = [p for p in (a.fixed or "").split(";") if p]
        names = a.workloads.split(",") if a.workloads else ["vgg16_n64", "resnet50_n32"]
        recs = run_scenes(names, [], a.reps, emit, acc64_plans=[None] + fixed)
        per_wl = collections.defaultdict(lambda: {"flop": 0.0, "us32": 0.0, "us64": 0.0})
        for r in recs:
            d = per_wl[r["workload"]]
            d["flop"] += r["gflop"] * 1e9
            d["us32"] += r["selector"]["us"]
            d["us64"] += r["acc64:selector"]["us"]
        emit({"summary": "acc64", "metric": "whole-workload TFLOPS, fp32 vs fp64 accumulation",
              "workloads": {w: {"fp32_tflops": round(d["flop"] / d["us32"] / 1e6, 2),
                                "acc64_tflops": round(d["flop"] / d["us64"] / 1e6, 2),
                                "acc64_pct_fp64_peak": round(100 * d["flop"] / d["us64"] / 1e6
                                                             / PEAK64_TFLOPS, 2)}
                            for w, d in per_wl.items()}})
    else:
        fixed = [p for p in (a.fixed or "tile=128x128,split=1;tile=32x64,split=1").split(";") if p]
        names = a.workloads.split(",") if a.workloads else ["batch_sweep"]
        recs = run_scenes(names, fixed, a.reps, emit)
        per_b = collections.defaultdict(lambda: collections.defaultdict(list))
        tiles = collections.defaultdict(dict)
        for r in recs:
            for key in ["selector"] + fixed:
                per_b[r["N"]][key].append(r[key]["pct_peak"])
            tiles[r["N"]][r["C"]] = r["selector_plan"]
        emit({"summary": "ablation", "metric": "mean % of the fp32 MFMA peak per batch size",
              "per_batch": {str(b): {k: _mean(v) for k, v in d.items()} for b, d in sorted(per_b.items())},
              # the paper's Table 2 comparison: mean efficiency of the selector
              # over that of each fixed mapping, minus one
              "selector_gain_pct": {str(b): {k: round(100 * (sum(d["selector"]) / sum(d[k]) - 1), 1)
                                             for k in fixed}
                                    for b, d in sorted(per_b.items())},
              "selector_plans": {str(b): v for b, v in sorted(tiles.items())}})
    if out:
        out.close()


if __name__ == "__main__":
    main()
