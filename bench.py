#!/usr/bin/env python3
"""Throughput of the MI355X fp32 implicit-GEMM convolution on one GPU.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload vgg16_n64]

A step is one forward pass of every conv layer of the workload (default: the
13 VGG-16 conv layers at batch 64, 224x224 input), each layer a call of the
C ABI's conv2d_fwd_f32 on device-resident seeded synthetic inputs.  Prints
one JSON line: aggregate fp32 TFLOPS (2*N*K*C*R*S*Ho*Wo per layer), the
per-layer TFLOPS and % of the 157.3 TFLOPS fp32-MFMA peak, the roofline
figures of the dominant kernel, and the fp64 CPU oracle timed on a bounded
sample of the same layers.
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

PEAK_TFLOPS = 157.3          # MI355X dense fp32 MFMA
HBM_GBS = 8000.0             # MI355X HBM3E
METRIC = "fp32 conv TFLOPS and % of MI355X fp32 MFMA peak per layer, 1 GPU"


def kernel_digest(name: str, launches) -> str:
    """Digest of one kernel's machine code (from the build's
    kernel_digests.json) and of the launches a step makes of it (layer, tile,
    schedule, grid): HBM-traffic counters taken on this kernel in this
    workload are reused exactly while both are unchanged.  None if the build
    recorded no digest for it."""
    path = os.path.join(ROOT, "paper_2307_04941_amd", "kernel_digests.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        code = json.load(f).get(name)
    if code is None:
        return None
    h = hashlib.sha256(code.encode())
    for r in launches:
        h.update(f"|{r['layer']}:{r['tile']}:{r['dp_tiles']}:{r['tail_tiles']}:{r['split']}:{r['grid']}".encode())
    return h.hexdigest()[:16]


def kernel_name(plan) -> str:
    """The main kernel's symbol as rocprofv3 prints it (its template arguments:
    layout, filter loader, patch loader, tile rows, columns, depth, waves, and
    false for the plain output stage the benchmark uses)."""
    fn = ("conv_igemm_f32_pt" if plan.get("persistent") else          # persistent whole tiles
          "conv_igemm_f32_m16" if plan["mt"] == 16 else "conv_igemm_f32")  # 16-row tiles: 16x16x4 MFMAs
    return (f"void mg3m::{fn}<{plan['layout']}, {plan['a_mode']}, {plan['b_mode']}, "
            f"{plan['mt']}, {plan['nt']}, {plan['kt']}, {plan['waves_m']}, {plan['waves_n']}, false>"
            f"(mg3m::KArgs)")


def layer_flops(L, Ho, Wo) -> float:
    return 2.0 * L.N * L.K * L.C * L.R * L.S * Ho * Wo


def layer_alg_bytes(L, Ho, Wo) -> float:
    # each tensor read or written once; input rows/cols never touched by a tap
    # (1x1 stride-2 layers) are not counted
    if L.R == 1 and L.S == 1 and L.pad == 0:
        ht, wt = Ho, Wo
    else:
        ht, wt = L.H, L.W
    return 4.0 * (L.N * L.C * ht * wt + L.K * L.C * L.R * L.S + L.N * L.K * Ho * Wo)


def cpu_baseline(layers, tensors, budget_s: float):
    """Time the fp64 oracle on a seeded sample of outputs of every layer,
    growing the sample until about `budget_s` seconds of CPU work."""
    import numpy as np
    import oracle
    cores = len(os.sched_getaffinity(0))
    os.environ.setdefault("OMP_NUM_THREADS", str(cores))
    rng = np.random.Generator(np.random.PCG64(7))
    pts = 256
    total_flops = 0.0
    total_t = 0.0
    n_pts = 0
    while True:
        t0 = time.perf_counter()
        for (L, Ho, Wo), (x, w) in zip(layers, tensors):
            n_out = L.N * L.K * Ho * Wo
            idx = rng.integers(0, n_out, pts)
            oracle.conv2d_points(x, w, idx, L.stride, L.pad, "HWCN")
            total_flops += 2.0 * L.C * L.R * L.S * pts
            n_pts += pts
        total_t += time.perf_counter() - t0
        if total_t >= budget_s or pts >= 1 << 22:
            break
        pts *= 2
    return {
        "value": total_flops / total_t / 1e12,
        "unit": "TFLOPS",
        "cores": int(os.environ.get("OMP_NUM_THREADS", cores)),
        "kind": "oracle",
        "sample": f"{n_pts} output elements drawn uniformly from every layer of the workload "
                  f"(same seeded inputs), {total_t:.1f} s of fp64 seven-loop direct convolution; "
                  f"throughput counts 2*C*R*S flop per output",
    }


def launch_floor_us(mg3m, torch, stream, reps=100):
    """Average time of back-to-back launches of an empty kernel on the stream
    (the floor under layers that run for a few microseconds)."""
    for _ in range(10):
        mg3m.mg3m_launch_empty(stream.cuda_stream)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(reps):
        mg3m.mg3m_launch_empty(stream.cuda_stream)
    e1.record(stream)
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) * 1e3 / reps


def ceilings(mg3m, torch, stream, dev):
    """The chip's sustained fp32-MFMA rate (an MFMA-only kernel, four waves
    per SIMD) and its streaming HBM bandwidth (16-byte copy and fill of
    1 GiB): best of five timed launches each, HIP events on the stream."""
    sp = stream.cuda_stream

    def best_ms(launch, reps=5):
        launch()
        torch.cuda.synchronize()
        out = []
        for _ in range(reps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            launch()
            e1.record(stream)
            torch.cuda.synchronize()
            out.append(e0.elapsed_time(e1))
        return min(out)

    blocks, iters = 256 * 4, 20000
    sink = torch.empty(blocks * 256, dtype=torch.float32, device=dev)
    flops = [0.0]

    def mfma():
        flops[0] = mg3m.mg3m_probe_mfma_f32(sink, blocks, iters, sp)
    ms_mfma = best_ms(mfma)
    nbytes = 1 << 30
    src = torch.zeros(nbytes // 4, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    ms_copy = best_ms(lambda: mg3m.mg3m_probe_copy(src, dst, nbytes, sp))
    ms_fill = best_ms(lambda: mg3m.mg3m_probe_fill(dst, nbytes, sp))
    del src, dst, sink
    return {
        "mfma_f32_tflops": round(flops[0] / ms_mfma / 1e9, 2),
        "mfma_f32_frac_of_peak": round(flops[0] / ms_mfma / 1e9 / PEAK_TFLOPS, 4),
        "copy_gbs": round(2 * nbytes / ms_copy / 1e6, 1),
        "fill_gbs": round(nbytes / ms_fill / 1e6, 1),
        "hbm_peak_gbs": HBM_GBS,
        "how": (f"mfma_probe: {blocks} work-groups x 4 waves x {iters} rounds of 8 independent "
                f"v_mfma_f32_32x32x2_f32 on registers; copy_probe / fill_probe: 16-byte accesses over "
                f"1 GiB, four in flight per thread, one 16 KB block per work-group (copy counts read + "
                f"write); best of 5"),
    }


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="vgg16_n64")
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="CPU work budget of the oracle baseline (0 = skip)")
    ap.add_argument("--layers", default=None,
                    help="comma-separated layer names of the workload to run (default: all); "
                         "for profiling single layers")
    ap.add_argument("--plan", default=None, help="plan override for every layer (diagnostics)")
    ap.add_argument("--cold-steps", type=int, default=3,
                    help="steps of the cold pass: a 512 MiB write before every layer, outside the "
                         "timed region (0 = skip)")
    ap.add_argument("--probes", action="store_true",
                    help="also measure the chip's sustained fp32-MFMA rate and streaming bandwidth")
    ap.add_argument("--probes-only", action="store_true",
                    help="only the launch floor and the ceiling probes (for profiling them)")
    ap.add_argument("--copy-mib", type=int, default=0,
                    help="before the warm-up, copy a buffer of this many MiB once (a plain copy "
                         "kernel of known size, to scale the HBM byte counters of a profile run)")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path "
              "(one process drives one GPU)", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import workloads
    from paper_2307_04941_amd import mg3m

    mg3m.load_library()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if args.probes_only:
        st = torch.cuda.current_stream()
        print(json.dumps({"launch_floor_us": round(launch_floor_us(mg3m, torch, st), 2),
                          "ceilings": ceilings(mg3m, torch, st, dev)}), flush=True)
        return
    layers_def = workloads.workload(args.workload)
    if args.layers:
        want = args.layers.split(",")
        unknown = [n for n in want if n not in {L.name for L in layers_def}]
        if unknown:
            print(f"unknown layer(s) {unknown} in workload {args.workload}", file=sys.stderr)
            sys.exit(2)
    # the seeds follow each layer's place in the whole workload
    chosen = [(i, L) for i, L in enumerate(layers_def) if not args.layers or L.name in args.layers.split(",")]

    # ---- inputs: seeded, generated on the host, resident in HBM before timing
    layers, tensors, dev_bufs = [], [], []
    for i, L in chosen:
        sx, sw = workloads.seeds(args.workload, i)
        x, w = workloads.make_tensors(L, sx, sw, "HWCN")
        Ho, Wo = mg3m.conv2d_out_dims(L.H, L.W, L.R, L.S, L.stride, L.pad)
        xd = torch.from_numpy(x).to(dev)
        wd = torch.from_numpy(w).to(dev)
        yd = torch.empty((Ho, Wo, L.K, L.N), dtype=torch.float32, device=dev)
        layers.append((L, Ho, Wo))
        tensors.append((x, w))
        dev_bufs.append((xd, wd, yd))
    torch.cuda.synchronize()

    stream = torch.cuda.current_stream()
    sp = stream.cuda_stream

    if args.copy_mib > 0:
        n = args.copy_mib * (1 << 20) // 4
        src = torch.zeros(n, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    # timing events without the system-scope fence of a default HIP event (a
    # default event writes back and invalidates the caches when it is
    # reached, which costs the next kernel; these only take timestamps)
    def new_event():
        return mg3m.TimingEvent()

    def one_step(evs=None):
        for j, ((L, Ho, Wo), (xd, wd, yd)) in enumerate(zip(layers, dev_bufs)):
            if evs is not None:
                mg3m.mg3m_time_next_kernel(evs[j][0], evs[j][1])
            if args.plan:
                mg3m.conv2d_fwd(xd, wd, L.stride, L.pad, "HWCN", plan=args.plan, out=yd)
            else:
                mg3m.conv2d_fwd_f32(xd, wd, yd, L.N, L.C, L.H, L.W, L.K, L.R, L.S,
                                    L.stride, L.pad, "HWCN", sp)
        if evs is not None:
            evs[-1][0].record(sp)

    for _ in range(args.warmup):
        one_step()
    torch.cuda.synchronize()

    # ---- timed region: exactly K steps.  Per layer and step, two timing
    # events around the main convolution kernel alone (mg3m_time_next_kernel
    # records them on the stream the kernel runs on), and one event at the end
    # of the step.  A layer's time runs from its main kernel's start to the
    # next layer's (the end of the step for the last layer): its kernels, any
    # tail reduction and the launch gaps.  Default HIP events in these places,
    # each with its cache-flushing fence, cost about 0.15 ms per VGG-16 step;
    # the timing events about 0.08 ms.
    evs = [[tuple(new_event() for _ in range(2)) for _ in layers] + [(new_event(),)]
           for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(args.steps):
        one_step(evs[k])
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0

    step_flops = sum(layer_flops(L, Ho, Wo) for (L, Ho, Wo) in layers)
    value = step_flops * args.steps / elapsed / 1e12

    # ---- cold pass (outside the contract's timed region): before every layer
    # a 512 MiB write (more than the 256 MB Infinity Cache and the 8 x 4 MB
    # L2) evicts what earlier work left in the caches; the layer is timed from
    # its main kernel's start to an event recorded after the call (its
    # kernels, any tail reduction, their launch gap).
    cold = None
    if args.cold_steps > 0:
        flush = torch.empty((512 << 20) // 4, dtype=torch.float32, device=dev)
        cold_us = np.zeros((args.cold_steps, len(layers)))
        for k in range(args.cold_steps):
            for j, ((L, Ho, Wo), (xd, wd, yd)) in enumerate(zip(layers, dev_bufs)):
                mg3m.mg3m_probe_fill(flush, flush.numel() * 4, sp)
                e0, e1, e2 = new_event(), new_event(), new_event()
                mg3m.mg3m_time_next_kernel(e0, e1)
                if args.plan:
                    mg3m.conv2d_fwd(xd, wd, L.stride, L.pad, "HWCN", plan=args.plan, out=yd)
                else:
                    mg3m.conv2d_fwd_f32(xd, wd, yd, L.N, L.C, L.H, L.W, L.K, L.R, L.S,
                                        L.stride, L.pad, "HWCN", sp)
                e2.record(sp)
                torch.cuda.synchronize()
                cold_us[k, j] = e0.elapsed_ms(e2) * 1e3
        del flush
        cold_layer = np.median(cold_us, axis=0)
        cold_step_us = float(cold_layer.sum())
        cold = {"value": round(step_flops / cold_step_us / 1e6, 3), "unit": "TFLOPS",
                "ms_per_step": round(cold_step_us / 1e3, 3), "steps": args.cold_steps,
                "flush_mib": 512,
                "how": "sum over layers of the median (over steps) of each layer's time, main kernel "
                       "start to the end of its call, each layer after a 512 MiB write"}

    per_layer = []
    for j, (L, Ho, Wo) in enumerate(layers):
        us_steps = np.array([evs[k][j][0].elapsed_ms(evs[k][j + 1][0]) for k in range(args.steps)]) * 1e3
        us = float(np.mean(us_steps))
        kus = float(np.mean([evs[k][j][0].elapsed_ms(evs[k][j][1]) for k in range(args.steps)])) * 1e3
        fl = layer_flops(L, Ho, Wo)
        by = layer_alg_bytes(L, Ho, Wo)
        plan = mg3m.conv2d_fwd_f32_plan_info(L.N, L.C, L.H, L.W, L.K, L.R, L.S, L.stride, L.pad,
                                             "HWCN", args.plan)
        ai = fl / by
        attainable = min(PEAK_TFLOPS, ai * HBM_GBS / 1e3)
        per_layer.append({
            "layer": L.name, "N": L.N, "C": L.C, "H": L.H, "K": L.K, "R": L.R, "stride": L.stride,
            "pad": L.pad, "us": round(us, 2), "us_min": round(float(us_steps.min()), 2),
            "us_p90": round(float(np.percentile(us_steps, 90)), 2), "kernel_us": round(kus, 2),
            "tflops": round(fl / us / 1e6, 2),
            "pct_peak": round(100 * fl / us / 1e6 / PEAK_TFLOPS, 1),
            "pct_roofline": round(100 * fl / us / 1e6 / attainable, 1),
            "bound": "mfma" if ai * HBM_GBS / 1e3 >= PEAK_TFLOPS else "hbm",
            "tile": f"{plan['mt']}x{plan['nt']}x{plan['kt']}", "split": plan["split"],
            "dp_tiles": plan["dp_tiles"], "tail_tiles": plan["tail_tiles"],
            "grid": plan["grid"], "kernel": kernel_name(plan),
            "flops": fl, "alg_bytes": by,
        })
        if cold is not None:
            cu = float(cold_layer[j])
            per_layer[-1].update({
                "cold_us": round(cu, 2), "cold_us_min": round(float(cold_us[:, j].min()), 2),
                "cold_us_p90": round(float(np.percentile(cold_us[:, j], 90)), 2),
                "cold_tflops": round(fl / cu / 1e6, 2), "cold_pct_peak": round(100 * fl / cu / 1e6 / PEAK_TFLOPS, 1)})

    # dominant kernel: the instantiation with the largest share of kernel time
    groups = {}
    for r in per_layer:
        g = groups.setdefault(r["kernel"], {"us": 0.0, "flops": 0.0, "n": 0, "layers": []})
        g["us"] += r["kernel_us"]
        g["flops"] += r["flops"]
        g["n"] += 1
        g["layers"].append(r["layer"])
    dname, dg = max(groups.items(), key=lambda kv: kv[1]["us"])
    achieved = dg["flops"] / dg["us"] / 1e6
    digest = kernel_digest(dname, [r for r in per_layer if r["kernel"] == dname])
    traffic = None
    prof = os.path.join(ROOT, "profiles", f"traffic_{args.workload}.json")
    if os.path.exists(prof) and not args.plan and digest is not None:
        with open(prof) as f:
            t = json.load(f)
        if t.get("kernel_digest") == digest and t.get("kernel") == dname:
            traffic = t.get("hbm_bytes_per_launch")
    roofline = {
        "bound": "mfma", "achieved": round(achieved, 2), "peak": PEAK_TFLOPS, "unit": "TFLOP/s",
        "frac": round(achieved / PEAK_TFLOPS, 4), "traffic": traffic,
        "kernel": dname,
        "layers": dg["layers"],
        "launches_per_step": dg["n"],
        "alg_flops_per_launch": dg["flops"] / dg["n"],
        "avg_launch_us": round(dg["us"] / dg["n"], 2),
    }

    # layers whose roofline time is under 10 us are bound by launch latency:
    # they are reported against the empty-kernel launch floor
    floor_us = round(launch_floor_us(mg3m, torch, stream), 2)
    for r in per_layer:
        r["roofline_us"] = round(max(r["flops"] / (PEAK_TFLOPS * 1e6), r["alg_bytes"] / (HBM_GBS * 1e3)), 2)
        r["latency_bound"] = r["roofline_us"] < 10.0

    cpu = None
    if args.cpu_seconds > 0:
        cpu = cpu_baseline(layers, tensors, args.cpu_seconds)

    out = {
        "metric": METRIC,
        "value": round(value, 3),
        "unit": "TFLOPS",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(elapsed / args.steps * 1e3, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic (seeded uniform[-1,1) inputs, He-normal filters; HWCN layout)",
        "config": {"workload": args.workload, "layers": len(layers),
                   "batch": layers[0][0].N, "layout": "HWCN",
                   "gflop_per_step": round(step_flops / 1e9, 3)},
        "pct_peak": round(100 * value / PEAK_TFLOPS, 2),
        "roofline": roofline,
        "cpu_baseline": cpu,
        "cold": cold,
        "launch_floor_us": floor_us,
        "layers": per_layer,
        "kernel_digest": digest,
    }
    if args.probes:
        out["ceilings"] = ceilings(mg3m, torch, stream, dev)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
