"""Summarise rocprofv3 output of a benchmark run into short text files.

    python -m paper_2307_04941_amd.rocprof_summary --workload vgg16_n64 \\
        --trace DIR --fetch DIR --write DIR --bench-log FILE --copy-mib 1024 --out DIR \\
        --command-trace "..." --command-fetch "..." --command-write "..."

--trace is a ``rocprofv3 --kernel-trace --stats -f csv`` directory, --fetch and
--write are ``rocprofv3 --pmc FETCH_SIZE`` / ``--pmc WRITE_SIZE`` directories of
runs that also copied --copy-mib MiB once with a plain copy kernel (bench.py
--copy-mib).  The dominant kernel is the one named in the benchmark's JSON
line (--bench-log).  HBM bytes per launch of that kernel are its FETCH_SIZE and
WRITE_SIZE (KiB per dispatch, averaged over its dispatches), each scaled by
the ratio of the copy's known size to what the same counter read for the copy.

Writes <out>/<kernel tag>_<workload>_kernel_stats.txt,
<out>/<kernel tag>_<workload>_traffic.txt and <out>/traffic_<workload>.json
(the figure bench.py reports as roofline.traffic while the dominant kernel's
code and launches are unchanged).

    python -m paper_2307_04941_amd.rocprof_summary --stats-only NAME --trace DIR \
        --out DIR --command-trace "..."

writes <out>/NAME_kernel_stats.txt only: the kernel-time table of any traced
program (e.g. a network forward through the executor), with the time grouped
by kernel family.

    python -m paper_2307_04941_amd.rocprof_summary --mfma DIR --workload vgg16_n64 \
        --bench-log FILE --out DIR --command-mfma "..."

writes <out>/<kernel tag>_<workload>_mfma.txt: the dominant kernel's MFMA
utilisation per launch from a ``rocprofv3 --pmc GRBM_GUI_ACTIVE
SQ_VALU_MFMA_BUSY_CYCLES SQ_BUSY_CU_CYCLES`` run, and its HBM GB/s.

    python -m paper_2307_04941_amd.rocprof_summary --waves DIR --workload vgg16_n64 \
        --bench-log FILE --out DIR --command-waves "..."

writes <out>/<kernel tag>_<workload>_waves.txt: where the dominant kernel's
waves spend their cycles (waiting at s_waitcnt or a barrier, waiting for an
issue slot, issuing) and its LDS bank-conflict cycles, from a ``rocprofv3
--pmc SQ_WAVE_CYCLES SQ_WAIT_ANY SQ_WAIT_INST_ANY SQ_ACTIVE_INST_ANY
SQ_LDS_BANK_CONFLICT`` run.

    python -m paper_2307_04941_amd.rocprof_summary --clock DIR --kernel SUBSTR \
        --groups uniform:13,int:13,zeros:13 --label NAME --out DIR --command-clock "..."

writes <out>/NAME_clock.txt: from a ``rocprofv3 --pmc GRBM_GUI_ACTIVE`` run,
the launches of the kernel whose name contains SUBSTR, in dispatch order,
cut into consecutive named groups of the given sizes (e.g. the data sets of
``experiments.py datavalues``); per group, the mean launch time, clock cycles
per XCD and effective clock.
"""
from __future__ import annotations

import argparse
import csv
import glob
import json
import os
import sys


def _csv(directory: str, suffix: str):
    files = glob.glob(os.path.join(directory, "**", f"*{suffix}"), recursive=True)
    if not files:
        raise FileNotFoundError(f"no *{suffix} under {directory}")
    with open(files[0]) as f:
        return list(csv.DictReader(f))


def per_dispatch(directory: str, counter: str):
    """[(dispatch id, kernel name, value)] for one counter (summed over
    the instances rocprofv3 reports for a dispatch)."""
    acc = {}
    for r in _csv(directory, "counter_collection.csv"):
        if r["Counter_Name"] != counter:
            continue
        key = int(r["Dispatch_Id"])
        name, val = r["Kernel_Name"], float(r["Counter_Value"])
        if key in acc:
            acc[key] = (name, acc[key][1] + val)
        else:
            acc[key] = (name, val)
    return [(k, v[0], v[1]) for k, v in sorted(acc.items())]


def copy_scale(rows, known_kib: float):
    """Known size / counter reading of the plain copy: the largest copy-kernel
    dispatch of the run (the calibration copy dwarfs the input uploads)."""
    copies = [v for _, n, v in rows if "copyBuffer" in n and v > 0]
    if not copies:
        raise ValueError("no copy kernel dispatch in the counter run")
    v = max(copies)
    return known_kib / v, v


FAMILIES = [("conv_igemm_f32<", ", false>", "convolution (fp32, plain output)"),
            ("conv_igemm_f32<", ", true>", "convolution (fp32, fused add/ReLU)"),
            ("conv_igemm_f32_pt<", ", false>", "convolution (fp32, persistent, plain output)"),
            ("conv_igemm_f32_pt<", ", true>", "convolution (fp32, persistent, fused add/ReLU)"),
            ("conv_igemm_f32_m16<", ", false>", "convolution (fp32, 16-row tile, plain output)"),
            ("conv_igemm_f32_m16<", ", true>", "convolution (fp32, 16-row tile, fused add/ReLU)"),
            ("conv_igemm_acc64<", "", "convolution (fp64 accumulation)"),
            ("maxpool", "", "max pooling"),
            ("tail_reduce", "", "split-K reduction"),
            ("filter_kcrs_to_rsck", "", "NCHW filter copy")]


def timed_launch_us(directory: str, kernel: str, steps, per_step):
    """Mean duration (us) of the kernel's last steps * per_step launches in a
    --kernel-trace run, i.e. those of the benchmark's timed steps, which come
    after its warm-up steps; None without a trace file or enough launches."""
    if not steps or not per_step:
        return None
    try:
        rows = _csv(directory, "kernel_trace.csv")
    except FileNotFoundError:
        return None
    ds = sorted((int(r["Dispatch_Id"]), int(r["End_Timestamp"]) - int(r["Start_Timestamp"]))
                for r in rows if r["Kernel_Name"] == kernel)
    n = int(steps) * int(per_step)
    if len(ds) < n:
        return None
    return sum(d for _, d in ds[-n:]) / n / 1e3, n


def kernel_tag(kernel: str) -> str:
    """Short file-name tag of a kernel: its function name (persistent and
    16-row kernels keep their suffix) and its integer template arguments."""
    fn = kernel[:kernel.index("<")].split("::")[-1]
    args = kernel[kernel.index("<") + 1:kernel.index(">")].replace(" ", "").split(",")
    base = fn.replace("conv_igemm_f32", "conv_igemm")
    return base + "_" + "_".join(v for v in args if v.lstrip("-").isdigit())


def family(name: str) -> str:
    for head, tail, label in FAMILIES:
        if head in name and tail in name:
            return label
    return "other"


def stats_only(a):
    stats = _csv(a.trace, "kernel_stats.csv")
    total = sum(float(r["TotalDurationNs"]) for r in stats)
    lines = [f"rocprofv3 kernel statistics: {a.stats_only}", f"command: {a.command_trace}", "",
             "time by kernel family:"]
    fam = {}
    for r in stats:
        f = family(r["Name"])
        calls, ns = fam.get(f, (0, 0.0))
        fam[f] = (calls + int(r["Calls"]), ns + float(r["TotalDurationNs"]))
    for f, (calls, ns) in sorted(fam.items(), key=lambda kv: -kv[1][1]):
        lines.append(f"  {f:36s} {calls:7d} calls {ns / 1e6:10.3f} ms {100 * ns / total:6.2f}%")
    lines += ["", " calls     avg_us   total_ms    pct  kernel"]
    for r in sorted(stats, key=lambda r: -float(r["TotalDurationNs"])):
        lines.append(f"{int(r['Calls']):6d} {float(r['AverageNs']) / 1e3:10.2f} "
                     f"{float(r['TotalDurationNs']) / 1e6:10.3f} {float(r['Percentage']):6.2f}  {r['Name']}")
    os.makedirs(a.out, exist_ok=True)
    path = os.path.join(a.out, f"{a.stats_only}_kernel_stats.txt")
    with open(path, "w") as f:
        f.write("\n".join(lines) + "\n")
    print("\n".join(lines[:12]))
    return 0


def mfma_summary(a):
    """MFMA utilisation of the dominant kernel from a ``rocprofv3 --pmc
    GRBM_GUI_ACTIVE SQ_VALU_MFMA_BUSY_CYCLES SQ_BUSY_CU_CYCLES`` run: per
    launch, MFMA-busy SIMD cycles over the SIMD cycles the GPU clocked while
    the kernel ran (the counters are summed over the XCDs), the effective
    clock, and the HBM bytes of the traffic summary over the launch time."""
    with open(a.bench_log) as f:
        bench = json.loads([ln for ln in f if ln.startswith("{")][-1])
    kernel = bench["roofline"]["kernel"]
    agent = next(r for r in _csv(a.mfma, "agent_info.csv") if int(r.get("Simd_Count") or 0) > 0)
    xcc, simds = int(agent["Num_Xcc"]), int(agent["Simd_Count"])
    clk_max = float(agent["Max_Engine_Clk_Fcompute"]) * 1e6
    acc = {}
    for r in _csv(a.mfma, "counter_collection.csv"):
        if r["Kernel_Name"] != kernel:
            continue
        d = acc.setdefault(int(r["Dispatch_Id"]), {"ns": int(r["End_Timestamp"]) - int(r["Start_Timestamp"])})
        d[r["Counter_Name"]] = d.get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
    if not acc:
        raise ValueError(f"no dispatch of {kernel} in {a.mfma}")
    traffic = None
    tpath = os.path.join(a.out, f"traffic_{a.label or a.workload}.json")
    if os.path.exists(tpath):
        with open(tpath) as f:
            t = json.load(f)
        if t.get("kernel") == kernel:
            traffic = t["hbm_bytes_per_launch"]
    args = kernel[kernel.index("<") + 1:kernel.index(">")].replace(" ", "").split(",")
    tag = kernel_tag(kernel)
    lines = [f"MFMA utilisation of {kernel}, workload {a.workload}",
             f"command: {a.command_mfma}", "",
             f"GPU: {xcc} XCDs, {simds} SIMDs, {clk_max / 1e9:.2f} GHz maximum engine clock",
             "MFMA busy = SQ_VALU_MFMA_BUSY_CYCLES / (GRBM_GUI_ACTIVE / XCDs x SIMDs); "
             "clock = GRBM_GUI_ACTIVE / XCDs / kernel time", "",
             f"{'dispatch':>8} {'us':>9} {'clock GHz':>10} {'MFMA busy':>10} {'x clock/max':>12}"]
    tot_busy = tot_cyc = tot_ns = 0.0
    for d, v in sorted(acc.items()):
        cyc = v["GRBM_GUI_ACTIVE"] / xcc
        busy = v["SQ_VALU_MFMA_BUSY_CYCLES"] / (cyc * simds)
        clk = cyc / (v["ns"] * 1e-9)
        lines.append(f"{d:8d} {v['ns'] / 1e3:9.1f} {clk / 1e9:10.3f} {100 * busy:9.1f}% {100 * busy * clk / clk_max:11.1f}%")
        tot_busy += v["SQ_VALU_MFMA_BUSY_CYCLES"]; tot_cyc += cyc; tot_ns += v["ns"]
    busy = tot_busy / (tot_cyc * simds)
    clk = tot_cyc / (tot_ns * 1e-9)
    lines += ["", f"all {len(acc)} dispatches: MFMA busy {100 * busy:.1f}% of the clocked SIMD cycles at "
              f"{clk / 1e9:.3f} GHz on average = {100 * busy * clk / clk_max:.1f}% of the MFMA cycles at "
              f"{clk_max / 1e9:.2f} GHz (the fp32 MFMA peak's clock)"]
    if traffic is not None:
        gbs = traffic / (tot_ns / len(acc) * 1e-9) / 1e9
        lines.append(f"HBM traffic {traffic / 1e6:.1f} MB per launch (traffic_{a.workload}.json) over the "
                     f"mean launch time here: {gbs:.0f} GB/s = {100 * gbs / 8000:.1f}% of the 8.0 TB/s HBM peak "
                     f"(counter runs serialise dispatches; the benchmark's own launches run faster)")
    with open(os.path.join(a.out, f"{tag}_{a.label or a.workload}_mfma.txt"), "w") as f:
        f.write("\n".join(lines) + "\n")
    print("\n".join(lines[-3:]))
    return 0


WAVE_COUNTERS = ("SQ_WAVE_CYCLES", "SQ_WAIT_ANY", "SQ_WAIT_INST_ANY", "SQ_ACTIVE_INST_ANY")


def waves_summary(a):
    """Where the dominant kernel's waves spend their cycles, from a
    ``rocprofv3 --pmc SQ_WAVE_CYCLES SQ_WAIT_ANY SQ_WAIT_INST_ANY
    SQ_ACTIVE_INST_ANY SQ_LDS_BANK_CONFLICT ...`` run: the wave-cycles
    waiting at s_waitcnt or a barrier, waiting for an issue slot (the MFMA
    pipe busy with another wave's MFMA, or a dependency), and issuing, each
    over all wave-cycles, summed over the kernel's dispatches; and the LDS
    cycles lost to bank conflicts."""
    with open(a.bench_log) as f:
        bench = json.loads([ln for ln in f if ln.startswith("{")][-1])
    kernel = bench["roofline"]["kernel"]
    tot, dispatches = {}, set()
    for r in _csv(a.waves, "counter_collection.csv"):
        if r["Kernel_Name"] != kernel:
            continue
        dispatches.add(int(r["Dispatch_Id"]))
        tot[r["Counter_Name"]] = tot.get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
    missing = [c for c in WAVE_COUNTERS if c not in tot]
    if missing or not tot["SQ_WAVE_CYCLES"]:
        raise ValueError(f"no {', '.join(missing) or 'SQ_WAVE_CYCLES'} for {kernel} in {a.waves}")
    wc = tot["SQ_WAVE_CYCLES"]
    lines = [f"Wave states of {kernel}, workload {a.workload}",
             f"command: {a.command_waves}", "",
             f"{len(dispatches)} dispatches; fractions of all wave-cycles (SQ_WAVE_CYCLES):",
             f"  waiting at s_waitcnt or a barrier (SQ_WAIT_ANY):        {100 * tot['SQ_WAIT_ANY'] / wc:5.1f}%",
             f"  waiting for an issue slot (SQ_WAIT_INST_ANY):           {100 * tot['SQ_WAIT_INST_ANY'] / wc:5.1f}%",
             f"  issuing (SQ_ACTIVE_INST_ANY):                           {100 * tot['SQ_ACTIVE_INST_ANY'] / wc:5.1f}%"]
    if "SQ_LDS_BANK_CONFLICT" in tot:
        lines.append(f"LDS cycles stalled by bank conflicts (SQ_LDS_BANK_CONFLICT), all dispatches: "
                     f"{tot['SQ_LDS_BANK_CONFLICT']:.0f}")
    os.makedirs(a.out, exist_ok=True)
    with open(os.path.join(a.out, f"{kernel_tag(kernel)}_{a.label or a.workload}_waves.txt"), "w") as f:
        f.write("\n".join(lines) + "\n")
    print("\n".join(lines))
    return 0


def clock_summary(a):
    """Effective clock per group of launches (see the module docstring)."""
    agent = next(r for r in _csv(a.clock, "agent_info.csv") if int(r.get("Simd_Count") or 0) > 0)
    xcc = int(agent["Num_Xcc"])
    clk_max = float(agent["Max_Engine_Clk_Fcompute"]) * 1e6
    acc = {}
    for r in _csv(a.clock, "counter_collection.csv"):
        if r["Counter_Name"] != "GRBM_GUI_ACTIVE" or a.kernel not in r["Kernel_Name"]:
            continue
        d = acc.setdefault(int(r["Dispatch_Id"]), {"ns": int(r["End_Timestamp"]) - int(r["Start_Timestamp"]),
                                                   "cyc": 0.0, "name": r["Kernel_Name"]})
        d["cyc"] += float(r["Counter_Value"])
    launches = [acc[k] for k in sorted(acc)]
    groups = [(g.split(":")[0], int(g.split(":")[1])) for g in a.groups.split(",")]
    if sum(n for _, n in groups) != len(launches):
        raise ValueError(f"{len(launches)} launches of *{a.kernel}* against groups of {sum(n for _, n in groups)}")
    names = sorted({d["name"] for d in launches})
    lines = [f"Effective clock by group of launches: {', '.join(names)}",
             f"command: {a.command_clock}", "",
             f"GPU: {xcc} XCDs, {clk_max / 1e9:.2f} GHz maximum engine clock; "
             "clock = GRBM_GUI_ACTIVE / XCDs / launch time", "",
             f"{'group':>10} {'launches':>9} {'mean us':>9} {'Mcycles/XCD':>12} {'clock GHz':>10}"]
    i = 0
    for g, n in groups:
        part = launches[i:i + n]
        i += n
        ns = sum(d["ns"] for d in part) / n
        cyc = sum(d["cyc"] for d in part) / n / xcc
        lines.append(f"{g:>10} {n:9d} {ns / 1e3:9.1f} {cyc / 1e6:12.3f} {cyc / ns:10.3f}")
    os.makedirs(a.out, exist_ok=True)
    with open(os.path.join(a.out, f"{a.label}_clock.txt"), "w") as f:
        f.write("\n".join(lines) + "\n")
    print("\n".join(lines))
    return 0


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("--stats-only", default=None, metavar="NAME")
    ap.add_argument("--workload")
    ap.add_argument("--label", default=None,
                    help="workload part of the output file names (default: --workload), e.g. for a run "
                         "of selected layers")
    ap.add_argument("--trace")
    ap.add_argument("--fetch")
    ap.add_argument("--write")
    ap.add_argument("--bench-log")
    ap.add_argument("--copy-mib", type=float)
    ap.add_argument("--out", required=True)
    ap.add_argument("--command-trace", default="")
    ap.add_argument("--command-fetch", default="")
    ap.add_argument("--command-write", default="")
    ap.add_argument("--mfma", default=None, metavar="DIR",
                    help="rocprofv3 --pmc GRBM_GUI_ACTIVE SQ_VALU_MFMA_BUSY_CYCLES ... directory: "
                         "write <kernel>_<workload>_mfma.txt (needs --workload, --bench-log)")
    ap.add_argument("--command-mfma", default="")
    ap.add_argument("--clock", default=None, metavar="DIR",
                    help="rocprofv3 --pmc GRBM_GUI_ACTIVE directory: write <label>_clock.txt "
                         "(needs --kernel, --groups, --label)")
    ap.add_argument("--waves", default=None, metavar="DIR",
                    help="rocprofv3 --pmc SQ_WAVE_CYCLES SQ_WAIT_ANY SQ_WAIT_INST_ANY SQ_ACTIVE_INST_ANY ... "
                         "directory: write <kernel>_<workload>_waves.txt (needs --workload, --bench-log)")
    ap.add_argument("--command-waves", default="")
    ap.add_argument("--kernel", default="conv_igemm")
    ap.add_argument("--groups", default=None, help="name:launches,... in dispatch order")
    ap.add_argument("--command-clock", default="")
    a = ap.parse_args(argv)
    if a.clock:
        if not (a.groups and a.label):
            ap.error("--clock needs --groups and --label")
        return clock_summary(a)
    if a.stats_only:
        return stats_only(a)
    if a.mfma:
        return mfma_summary(a)
    if a.waves:
        if not (a.workload and a.bench_log):
            ap.error("--waves needs --workload and --bench-log")
        return waves_summary(a)
    if a.trace is None:
        ap.error("--trace is required without --mfma")
    for need in ("workload", "fetch", "write", "bench_log", "copy_mib"):
        if getattr(a, need) is None:
            ap.error(f"--{need.replace('_', '-')} is required without --stats-only")

    with open(a.bench_log) as f:
        bench = json.loads([ln for ln in f if ln.startswith("{")][-1])
    kernel = bench["roofline"]["kernel"]
    args = kernel[kernel.index("<") + 1:kernel.index(">")].replace(" ", "").split(",")
    tag = kernel_tag(kernel)
    os.makedirs(a.out, exist_ok=True)

    # ---- kernel statistics
    stats = _csv(a.trace, "kernel_stats.csv")
    lines = [f"rocprofv3 kernel statistics, workload {a.workload}",
             f"command: {a.command_trace}", "",
             f"{'calls':>6} {'avg_us':>10} {'total_ms':>10} {'pct':>6}  kernel"]
    dom = None
    for r in sorted(stats, key=lambda r: -float(r["TotalDurationNs"])):
        lines.append(f"{int(r['Calls']):6d} {float(r['AverageNs']) / 1e3:10.2f} "
                     f"{float(r['TotalDurationNs']) / 1e6:10.3f} {float(r['Percentage']):6.2f}  {r['Name']}")
        if r["Name"] == kernel:
            dom = r
    roof = bench["roofline"]
    lines += ["", f"dominant kernel (bench.py): {kernel}",
              f"  bench.py HIP-event average per launch: {roof['avg_launch_us']} us over its "
              f"{roof['launches_per_step']} launches per step ({', '.join(roof['layers'])})"]
    if dom is not None:
        lines.append(f"  rocprofv3 average per launch:          {float(dom['AverageNs']) / 1e3:.2f} us "
                     f"over {dom['Calls']} calls (warm-up included)")
    timed = timed_launch_us(a.trace, kernel, bench.get("steps"), roof.get("launches_per_step"))
    if timed is not None:
        lines.append(f"  rocprofv3 average over the timed steps: {timed[0]:.2f} us over the last {timed[1]} calls "
                     f"({bench['steps']} steps x {roof['launches_per_step']} launches; the warm-up's are left out)")
    lines += [f"  achieved {roof['achieved']} TFLOP/s of {roof['peak']} ({100 * roof['frac']:.1f}%)",
              f"bench.py value: {bench['value']} {bench['unit']} ({bench.get('pct_peak')}% of peak), "
              f"{bench['ms_per_step']} ms per step, kernel digest {bench['kernel_digest']}"]
    with open(os.path.join(a.out, f"{tag}_{a.label or a.workload}_kernel_stats.txt"), "w") as f:
        f.write("\n".join(lines) + "\n")

    # ---- HBM traffic of the dominant kernel
    known_kib = a.copy_mib * 1024.0
    fetch = per_dispatch(a.fetch, "FETCH_SIZE")
    write = per_dispatch(a.write, "WRITE_SIZE")
    fscale, fcopy = copy_scale(fetch, known_kib)
    wscale, wcopy = copy_scale(write, known_kib)
    fk = [v for _, n, v in fetch if n == kernel]
    wk = [v for _, n, v in write if n == kernel]
    if not fk or not wk:
        raise ValueError(f"no dispatch of {kernel} in the counter runs")
    fetch_b = sum(fk) / len(fk) * fscale * 1024.0
    write_b = sum(wk) / len(wk) * wscale * 1024.0
    alg_flops = roof["alg_flops_per_launch"]
    layers = [r for r in bench["layers"] if r["kernel"] == kernel]
    alg_bytes = sum(r["alg_bytes"] for r in layers) / len(layers)
    out = {
        "workload": a.workload, "kernel": kernel, "kernel_digest": bench["kernel_digest"],
        "hbm_bytes_per_launch": round(fetch_b + write_b),
        "fetch_bytes_per_launch": round(fetch_b), "write_bytes_per_launch": round(write_b),
        "fetch_scale": round(fscale, 4), "write_scale": round(wscale, 4),
        "copy_bytes": round(known_kib * 1024), "copy_fetch_kib": fcopy, "copy_write_kib": wcopy,
        "dispatches": len(fk), "alg_bytes_per_launch": round(alg_bytes),
        "alg_flops_per_launch": alg_flops,
        "command_fetch": a.command_fetch, "command_write": a.command_write,
    }
    with open(os.path.join(a.out, f"traffic_{a.label or a.workload}.json"), "w") as f:
        json.dump(out, f, indent=1)
    txt = [f"HBM traffic of {kernel}, workload {a.workload}",
           f"FETCH_SIZE run: {a.command_fetch}", f"WRITE_SIZE run: {a.command_write}", "",
           f"plain copy of {a.copy_mib:.0f} MiB: FETCH_SIZE read {fcopy:.0f} KiB (scale {fscale:.4f}), "
           f"WRITE_SIZE read {wcopy:.0f} KiB (scale {wscale:.4f})",
           f"dominant kernel, {len(fk)} dispatches: FETCH {fetch_b / 1e6:.1f} MB + WRITE {write_b / 1e6:.1f} MB "
           f"per launch (scaled) = {(fetch_b + write_b) / 1e6:.1f} MB",
           f"algorithmic bytes per launch (each tensor once): {alg_bytes / 1e6:.1f} MB; "
           f"measured / algorithmic = {(fetch_b + write_b) / alg_bytes:.2f}",
           "", "per dispatch (KiB, unscaled): FETCH_SIZE / WRITE_SIZE"]
    for (d, _, fv), (_, _, wv) in zip([x for x in fetch if x[1] == kernel], [x for x in write if x[1] == kernel]):
        txt.append(f"  dispatch {d}: {fv:.0f} / {wv:.0f}")
    with open(os.path.join(a.out, f"{tag}_{a.label or a.workload}_traffic.txt"), "w") as f:
        f.write("\n".join(txt) + "\n")
    print(json.dumps(out))


if __name__ == "__main__":
    sys.exit(main())
