"""The profile summariser on small synthetic rocprofv3 outputs: HBM traffic
scaled by the plain copy's known size, and MFMA utilisation from the busy and
clock counters.  CPU only."""
import csv
import json
import os

import pytest

from paper_2307_04941_amd import rocprof_summary as rs

KERNEL = "void mg3m::conv_igemm_f32<0, 0, 3, 128, 128, 16, 2, 2, false>(mg3m::KArgs)"
COLS = ["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value", "Start_Timestamp", "End_Timestamp"]


def _counters(d, rows):
    os.makedirs(d, exist_ok=True)
    with open(os.path.join(d, "run_counter_collection.csv"), "w", newline="") as f:
        w = csv.DictWriter(f, COLS)
        w.writeheader()
        for r in rows:
            w.writerow(dict(zip(COLS, r)))


def _bench_log(path, layers):
    line = {"value": 1.0, "unit": "TFLOPS", "ms_per_step": 1.0, "pct_peak": 1.0, "kernel_digest": "abc",
            "roofline": {"kernel": KERNEL, "achieved": 1.0, "peak": 157.3, "frac": 0.01,
                         "alg_flops_per_launch": 1e9, "avg_launch_us": 1.0, "launches_per_step": 1,
                         "layers": ["l0"]},
            "layers": layers}
    with open(path, "w") as f:
        f.write("some warning\n" + json.dumps(line) + "\n")


def test_traffic_scaled_by_the_copy(tmp_path):
    # FETCH_SIZE reads half the copy's size (scale 2), WRITE_SIZE all of it (scale 1)
    _counters(tmp_path / "fetch", [(1, "__amd_rocclr_copyBuffer", "FETCH_SIZE", 512.0, 0, 1),
                                   (2, KERNEL, "FETCH_SIZE", 100.0, 0, 1),
                                   (3, KERNEL, "FETCH_SIZE", 300.0, 0, 1)])
    _counters(tmp_path / "write", [(1, "__amd_rocclr_copyBuffer", "WRITE_SIZE", 1024.0, 0, 1),
                                   (2, KERNEL, "WRITE_SIZE", 50.0, 0, 1),
                                   (3, KERNEL, "WRITE_SIZE", 150.0, 0, 1)])
    trace = tmp_path / "trace"
    os.makedirs(trace)
    with open(trace / "run_kernel_stats.csv", "w", newline="") as f:
        w = csv.DictWriter(f, ["Name", "Calls", "TotalDurationNs", "AverageNs", "Percentage"])
        w.writeheader()
        w.writerow({"Name": KERNEL, "Calls": 2, "TotalDurationNs": 2000, "AverageNs": 1000, "Percentage": 100})
    _bench_log(tmp_path / "bench.log", [{"kernel": KERNEL, "alg_bytes": 1000.0}])
    out = tmp_path / "out"
    rs.main(["--workload", "w", "--trace", str(trace), "--fetch", str(tmp_path / "fetch"),
             "--write", str(tmp_path / "write"), "--bench-log", str(tmp_path / "bench.log"),
             "--copy-mib", str(1024 / 1024), "--out", str(out)])
    t = json.load(open(out / "traffic_w.json"))
    # copy of 1 MiB = 1024 KiB: fetch scale 1024/512 = 2, write scale 1
    assert t["fetch_scale"] == pytest.approx(2.0) and t["write_scale"] == pytest.approx(1.0)
    assert t["fetch_bytes_per_launch"] == round(200.0 * 2.0 * 1024)
    assert t["write_bytes_per_launch"] == round(100.0 * 1.0 * 1024)
    assert t["hbm_bytes_per_launch"] == t["fetch_bytes_per_launch"] + t["write_bytes_per_launch"]


def test_mfma_utilisation(tmp_path):
    d = tmp_path / "mfma"
    os.makedirs(d)
    with open(d / "run_agent_info.csv", "w", newline="") as f:
        w = csv.DictWriter(f, ["Agent_Type", "Simd_Count", "Num_Xcc", "Max_Engine_Clk_Fcompute"])
        w.writeheader()
        w.writerow({"Agent_Type": "CPU", "Simd_Count": 0, "Num_Xcc": 0, "Max_Engine_Clk_Fcompute": 0})
        w.writerow({"Agent_Type": "GPU", "Simd_Count": 1024, "Num_Xcc": 8, "Max_Engine_Clk_Fcompute": 2400})
    # 1000 us at 2.0 GHz: 2e6 cycles per XCD, summed over 8 XCDs; MFMA busy on
    # 90% of 1024 SIMDs' cycles
    cyc = 2.0e6
    _counters(d, [(5, KERNEL, "GRBM_GUI_ACTIVE", 8 * cyc, 0, 1_000_000),
                  (5, KERNEL, "SQ_VALU_MFMA_BUSY_CYCLES", 0.9 * cyc * 1024, 0, 1_000_000),
                  (6, "other", "GRBM_GUI_ACTIVE", 1.0, 0, 10)])
    _bench_log(tmp_path / "bench.log", [])
    out = tmp_path / "out"
    os.makedirs(out)
    with open(out / "traffic_w.json", "w") as f:
        json.dump({"kernel": KERNEL, "hbm_bytes_per_launch": 4.0e9}, f)
    rs.main(["--mfma", str(d), "--workload", "w", "--bench-log", str(tmp_path / "bench.log"),
             "--out", str(out)])
    text = open(out / "conv_igemm_0_0_3_128_128_16_2_2_w_mfma.txt").read()
    assert "MFMA busy 90.0% of the clocked SIMD cycles at 2.000 GHz" in text
    assert "= 75.0% of the MFMA cycles at 2.40 GHz" in text          # 0.9 * 2.0 / 2.4
    assert "4000 GB/s = 50.0% of the 8.0 TB/s" in text                # 4 GB in 1 ms


def test_clock_by_group(tmp_path):
    d = tmp_path / "clock"
    os.makedirs(d)
    with open(d / "run_agent_info.csv", "w", newline="") as f:
        w = csv.DictWriter(f, ["Agent_Type", "Simd_Count", "Num_Xcc", "Max_Engine_Clk_Fcompute"])
        w.writeheader()
        w.writerow({"Agent_Type": "GPU", "Simd_Count": 1024, "Num_Xcc": 8, "Max_Engine_Clk_Fcompute": 2400})
    # two launches of 2e6 cycles per XCD at 2.0 GHz (1000 us), then two at
    # 2.4 GHz; another kernel in between does not count
    rows = [(1, KERNEL, "GRBM_GUI_ACTIVE", 8 * 2.0e6, 0, 1_000_000),
            (2, KERNEL, "GRBM_GUI_ACTIVE", 8 * 2.0e6, 0, 1_000_000),
            (3, "other", "GRBM_GUI_ACTIVE", 5.0, 0, 10),
            (4, KERNEL, "GRBM_GUI_ACTIVE", 8 * 2.0e6, 0, 833_333),
            (5, KERNEL, "GRBM_GUI_ACTIVE", 8 * 2.0e6, 0, 833_333)]
    _counters(d, rows)
    out = tmp_path / "out"
    rs.main(["--clock", str(d), "--kernel", "conv_igemm", "--groups", "slow:2,fast:2", "--label", "t",
             "--out", str(out)])
    text = open(out / "t_clock.txt").read().splitlines()
    slow = next(ln for ln in text if ln.strip().startswith("slow")).split()
    fast = next(ln for ln in text if ln.strip().startswith("fast")).split()
    assert slow[1:] == ["2", "1000.0", "2.000", "2.000"], slow
    assert fast[1:] == ["2", "833.3", "2.000", "2.400"], fast
    with pytest.raises(ValueError):         # the group sizes must cover every launch
        rs.main(["--clock", str(d), "--groups", "a:3", "--label", "t", "--out", str(out)])


def test_timed_launch_average_leaves_out_the_warm_up(tmp_path):
    d = tmp_path / "trace"
    os.makedirs(d)
    with open(d / "run_kernel_trace.csv", "w", newline="") as f:
        w = csv.DictWriter(f, ["Dispatch_Id", "Kernel_Name", "Start_Timestamp", "End_Timestamp"])
        w.writeheader()
        # two warm-up launches of 5 us, then 2 steps x 2 launches of 1, 2, 3, 4 us; another kernel between
        for i, us in enumerate([5, 5, 1, 2, 3, 4]):
            w.writerow({"Dispatch_Id": 2 * i + 1, "Kernel_Name": KERNEL, "Start_Timestamp": 0,
                        "End_Timestamp": us * 1000})
            w.writerow({"Dispatch_Id": 2 * i + 2, "Kernel_Name": "other", "Start_Timestamp": 0,
                        "End_Timestamp": 99_000})
    assert rs.timed_launch_us(str(d), KERNEL, 2, 2) == (2.5, 4)
    assert rs.timed_launch_us(str(d), KERNEL, 4, 2) is None          # fewer launches than the steps need
    assert rs.timed_launch_us(str(tmp_path / "none"), KERNEL, 2, 2) is None


def test_wave_states(tmp_path):
    d = tmp_path / "waves"
    os.makedirs(d)
    # two dispatches of the dominant kernel: 1000 + 3000 wave-cycles, of which
    # 200 + 600 waiting, 700 + 2100 waiting for issue, 100 + 300 issuing; the
    # other kernel does not count
    rows = []
    for disp, scale in ((1, 1.0), (3, 3.0)):
        for name, v in (("SQ_WAVE_CYCLES", 1000), ("SQ_WAIT_ANY", 200), ("SQ_WAIT_INST_ANY", 700),
                        ("SQ_ACTIVE_INST_ANY", 100), ("SQ_LDS_BANK_CONFLICT", 0)):
            rows.append((disp, KERNEL, name, v * scale, 0, 1000))
    rows.append((2, "other", "SQ_WAIT_ANY", 1e9, 0, 10))
    _counters(d, rows)
    _bench_log(tmp_path / "bench.log", [])
    out = tmp_path / "out"
    rs.main(["--waves", str(d), "--workload", "w", "--bench-log", str(tmp_path / "bench.log"), "--out", str(out)])
    text = open(out / f"{rs.kernel_tag(KERNEL)}_w_waves.txt").read()
    assert "2 dispatches" in text
    lines = text.splitlines()
    pct = [float(ln.split()[-1].rstrip("%")) for ln in lines if ln.strip().startswith(("waiting", "issuing"))]
    assert pct == [20.0, 70.0, 10.0], pct
    assert "bank conflicts (SQ_LDS_BANK_CONFLICT), all dispatches: 0" in text
    with pytest.raises(ValueError):          # a counter the summary needs is missing
        _counters(d, [r for r in rows if r[2] != "SQ_WAIT_INST_ANY"])
        rs.main(["--waves", str(d), "--workload", "w", "--bench-log", str(tmp_path / "bench.log"),
                 "--out", str(out)])
