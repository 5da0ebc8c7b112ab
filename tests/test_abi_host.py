"""Host-side checks of the C ABI (no GPU needed): the library loads and
exports every function include/mg3m.h declares; validation rejects bad
arguments with the documented status before anything reaches the GPU; the
planner's plans cover the output and partition the reduction; the padding
metric reproduces the paper's printed example."""
import glob
import json
import os
import re
import sys

import numpy as np
import pytest

import oracle
import workloads
from paper_2307_04941_amd import mg3m

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "mg3m.h")
GOLDEN = os.path.join(ROOT, "tests", "golden")

# fake, never dereferenced device addresses: every call below fails validation
X, Wp, Y = 0x100000, 0x200000, 0x300000


def declared_functions(header=HEADER):
    text = open(header).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(\w+)\s*\(", text, flags=re.M)))


def test_library_exports_every_declared_function():
    lib = mg3m.load_library()
    names = declared_functions()
    assert "conv2d_fwd_f32" in names and len(names) >= 9, names
    headers = sorted(glob.glob(os.path.join(ROOT, "include", "*.h")))
    assert len(headers) >= 2, headers
    for h in headers:
        for n in declared_functions(h):
            assert hasattr(lib, n), f"{n} declared in {os.path.basename(h)} but not exported"


def test_measurement_calls_validate_before_launching():
    """The measurement kernels' argument checks (no GPU needed)."""
    lib = mg3m.load_library()
    import ctypes
    fl = ctypes.c_double()
    assert lib.mg3m_probe_mfma_f32(None, 1, 1, None, ctypes.byref(fl)) == 1
    assert lib.mg3m_probe_mfma_f32(X, 0, 1, None, ctypes.byref(fl)) == 10
    assert lib.mg3m_probe_mfma_f32(X, 1, 0, None, ctypes.byref(fl)) == 10
    assert lib.mg3m_probe_copy(X, Y, 15, None) == 10
    assert lib.mg3m_probe_copy(X + 4, Y, 64, None) == 9
    assert lib.mg3m_probe_copy(X, X + 32, 64, None) == 5
    assert lib.mg3m_probe_fill(None, 64, None) == 1
    assert lib.mg3m_probe_fill(Y, 0, None) == 10
    assert lib.mg3m_timing_event_create(None) == 1
    assert lib.mg3m_timing_event_record(None, None) == 1
    assert lib.mg3m_timing_event_elapsed_ms(None, None, None) == 1
    assert lib.mg3m_timing_event_destroy(None) == 1


def test_status_strings():
    for code in range(0, 11):
        s = mg3m.mg3m_status_string(code)
        assert s.startswith("MG3M_")
    assert "unknown" in mg3m.mg3m_status_string(99)


def _call(*shape, layout=0, x=X, w=Wp, y=Y):
    lib = mg3m.load_library()
    return lib.conv2d_fwd_f32(x, w, y, *shape, layout, None)


GOOD = (2, 8, 10, 10, 16, 3, 3, 1, 1)


@pytest.mark.parametrize("kw,status", [
    (dict(x=None), 1), (dict(w=None), 1), (dict(y=None), 1),
    (dict(x=X + 2), 9), (dict(y=Y + 1), 9),
    (dict(layout=2), 3), (dict(layout=-1), 3),
])
def test_pointer_and_layout_errors(kw, status):
    assert _call(*GOOD, **kw) == status
    assert mg3m.mg3m_last_error() != ""


@pytest.mark.parametrize("shape", [
    (0, 8, 10, 10, 16, 3, 3, 1, 1), (2, 0, 10, 10, 16, 3, 3, 1, 1), (2, 8, 10, 10, 0, 3, 3, 1, 1),
    (2, 8, 10, 10, 16, 3, 3, 0, 1), (2, 8, 10, 10, 16, 3, 3, 1, -1), (2, 8, 2, 2, 16, 5, 5, 1, 0),
    (2, 8, 10, 10, 16, 0, 3, 1, 1),
])
def test_shape_errors(shape):
    assert _call(*shape) == 2


def test_too_large():
    assert _call(1 << 16, 1 << 10, 64, 64, 16, 3, 3, 1, 1) == 4


def test_alias():
    # y placed inside x
    assert _call(*GOOD, x=X, y=X + 64) == 5


def test_nchw_tap_major_plan_needs_the_filter_copy_workspace():
    lib = mg3m.load_library()
    shape = (4, 32, 10, 10, 64, 3, 3, 1, 1)
    p = mg3m.conv2d_fwd_f32_plan_info(*shape, "NCHW", "split=1")
    assert p["b_mode"] == 5 and p["a_mode"] == 0
    assert mg3m.conv2d_fwd_f32_workspace_bytes(*shape, "NCHW", "split=1") == 4 * 64 * 288
    assert lib.conv2d_fwd_f32_ex(X, Wp, Y, *shape, 1, None, 0, b"split=1", None) == 6


def test_workspace_and_plan_errors():
    lib = mg3m.load_library()
    shape = (4, 64, 14, 14, 96, 3, 3, 1, 1)
    # forced split-K without a workspace
    rc = lib.conv2d_fwd_f32_ex(X, Wp, Y, *shape, 0, None, 0, b"split=4", None)
    assert rc == 6
    for bad in (b"tile=7x7", b"split=0", b"split=x", b"bogus=1", b"tile=128", b"xcd=1", b"tail=1", b"tail=x"):
        rc = lib.conv2d_fwd_f32_ex(X, Wp, Y, *shape, 0, None, 0, bad, None)
        assert rc == 7, bad


def test_out_dims_match_oracle():
    rng = np.random.Generator(np.random.PCG64(1))
    for _ in range(300):
        H, W = (int(v) for v in rng.integers(1, 40, 2))
        R = int(rng.integers(1, 8))
        st, pd = int(rng.integers(1, 5)), int(rng.integers(0, 5))
        if H + 2 * pd < R or W + 2 * pd < R:
            with pytest.raises(mg3m.Mg3mError):
                mg3m.conv2d_out_dims(H, W, R, R, st, pd)
            continue
        assert mg3m.conv2d_out_dims(H, W, R, R, st, pd) == oracle.out_dims(H, W, R, R, st, pd)


def _check_plan(shape, layout, plan=None):
    N, C, H, W, K, R, S, st, pd = shape
    p = mg3m.conv2d_fwd_f32_plan_info(N, C, H, W, K, R, S, st, pd, layout, plan)
    Ho, Wo = mg3m.conv2d_out_dims(H, W, R, S, st, pd)
    Mg, Ng, Kg = K, N * Ho * Wo, C * R * S
    assert (p["Mg"], p["Ng"], p["Kg"]) == (Mg, Ng, Kg)
    # tiles cover the output exactly once
    assert (p["tiles_m"] - 1) * p["mt"] < Mg <= p["tiles_m"] * p["mt"]
    assert (p["tiles_n"] - 1) * p["nt"] < Ng <= p["tiles_n"] * p["nt"]
    # whole tiles and tail tiles partition the tiles; the tail work-groups'
    # runs partition the tail tiles' k-tiles, none empty and none longer than
    # a tile
    kt = p["k_tiles"]
    assert kt == -(-Kg // p["kt"])
    tiles = p["tiles_m"] * p["tiles_n"]
    assert p["dp_tiles"] + p["tail_tiles"] == tiles
    tail, wgs = p["tail_tiles"], p["tail_wgs"]
    if tail:
        assert tail < wgs <= tail * kt < 2**31
        assert p["k_tiles_per_wg"] == -(-tail * kt // wgs) <= kt
        assert p["split"] == -(-wgs // tail) >= 2
    else:
        assert wgs == 0 and p["split"] == 1 and p["k_tiles_per_wg"] == kt
    # an NCHW call may run as HWCN on copies of x, w and y (via_hwcn): its
    # kernels are then the HWCN ones
    via = p["via_hwcn"] == 1
    assert not via or layout == "NCHW"
    klayout = "HWCN" if via else layout
    assert p["layout"] == (0 if klayout == "HWCN" else 1)
    if p["persistent"]:
        # persistent: every tile whole, fewer work-groups than tiles, each
        # looping over them
        assert tail == 0 and 1 <= p["grid"] < p["dp_tiles"] and p["grid"] % 256 == 0 or p["grid"] == p["dp_tiles"]
        assert p["b_mode"] in (0, 3, 6) and klayout == "HWCN" and p["mt"] != 16
    else:
        assert p["grid"] == p["dp_tiles"] + wgs <= 2**31 - 1
    # partials (slots up to wgs + tail - 2), plus the [R][S][C][K] filter copy
    # of a tap-major NCHW plan (b_mode 5), or the HWCN copies of x, w and y
    r256 = lambda b: -(-b // 256) * 256
    copy = r256(4 * Mg * Kg) if p["b_mode"] == 5 else 0
    if via:
        copy = r256(4 * N * C * H * W) + r256(4 * Mg * Kg) + r256(4 * Mg * Ng)
    # the direct-to-LDS one-tap loaders: HWCN, 32x32x2-MFMA tiles
    assert p["b_mode"] != 6 or (klayout == "HWCN" and p["mt"] != 16
                                and N % 4 == 0 and K % 4 == 0 and C % p["kt"] == 0)
    assert p["b_mode"] != 5 or (klayout == "NCHW" and C % p["kt"] == 0 and K % 4 == 0 and R * S > 1
                                and (st if isinstance(st, int) else st[1]) == 1)
    slots = wgs + tail - 1 if tail else 0
    assert p["workspace_bytes"] == 4 * slots * p["mt"] * p["nt"] + copy
    assert 0 < p["lds_bytes"] <= 160 * 1024
    assert 0 < p["pad_efficiency"] <= 1.0
    assert p["est_us"] > 0
    return p


def test_plans_for_every_catalogue_layer():
    for wl, (_, layers) in workloads.WORKLOADS.items():
        for L in layers:
            for layout in ("HWCN", "NCHW"):
                _check_plan((L.N, L.C, L.H, L.W, L.K, L.R, L.S, L.stride, L.pad), layout)


def test_plans_random_grid_and_overrides():
    rng = np.random.Generator(np.random.PCG64(2))
    tiles = ["128x128", "64x256", "256x64", "64x128", "128x64", "64x64", "32x128", "32x64",
             "128x32", "64x32", "256x128", "128x256", "128x128,kt=32", "16x64"]
    for _ in range(200):
        N = int(rng.integers(1, 65))
        C, K = (int(v) for v in rng.integers(1, 600, 2))
        H = int(rng.integers(1, 60))
        R = int(rng.choice([1, 3, 5, 7]))
        st, pd = int(rng.integers(1, 4)), int(rng.integers(0, 4))
        if H + 2 * pd < R:
            continue
        shape = (N, C, H, H, K, R, R, st, pd)
        _check_plan(shape, "HWCN")
        t = str(rng.choice(tiles))
        sp = int(rng.integers(1, 20))
        p = _check_plan(shape, "NCHW", f"tile={t},split={sp}")
        assert f"{p['mt']}x{p['nt']}" == t.split(",")[0]
        assert p["kt"] == (32 if "kt=32" in t else 16)
        assert p["split"] <= sp


def test_one_hip_runtime_per_process():
    """torch bundles HIP and HSA runtimes under ROCm's sonames: the binding
    loads torch first so that the library binds to those, and the process
    holds one HIP runtime whichever of the two the caller touches first."""
    import subprocess
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    code = ("from paper_2307_04941_amd import mg3m; mg3m.load_library(); import torch; "
            "m = open('/proc/self/maps').read(); "
            "print(len({l.split()[-1] for l in m.splitlines() if 'libamdhip64' in l}))")
    out = subprocess.run([sys.executable, "-c", code], cwd=root, capture_output=True, text=True, timeout=300)
    assert out.returncode == 0, out.stderr
    assert out.stdout.strip() == "1"


def test_stream_k_override():
    """sk=<g>: the tiles left over after whole rounds, their k-tiles dealt
    out to g work-groups; g must lie between the tail tiles and their
    k-tiles in total (g equal to the tail tiles runs them whole)."""
    small = (4, 64, 14, 14, 256, 3, 3, 1, 1)          # 256x64: 13 tiles, below one round
    base = _check_plan(small, "HWCN", "tile=256x64,tail=2")
    tail, kt = base["tail_tiles"], base["k_tiles"]
    assert (base["dp_tiles"], tail, kt) == (0, 13, 36)
    for g in (tail + 1, 27, 100, 467, tail * kt):
        p = _check_plan(small, "HWCN", f"tile=256x64,sk={g}")
        assert (p["dp_tiles"], p["tail_tiles"], p["tail_wgs"]) == (0, tail, g)
    p = _check_plan(small, "HWCN", f"tile=256x64,sk={tail}")
    assert (p["dp_tiles"], p["tail_wgs"]) == (13, 0)
    rounds = (24, 16, 111, 111, 32, 3, 3, 1, 1)       # whole rounds first
    r = _check_plan(rounds, "HWCN", "tile=256x64,tail=2")
    assert r["dp_tiles"] > 0 and r["tail_tiles"] > 0
    p = _check_plan(rounds, "HWCN", f"tile=256x64,sk={r['tail_tiles'] + 100}")
    assert (p["dp_tiles"], p["tail_tiles"], p["tail_wgs"]) == (r["dp_tiles"], r["tail_tiles"], r["tail_tiles"] + 100)
    # runs spanning two tiles only with the one-tap HWCN loader (b_mode 3) of
    # the fp32 kernel; runs that fall on tile boundaries are a split anywhere
    for layout, shape, via in (("NCHW", small, ",via=none"), ("HWCN", (3, 64, 14, 14, 256, 3, 3, 1, 1), "")):
        with pytest.raises(mg3m.Mg3mError) as ei:
            mg3m.conv2d_fwd_f32_plan_info(*shape, layout, f"tile=256x64,sk={tail + 1}{via}")
        assert ei.value.status == 7 and "one-tap HWCN" in mg3m.mg3m_last_error()
    # an NCHW call takes such runs when it runs as HWCN
    p = _check_plan(small, "NCHW", f"tile=256x64,sk={tail + 1}")
    assert p["via_hwcn"] == 1 and p["tail_wgs"] == tail + 1
    p = _check_plan(small, "NCHW", f"tile=256x64,sk={4 * tail},via=none")
    assert (p["tail_wgs"], p["split"], p["k_tiles_per_wg"]) == (4 * tail, 4, 9)
    for bad in (f"tile=256x64,sk={tail - 1}", f"tile=256x64,sk={tail * kt + 1}", "sk=0", "sk=x",
                "split=2,sk=20", "tail=2,sk=20", "split=2,tail=3"):
        with pytest.raises(mg3m.Mg3mError) as ei:
            mg3m.conv2d_fwd_f32_plan_info(*small, "HWCN", bad)
        assert ei.value.status == 7, bad


def test_selector_uses_full_rounds_for_small_layers():
    """A layer with fewer tiles than one round of resident work-groups
    (VGG-16's 14x14 layers at N=64) gets its reduction shared out over one
    full round, not a split that leaves part of a second round."""
    p = _check_plan((64, 512, 14, 14, 512, 3, 3, 1, 1), "HWCN")
    assert p["dp_tiles"] == 0 and p["tail_tiles"] > 0
    assert p["tail_wgs"] % 256 == 0


def test_plan_string_roundtrip():
    s = mg3m.conv2d_fwd_f32_plan_string(64, 512, 28, 28, 512, 3, 3, 1, 1, "HWCN", "tile=128x128,split=2")
    assert s.startswith("tile=128x128,") and "split=2" in s
    lib = mg3m.load_library()
    import ctypes
    buf = ctypes.create_string_buffer(8)
    assert lib.conv2d_fwd_f32_plan_string(64, 512, 28, 28, 512, 3, 3, 1, 1, 0, None, buf, 8) == 10


def test_padding_overhead_reproduces_paper_example():
    g = json.load(open(os.path.join(GOLDEN, "paper_arithmetic.json")))["padding_overhead"]
    f, d = mg3m.mg3m_padding_overhead(g["K"], g["N"], g["C"], g["Kr"], g["Nr"])
    assert round(100 * f, g["printed_decimals"]) == g["extra_compute_pct"]
    assert round(100 * d, g["printed_decimals"]) == g["extra_data_pct"]
    f0, d0 = mg3m.mg3m_padding_overhead(32, 48, 16, 4, 16)
    assert f0 == 0.0 and d0 == 0.0


def test_inception_5x5_layer_matches_paper_mm_unit():
    g = json.load(open(os.path.join(GOLDEN, "paper_arithmetic.json")))["inception3a_5x5_mm_unit"]
    L = [l for l in workloads.workload("alexnet_inception_n128") if l.name == "incep3a_5x5"][0]
    assert (L.K, L.N, L.C) == (g["M_oc"], g["N_batch"], g["K_ic"])


def test_time_next_kernel_arguments():
    lib = mg3m.load_library()
    assert lib.mg3m_time_next_kernel(None, None) == 0
    assert lib.mg3m_time_next_kernel(0x1000, None) == 10       # MG3M_ERR_ARG: one event only
    assert lib.mg3m_time_next_kernel(None, 0x1000) == 10
    assert lib.mg3m_time_next_kernel(None, None) == 0          # cleared again


def test_bench_refuses_more_than_one_gpu():
    import subprocess
    import sys
    p = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert p.returncode == 2
    assert "one GPU" in p.stderr


def test_out_dims_hw_match_oracle():
    rng = np.random.Generator(np.random.PCG64(3))
    for _ in range(300):
        H, W = (int(v) for v in rng.integers(1, 40, 2))
        R, S = (int(v) for v in rng.integers(1, 8, 2))
        sh, sw = (int(v) for v in rng.integers(1, 5, 2))
        ph, pw = (int(v) for v in rng.integers(0, 5, 2))
        if H + 2 * ph < R or W + 2 * pw < S:
            with pytest.raises(mg3m.Mg3mError):
                mg3m.conv2d_out_dims_hw(H, W, R, S, sh, sw, ph, pw)
            continue
        assert mg3m.conv2d_out_dims_hw(H, W, R, S, sh, sw, ph, pw) == \
            oracle.out_dims(H, W, R, S, (sh, sw), (ph, pw))


@pytest.mark.parametrize("args,status", [
    ((2, 8, 10, 10, 16, 3, 3, 0, 1, 1, 1), 2), ((2, 8, 10, 10, 16, 3, 3, 1, 0, 1, 1), 2),
    ((2, 8, 10, 10, 16, 3, 3, 1, 1, -1, 1), 2), ((2, 8, 10, 10, 16, 3, 3, 1, 1, 1, -1), 2),
    ((2, 8, 2, 10, 16, 5, 3, 1, 1, 0, 1), 2),
])
def test_hw_shape_errors(args, status):
    lib = mg3m.load_library()
    assert lib.conv2d_fwd_f32_hw(X, Wp, Y, *args, 0, None, 0, None, None) == status


# ------------------------------------------------ fp64-accumulating entry point
TILES64 = ["128x128", "64x256", "256x64", "64x128", "128x64", "64x64", "32x64", "64x32"]


def _acc64_plan(shape, layout, plan=None):
    N, C, H, W, K, R, S, (sh, sw), (ph, pw) = shape
    text = mg3m.conv2d_fwd_f32_acc64_plan_string(N, C, H, W, K, R, S, sh, sw, ph, pw, layout, plan)
    assert text.startswith("acc=f64,")
    f = dict(kv.split("=", 1) for kv in text.split(","))
    Ho, Wo = mg3m.conv2d_out_dims_hw(H, W, R, S, sh, sw, ph, pw)
    Mg, Ng, Kg = K, N * Ho * Wo, C * R * S
    assert (int(f["Mg"]), int(f["Ng"]), int(f["Kg"])) == (Mg, Ng, Kg)
    mt, nt = (int(v) for v in f["tile"].split("x"))
    tm, tn = (int(v) for v in f["tiles"].split("x"))
    assert (tm - 1) * mt < Mg <= tm * mt and (tn - 1) * nt < Ng <= tn * nt
    # whole tiles and tail tiles partition the tiles; fp64 partials
    kt, split, dp, tail = int(f["k_tiles"]), int(f["split"]), int(f["dp_tiles"]), int(f["tail_tiles"])
    wgs = int(f["tail_wgs"])
    assert f["kt"] == "16" and kt == -(-Kg // 16)
    assert dp + tail == tm * tn
    assert int(f["grid"]) == dp + wgs
    assert (split >= 2 and tail < wgs <= tail * kt) if tail else (split == 1 and wgs == 0)
    copy = -(-4 * Mg * Kg // 256) * 256 if f["b"] == "vec_w_tap" else 0
    assert int(f["ws"]) == 8 * ((wgs + tail - 1) if tail else 0) * mt * nt + copy
    assert f["e"] == "elem"
    assert 0 < int(f["lds"]) <= 160 * 1024
    return f


def test_acc64_plans_for_catalogue_layers_and_overrides():
    for wl, (_, layers) in workloads.WORKLOADS.items():
        for L in layers:
            for layout in ("HWCN", "NCHW"):
                _acc64_plan((L.N, L.C, L.H, L.W, L.K, L.R, L.S, (L.stride,) * 2, (L.pad,) * 2), layout)
    rng = np.random.Generator(np.random.PCG64(4))
    for _ in range(100):
        N = int(rng.integers(1, 33))
        C, K = (int(v) for v in rng.integers(1, 300, 2))
        H, W = (int(v) for v in rng.integers(1, 40, 2))
        R, S = (int(v) for v in rng.choice([1, 2, 3, 5], 2))
        sh, sw = (int(v) for v in rng.integers(1, 4, 2))
        ph, pw = (int(v) for v in rng.integers(0, 3, 2))
        if H + 2 * ph < R or W + 2 * pw < S:
            continue
        shape = (N, C, H, W, K, R, S, (sh, sw), (ph, pw))
        t = str(rng.choice(TILES64))
        sp = int(rng.integers(1, 20))
        for layout in ("HWCN", "NCHW"):
            _acc64_plan(shape, layout)
            assert _acc64_plan(shape, layout, f"tile={t}")["tile"] == t
            f = _acc64_plan(shape, layout, f"tile={t},split={sp}")
            assert int(f["split"]) <= sp and f["tile"] == t
            _acc64_plan(shape, layout, f"tile={t},tail={max(2, sp)}")


def test_acc64_errors():
    lib = mg3m.load_library()
    good = (4, 64, 14, 14, 96, 3, 3, 1, 1, 1, 1, 0)
    for bad in (b"kt=32", b"tile=256x128", b"tile=7x7", b"bogus=1", b"split=0", b"tail=1"):
        assert lib.conv2d_fwd_f32_acc64(X, Wp, Y, *good, bad, None) == 7, bad
    assert lib.conv2d_fwd_f32_acc64(None, Wp, Y, *good, None, None) == 1
    assert lib.conv2d_fwd_f32_acc64(X, Wp, Y + 2, *good, None, None) == 9
    assert lib.conv2d_fwd_f32_acc64(X, Wp, X + 64, *good, None, None) == 5
    assert lib.conv2d_fwd_f32_acc64(X, Wp, Y, 4, 64, 14, 14, 96, 3, 3, 1, 1, 1, 1, 2, None, None) == 3
    assert lib.conv2d_fwd_f32_acc64(X, Wp, Y, 4, 64, 2, 14, 96, 5, 3, 1, 1, 0, 1, 0, None, None) == 2
    assert lib.conv2d_fwd_f32_acc64(X, Wp, Y, 1 << 16, 1 << 10, 64, 64, 16, 3, 3, 1, 1, 1, 1, 0,
                                    None, None) == 4
    assert mg3m.mg3m_last_error() != ""
    # split and tail overrides are accepted (fp64 partials)
    assert "split=2" in mg3m.conv2d_fwd_f32_acc64_plan_string(4, 64, 14, 14, 96, 3, 3, 1, 1, 1, 1,
                                                               "HWCN", "tile=64x64,split=2")


# ------------------------------------------------------------ network executor
def _layers(specs):
    arr = (mg3m.Layer * len(specs))()
    for i, d in enumerate(specs):
        arr[i] = mg3m.Layer(d.get("op", 0), d.get("input", i), d.get("add", -1), d.get("relu", 0),
                            d.get("K", 8), d.get("R", 3), d.get("S", 3), d.get("stride", 1), d.get("pad", 1),
                            d.get("w", Wp))
    return arr


@pytest.mark.parametrize("specs,status", [
    ([], 10),                                                         # no layers
    ([{"input": 1}], 10),                                             # reads a later activation
    ([{"input": -1}], 10),
    ([{"op": 7}], 10),                                                # unknown op
    ([{"w": None}], 1),                                               # conv without a filter
    ([{"relu": 2}], 10),
    ([{"K": 8}, {"K": 16, "add": 1}], 2),                             # residual of another shape
    ([{"K": 8}, {"K": 8, "add": 2}], 10),                             # residual from the future
    ([{"op": 1, "R": 2, "pad": 2}], 2),                               # pool padding over half the window
    ([{"op": 1, "R": 2, "pad": 0, "relu": 1}], 10),                   # pool with an activation
    ([{"R": 9, "pad": 0}], 2),                                        # filter larger than the input
])
def test_net_create_rejects_bad_chains(specs, status):
    import ctypes
    lib = mg3m.load_library()
    h = ctypes.c_void_p()
    arr = _layers(specs) if specs else (mg3m.Layer * 1)()
    rc = lib.mg3m_net_create(arr, len(specs), 2, 4, 6, 6, 0, 0, ctypes.byref(h))
    assert rc == status, mg3m.mg3m_last_error()
    assert not h.value
    assert mg3m.mg3m_last_error() != ""


def test_net_create_argument_errors():
    import ctypes
    lib = mg3m.load_library()
    h = ctypes.c_void_p()
    arr = _layers([{}])
    assert lib.mg3m_net_create(arr, 1, 2, 4, 6, 6, 3, 0, ctypes.byref(h)) == 3       # layout
    assert lib.mg3m_net_create(arr, 1, 0, 4, 6, 6, 0, 0, ctypes.byref(h)) == 2       # N
    assert lib.mg3m_net_create(arr, 1, 2, 4, 6, 6, 0, 2, ctypes.byref(h)) == 10      # keep_all
    assert lib.mg3m_net_create(None, 1, 2, 4, 6, 6, 0, 0, ctypes.byref(h)) == 1
    assert lib.mg3m_net_destroy(None) == 0


def test_network_definitions_shapes_and_flops():
    import workloads.nets as nets
    fl, shapes = nets.conv_flops(nets.vgg16_features(), (64, 3, 224, 224))
    vgg = workloads.workload("vgg16_n64")
    assert fl == pytest.approx(sum(2.0 * L.N * L.K * L.C * L.R * L.S *
                                   oracle.out_dims(L.H, L.W, L.R, L.S, L.stride, L.pad)[0] ** 2 for L in vgg))
    assert shapes[-1] == (64, 512, 7, 7)
    fl, shapes = nets.conv_flops(nets.resnet50_trunk(), (1, 3, 224, 224))
    assert shapes[-1] == (1, 2048, 7, 7)
    assert 8.0e9 < fl < 8.4e9            # ~4.1 GMAC per image in the convolutions
    fl, shapes = nets.conv_flops(nets.alexnet_features(), (1, 3, 224, 224))
    assert shapes[-1] == (1, 256, 6, 6)


def test_maxpool_dims_and_errors():
    assert mg3m.maxpool2d_out_dims(224, 224, 2, 2, 2, 2, 0, 0) == (112, 112)
    assert mg3m.maxpool2d_out_dims(112, 112, 3, 3, 2, 2, 1, 1) == (56, 56)
    assert mg3m.maxpool2d_out_dims(55, 55, 3, 3, 2, 2, 0, 0) == (27, 27)
    lib = mg3m.load_library()
    assert lib.maxpool2d_f32(X, Y, 2, 4, 8, 8, 2, 2, 2, 2, 2, 0, 0, None) == 2        # pad > R/2
    assert lib.maxpool2d_f32(X, Y, 2, 4, 8, 8, 2, 2, 0, 2, 0, 0, 0, None) == 2        # stride 0
    assert lib.maxpool2d_f32(X, X + 8, 2, 4, 8, 8, 2, 2, 2, 2, 0, 0, 0, None) == 5    # y overlaps x
    assert lib.maxpool2d_f32(None, Y, 2, 4, 8, 8, 2, 2, 2, 2, 0, 0, 0, None) == 1
    assert lib.maxpool2d_f32(X, Y, 2, 4, 8, 8, 2, 2, 2, 2, 0, 0, 5, None) == 3


def test_fused_conv_argument_errors():
    lib = mg3m.load_library()
    shape = (2, 8, 10, 10, 16, 3, 3, 1, 1, 1, 1, 0)
    assert lib.conv2d_fwd_f32_fused(X, Wp, Y, None, 2, *shape, None, 0, None, None) == 10   # relu
    assert lib.conv2d_fwd_f32_fused(X, Wp, Y, Y + 8, 1, *shape, None, 0, None, None) == 5   # add overlaps y
    assert lib.conv2d_fwd_f32_fused(X, Wp, Y, Y + 2, 1, *shape, None, 0, None, None) == 9   # misaligned add


def test_injected_launch_failure(monkeypatch):
    """MG3M_TEST_FAIL_LAUNCH=1: validation passes, the launch reports failure."""
    lib = mg3m.load_library()
    monkeypatch.setenv("MG3M_TEST_FAIL_LAUNCH", "1")
    rc = lib.conv2d_fwd_f32_ex(X, Wp, Y, *GOOD, 0, None, 0, b"split=1", None)
    assert rc == 8
    assert "injected" in mg3m.mg3m_last_error()
    monkeypatch.setenv("MG3M_TEST_FAIL_LAUNCH", "0")
    assert lib.conv2d_fwd_f32_ex(X, Wp, Y, 0, *GOOD[1:], 0, None, 0, b"split=1", None) == 2


def test_sixteen_row_tile_selection():
    """The 16x16x4-MFMA tile (16x64) serves layers whose output channels would
    leave a 32-row block at most half full; it takes split plans but no
    stream-K runs; a forced 16x64 plan applies to any shape."""
    k16 = mg3m.conv2d_fwd_f32_plan_info(128, 16, 56, 56, 16, 3, 3, 1, 1, "HWCN")
    assert (k16["mt"], k16["nt"]) == (16, 64)
    for K in (32, 64, 256):
        p = mg3m.conv2d_fwd_f32_plan_info(4, 64, 14, 14, K, 3, 3, 1, 1, "HWCN")
        assert p["mt"] != 16, K
    forced = mg3m.conv2d_fwd_f32_plan_info(4, 64, 14, 14, 256, 3, 3, 1, 1, "HWCN", "tile=16x64,split=3")
    assert (forced["mt"], forced["nt"], forced["split"]) == (16, 64, 3)
    # 13 tail tiles of 36 k-tiles: 40 work-groups would cross tile boundaries
    with pytest.raises(RuntimeError, match="MG3M_ERR_PLAN"):
        mg3m.conv2d_fwd_f32_plan_info(4, 64, 14, 14, 16, 3, 3, 1, 1, "HWCN", "tile=16x64,sk=40")


@pytest.mark.parametrize("bad", ["tile=64x64;kt=32", "tile=64x", "tile=x64", "tile=64x64x", "tile=6 4x64",
                                 "tile=64x64 ", "tile=0x64", "tile=-64x64", "tile=64x99999999999"])
def test_override_tile_halves_must_be_whole_numbers(bad):
    """Both halves of tile=<MT>x<NT> must be whole decimal numbers: a stray
    separator (';' for ',') must not be read as a tile with the default
    depth."""
    with pytest.raises(mg3m.Mg3mError) as ei:
        mg3m.conv2d_fwd_f32_plan_info(32, 512, 7, 7, 2048, 1, 1, 1, 0, "HWCN", bad)
    assert ei.value.status == 7, bad
    # the well-formed spelling of the same request is accepted
    p = mg3m.conv2d_fwd_f32_plan_info(32, 512, 7, 7, 2048, 1, 1, 1, 0, "HWCN", "tile=64x64,kt=32")
    assert (p["mt"], p["nt"], p["kt"]) == (64, 64, 32)


def test_noalloc_validation_before_any_device_call():
    """conv2d_fwd_f32_noalloc validates pointers and shape, and rejects a
    shape whose every plan needs more workspace than its fixed scratch array
    (a tap-major NCHW filter copy of 151 MB against 128 MiB), before it
    looks the array up: these calls need no GPU."""
    lib = mg3m.load_library()
    shape = (1, 1024, 3, 3, 4096, 3, 3, 1, 1)
    assert lib.conv2d_fwd_f32_noalloc(None, Wp, Y, *shape, 1, None) == 1
    assert lib.conv2d_fwd_f32_noalloc(X + 2, Wp, Y, *shape, 1, None) == 9
    assert lib.conv2d_fwd_f32_noalloc(X, Wp, Y, *shape, 5, None) == 3
    assert lib.conv2d_fwd_f32_noalloc(X, Wp, Y, 1, 1, 2, 2, 1, 5, 5, 1, 0, 0, None) == 2
    assert lib.conv2d_fwd_f32_noalloc(X, Wp, Y, *shape, 1, None) == 6
    msg = mg3m.mg3m_last_error()
    assert "134217728" in msg and "150994944" in msg, msg


def test_one_tap_loaders_default_to_direct_lds():
    """Where the one-tap HWCN loaders apply, the selector's plans load straight
    into LDS (b_mode 6), persistent ones included, unless they are on the
    16-row tile; dma=0 keeps the same plan with the loaders staging through
    VGPRs (b_mode 3), and dma=1 is refused where the direct-to-LDS form does
    not apply."""
    shape = (64, 256, 56, 56, 256, 3, 3, 1, 1)
    p = mg3m.conv2d_fwd_f32_plan_info(*shape, "HWCN")
    q = mg3m.conv2d_fwd_f32_plan_info(*shape, "HWCN", "dma=0")
    assert p["b_mode"] == 6 and q["b_mode"] == 3
    same = ("mt", "nt", "kt", "split", "dp_tiles", "tail_tiles", "tail_wgs", "grid", "workspace_bytes")
    assert all(p[k] == q[k] for k in same), (p, q)
    for plan, b_mode in (("tile=128x128,persist=2", 6), ("tile=128x128,persist=2,dma=0", 3)):
        r = mg3m.conv2d_fwd_f32_plan_info(*shape, "HWCN", plan)
        assert r["persistent"] == 1 and r["b_mode"] == b_mode and r["grid"] == 512, (plan, r)
    for bad in ("tile=16x64,dma=1", "tile=16x64,persist=2"):
        with pytest.raises(mg3m.Mg3mError):
            mg3m.conv2d_fwd_f32_plan_info(*shape, "HWCN", bad)
    # the three-channel stem has no one-tap loader
    with pytest.raises(mg3m.Mg3mError):
        mg3m.conv2d_fwd_f32_plan_info(64, 3, 224, 224, 64, 3, 3, 1, 1, "HWCN", "tile=64x256,persist=3,dma=1")
    assert mg3m.conv2d_fwd_f32_plan_info(*shape, "NCHW", "via=none")["b_mode"] == 5
    with pytest.raises(mg3m.Mg3mError):
        mg3m.conv2d_fwd_f32_plan_info(*shape, "NCHW", "dma=1,via=none")
    v = mg3m.conv2d_fwd_f32_plan_info(*shape, "NCHW", "dma=1")
    assert v["via_hwcn"] == 1 and v["b_mode"] == 6


def test_selector_picks_persistent_and_deep_64x64_tiles():
    """The selector's picks where the cost model's persistent and 64x64 kt=32
    terms decide (each measured on MI355X against the previous pick): VGG-16
    conv1 (27-row reduction, 12 rounds of tiles) runs persistent; the
    ResNet-50 1x1 layers run the four-wave 64x64 tile with a 32-deep step;
    its 3x3 layers with 128 or more channels do not (the tile's multi-tap
    factor), nor do VGG-16's deep layers."""
    p = mg3m.conv2d_fwd_f32_plan_info(64, 3, 224, 224, 64, 3, 3, 1, 1, "HWCN")
    assert p["persistent"] == 1 and (p["mt"], p["nt"]) == (64, 256), p
    assert p["grid"] == 256 * 4 and p["dp_tiles"] == 12544, p     # 126 registers: 4 work-groups per CU
    for L in workloads.workload("resnet50_n32"):
        p = mg3m.conv2d_fwd_f32_plan_info(L.N, L.C, L.H, L.W, L.K, L.R, L.S, L.stride, L.pad, "HWCN")
        deep64 = (p["mt"], p["nt"], p["kt"]) == (64, 64, 32)
        if L.R == 1 and L.name not in ("rn50_c5_1x1a_first", "rn50_c5_ds_s2"):
            assert deep64, (L.name, p)
        if L.R == 3 and L.C >= 128:
            assert not deep64, (L.name, p)
    for L in workloads.workload("vgg16_n64")[1:]:
        p = mg3m.conv2d_fwd_f32_plan_info(L.N, L.C, L.H, L.W, L.K, L.R, L.S, L.stride, L.pad, "HWCN")
        assert p["persistent"] == 0 and (p["mt"], p["kt"]) != (64, 32), (L.name, p)


def test_force_plan_environment(monkeypatch):
    """MG3M_FORCE_PLAN stands in for a missing override (plain calls and
    plan queries), an explicit override still wins, and a forced plan that
    does not apply fails with MG3M_ERR_PLAN naming the variable."""
    shape = (8, 64, 28, 28, 128, 3, 3, 1, 1)
    chosen = mg3m.conv2d_fwd_f32_plan_string(*shape, "HWCN")
    assert not chosen.startswith("tile=32x64,"), chosen
    monkeypatch.setenv("MG3M_FORCE_PLAN", "tile=32x64,split=3")
    forced = mg3m.conv2d_fwd_f32_plan_string(*shape, "HWCN")
    assert forced.startswith("tile=32x64,") and ",split=3," in forced, forced
    explicit = mg3m.conv2d_fwd_f32_plan_string(*shape, "HWCN", "tile=128x128")
    assert explicit.startswith("tile=128x128,"), explicit
    monkeypatch.setenv("MG3M_FORCE_PLAN", "tile=48x48")
    with pytest.raises(mg3m.Mg3mError) as e:
        mg3m.conv2d_fwd_f32_plan_string(*shape, "HWCN")
    assert e.value.status == 7 and "MG3M_FORCE_PLAN" in str(e.value)
    monkeypatch.delenv("MG3M_FORCE_PLAN")
    assert mg3m.conv2d_fwd_f32_plan_string(*shape, "HWCN") == chosen


def test_log_prints_each_new_plan_once():
    """MG3M_LOG=1: one stderr line per plan the library makes, none for a
    plan it already holds."""
    import subprocess
    code = ("from paper_2307_04941_amd import mg3m\n"
            "for _ in range(3):\n"
            "    mg3m.conv2d_fwd_f32_plan_string(4, 16, 12, 12, 32, 3, 3, 1, 1, 'HWCN')\n"
            "mg3m.conv2d_fwd_f32_plan_string(4, 16, 12, 12, 32, 3, 3, 1, 1, 'NCHW')\n")
    env = dict(os.environ, MG3M_LOG="1")
    env.pop("MG3M_FORCE_PLAN", None)
    out = subprocess.run([sys.executable, "-c", code], cwd=ROOT, env=env, capture_output=True, text=True,
                         timeout=120)
    assert out.returncode == 0, out.stderr
    lines = [ln for ln in out.stderr.splitlines() if ln.startswith("mg3m plan:")]
    assert len(lines) == 2, out.stderr
    assert "HWCN" in lines[0] and "NCHW" in lines[1] and "tile=" in lines[0], lines
    env["MG3M_LOG"] = "0"
    quiet = subprocess.run([sys.executable, "-c", code], cwd=ROOT, env=env, capture_output=True, text=True,
                           timeout=120)
    assert quiet.returncode == 0 and "mg3m plan:" not in quiet.stderr


@pytest.mark.parametrize("bad", ["waves=2", "waves=2x", "waves=x2", "waves=0x2", "waves=9x1", "waves=2x2x2",
                                 "waves=2 x2"])
def test_override_waves_key(bad):
    """waves=<WM>x<WN> picks among tiles of one shape by their wave grid, so
    the tile part of a plan string (tile, waves, kt) reads back as an
    override naming the same kernel tile; malformed values are rejected."""
    shape = (32, 64, 56, 56, 256, 1, 1, 1, 0)
    p = mg3m.conv2d_fwd_f32_plan_info(*shape, "HWCN", "tile=64x64,waves=2x2,kt=32")
    assert (p["mt"], p["nt"], p["kt"], p["waves_m"], p["waves_n"]) == (64, 64, 32, 2, 2), p
    p = mg3m.conv2d_fwd_f32_plan_info(*shape, "HWCN", "tile=64x64,waves=1x1")
    assert (p["mt"], p["nt"], p["kt"], p["waves_m"], p["waves_n"]) == (64, 64, 16, 1, 1), p
    for layer_shape in [(64, 256, 56, 56, 256, 3, 3, 1, 1), (32, 1024, 14, 14, 256, 1, 1, 1, 0), shape]:
        text = mg3m.conv2d_fwd_f32_plan_string(*layer_shape, "HWCN")
        head = ",".join(f for f in text.split(",") if f.split("=")[0] in ("tile", "waves", "kt"))
        again = mg3m.conv2d_fwd_f32_plan_info(*layer_shape, "HWCN", head)
        first = mg3m.conv2d_fwd_f32_plan_info(*layer_shape, "HWCN")
        assert all(again[k] == first[k] for k in ("mt", "nt", "kt", "waves_m", "waves_n")), (head, again)
    with pytest.raises(mg3m.Mg3mError) as ei:
        mg3m.conv2d_fwd_f32_plan_info(*shape, "HWCN", bad)
    assert ei.value.status == 7, bad
    with pytest.raises(mg3m.Mg3mError):
        mg3m.conv2d_fwd_f32_plan_info(*shape, "HWCN", "tile=64x64,waves=3x1")


def test_selector_runs_strided_nchw_layers_as_hwcn():
    """NCHW layers whose row loader goes element by element (column stride
    above 1) are priced at 0.6 of the tuned rate: ResNet-50's 7x7 stride-2
    stem and its 3x3 stride-2 layers run as HWCN on workspace copies (each
    timed faster that way on MI355X), while VGG-16's stride-1 stem and
    ResNet-50's first 1x1 layers keep the NCHW kernels."""
    rn = {L.name: L for L in workloads.workload("resnet50_n32")}
    vgg = {L.name: L for L in workloads.workload("vgg16_n64")}

    def via(L):
        return mg3m.conv2d_fwd_f32_plan_info(L.N, L.C, L.H, L.W, L.K, L.R, L.S, L.stride, L.pad,
                                             "NCHW")["via_hwcn"]
    for name in ("rn50_stem", "rn50_c3_3x3_s2", "rn50_c4_3x3_s2", "rn50_c5_3x3_s2"):
        assert via(rn[name]) == 1, name
    for name in ("rn50_c2_1x1a_first", "rn50_c3_1x1b"):
        assert via(rn[name]) == 0, name
    assert via(vgg["vgg16_conv1"]) == 0
