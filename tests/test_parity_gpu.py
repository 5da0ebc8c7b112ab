"""GPU parity: the HIP implicit-GEMM convolution (through the C ABI) against
the fp64 oracle, element by element, |gpu - oracle| <= 1e-5 * sum|x*w|
(and bit-exact on small-integer data, where every partial sum is an integer
below 2^24 and fp32 is exact in any order)."""
import numpy as np
import pytest

import oracle
import workloads
from paper_2307_04941_amd import mg3m
from tests.gpu_util import assert_parity, make, run_gpu, say, to_dev

pytestmark = pytest.mark.gpu

TILES = ["128x128", "64x256", "256x64", "64x128", "128x64", "64x64", "32x128", "32x64",
         "128x32", "64x32", "256x128", "128x256", "128x128,kt=32", "16x64", "64x64,kt=32"]


def _small_grid():
    rng = np.random.Generator(np.random.PCG64(20230704))
    cases = []
    while len(cases) < 36:
        N = int(rng.choice([1, 2, 3, 4, 5, 8]))
        C = int(rng.choice([1, 3, 4, 5, 8, 16, 20]))
        K = int(rng.choice([1, 3, 16, 17, 30, 33, 64, 96]))
        H, W = (int(v) for v in rng.integers(1, 15, 2))
        R, S = (int(v) for v in rng.choice([1, 2, 3, 5], 2))
        st = int(rng.integers(1, 4))
        pd = int(rng.integers(0, 4))
        if H + 2 * pd < R or W + 2 * pd < S:
            continue
        cases.append((N, C, H, W, K, R, S, st, pd))
    return cases


SMALL = _small_grid()


@pytest.mark.parametrize("layout", ["HWCN", "NCHW"])
@pytest.mark.parametrize("case", range(len(SMALL)))
def test_small_grid(case, layout):
    shape = SMALL[case]
    say(f"small grid {case} {layout} shape={shape}")
    x, w, st, pd = make(shape, 1000 + case, layout)
    acc, mag = oracle.conv2d(x, w, st, pd, layout)
    y = run_gpu(x, w, st, pd, layout)
    assert_parity(y, acc, mag, f"{shape} {layout}")


# One ragged shape (every GEMM dimension has a tail) forced through every tile
# and several split-K factors, in each loader mode.
FORCED_SHAPES = {
    "vec_n": (4, 20, 13, 11, 70, 3, 3, 1, 1),     # N % 4 == 0: batch-vector gather
    "vec_c": (1, 24, 17, 15, 70, 3, 3, 2, 1),     # N == 1, C % 4 == 0: channel-vector gather
    "scalar": (3, 5, 12, 13, 45, 3, 2, 1, 2),     # element-wise gather
}


@pytest.mark.parametrize("mode", sorted(FORCED_SHAPES))
@pytest.mark.parametrize("tile", TILES)
def test_every_tile_and_split(tile, mode):
    shape = FORCED_SHAPES[mode]
    x, w, st, pd = make(shape, 77, "HWCN")
    acc, mag = oracle.conv2d(x, w, st, pd, "HWCN")
    for split in (1, 2, 5):
        plan = f"tile={tile},split={split}"
        say(f"forced {mode} {plan} shape={shape}")
        y = run_gpu(x, w, st, pd, "HWCN", plan=plan)
        assert_parity(y, acc, mag, f"{shape} {plan}")


# The tuned HWCN loader (one filter tap per staged slab: N % 4 == 0 and C a
# multiple of every tile's kt, 16 and 32): a ragged 3x3 shape and a 1x1 shape
# (every GEMM dimension has a tail), and a shape with more tiles than one
# round of resident work-groups of any tile, so that tail=3 leaves whole
# tiles and split tail tiles in one launch.  Integer data: exact.
TAP_SHAPES = [(4, 64, 13, 11, 68, 3, 3, 1, 1), (4, 64, 9, 7, 68, 1, 1, 1, 0)]
TAP_HYBRID = (32, 32, 95, 95, 64, 3, 3, 1, 1)
_oracle_cache = {}


def _int_case(shape, seed):
    key = (shape, seed)
    if key not in _oracle_cache:
        x, w, st, pd = make(shape, seed, "HWCN", dist="int")
        acc, _ = oracle.conv2d(x, w, st, pd, "HWCN")
        _oracle_cache[key] = (x, w, st, pd, acc.astype(np.float32))
    return _oracle_cache[key]


@pytest.mark.parametrize("dma", [0, 1], ids=["lds_via_vgprs", "direct_to_lds"])
@pytest.mark.parametrize("tile", TILES)
def test_every_tile_vec_n_tap(tile, dma):
    """dma=0: the loaders staging through VGPRs (b_mode 3); dma=1: the same
    loaders in their direct-to-LDS form (b_mode 6, the default where it
    applies; not built for the 16-row tile)."""
    if dma and tile == "16x64":
        with pytest.raises(mg3m.Mg3mError):
            mg3m.conv2d_fwd_f32_plan_info(*TAP_SHAPES[0], "HWCN", f"tile={tile},dma=1")
        return
    suffix = ",dma=1" if dma else ",dma=0"
    for si, shape in enumerate(TAP_SHAPES):
        x, w, st, pd, exact = _int_case(shape, 90 + si)
        for split in (1, 2, 5):
            plan = f"tile={tile},split={split}{suffix}"
            info = mg3m.conv2d_fwd_f32_plan_info(*shape, "HWCN", plan)
            assert info["b_mode"] == (6 if dma else 3), info
            say(f"forced vec_n_tap {plan} shape={shape}")
            y = run_gpu(x, w, st, pd, "HWCN", plan=plan)
            assert np.array_equal(y, exact), f"{shape} {plan}: not bit-exact"
    x, w, st, pd, exact = _int_case(TAP_HYBRID, 95)
    plan = f"tile={tile},tail=3{suffix}"
    info = mg3m.conv2d_fwd_f32_plan_info(*TAP_HYBRID, "HWCN", plan)
    assert info["b_mode"] == (6 if dma else 3) and info["dp_tiles"] > 0 and info["tail_tiles"] > 0, info
    say(f"forced vec_n_tap hybrid {plan}: dp_tiles {info['dp_tiles']} tail_tiles {info['tail_tiles']}")
    y = run_gpu(x, w, st, pd, "HWCN", plan=plan)
    assert np.array_equal(y, exact), f"{TAP_HYBRID} {plan}: not bit-exact"


# Persistent whole tiles (persist=<w>: min(tiles, 256*w) work-groups looping
# over the tiles, the next tile's first stage loaded during the last stage of
# the current one): both batch-vector loaders, a reduction of 27 rows (the
# three-channel 3x3 stems: the last stage skips the k-pairs past Kg), a 1x1
# shape, and a shape with several tiles per work-group.  Integer data: exact.
PERSIST_SHAPES = [((4, 3, 13, 11, 68, 3, 3, 1, 1), 0), ((4, 64, 13, 11, 68, 3, 3, 1, 1), 3),
                  ((4, 64, 9, 7, 68, 1, 1, 1, 0), 3), ((32, 3, 64, 64, 64, 3, 3, 1, 1), 0),
                  (TAP_HYBRID, 3)]


@pytest.mark.parametrize("tile", [t for t in TILES if t != "16x64"])
def test_every_tile_persistent(tile):
    """... and the one-tap shapes again with the loaders that load straight
    into LDS (dma=1, b_mode 6)."""
    for si, (shape, b_mode) in enumerate(PERSIST_SHAPES):
        x, w, st, pd, exact = _int_case(shape, 97 + si)
        for dma in ((0, 1) if b_mode == 3 else (0,)):
            for wgs in (1, 2, 3):
                plan = f"tile={tile},persist={wgs}" + (",dma=1" if dma else ",dma=0")
                info = mg3m.conv2d_fwd_f32_plan_info(*shape, "HWCN", plan)
                assert info["persistent"] == 1 and info["b_mode"] == (6 if dma else b_mode), info
                assert info["grid"] == min(info["dp_tiles"], 256 * wgs) and info["tail_tiles"] == 0, info
                say(f"persistent {plan} shape={shape}: grid {info['grid']} tiles {info['dp_tiles']}")
                y = run_gpu(x, w, st, pd, "HWCN", plan=plan)
                assert np.array_equal(y, exact), f"{shape} {plan}: not bit-exact"


@pytest.mark.parametrize("tile", TILES)
def test_every_tile_nchw_tap_major(tile):
    """NCHW with C a multiple of kt: the filter is copied to [R][S][C][K] in
    the workspace and every stage is one tap over a channel slab; the
    partials of split plans sit after the copy.  Integer data: exact."""
    shape = (3, 32, 10, 9, 40, 3, 3, 1, 1)
    x, w, st, pd = make(shape, 81, "NCHW", dist="int")
    acc, _ = oracle.conv2d(x, w, st, pd, "NCHW")
    for split in (1, 3):
        plan = f"tile={tile},split={split},via=none"
        info = mg3m.conv2d_fwd_f32_plan_info(*shape, "NCHW", plan)
        assert info["b_mode"] == 5, info
        say(f"forced NCHW tap-major {plan}: workspace {info['workspace_bytes']}")
        y = run_gpu(x, w, st, pd, "NCHW", plan=plan)
        assert np.array_equal(y, acc.astype(np.float32)), plan


@pytest.mark.parametrize("tile", TILES)
def test_every_tile_nchw(tile):
    shape = (2, 6, 11, 9, 37, 3, 3, 1, 1)
    x, w, st, pd = make(shape, 78, "NCHW")
    acc, mag = oracle.conv2d(x, w, st, pd, "NCHW")
    for split in (1, 3):
        plan = f"tile={tile},split={split},via=none"
        say(f"forced NCHW {plan}")
        y = run_gpu(x, w, st, pd, "NCHW", plan=plan)
        assert_parity(y, acc, mag, f"{shape} {plan}")


# Enough output tiles for more than one round of resident work-groups, so that
# tail=n splits only the leftover tiles (e.g. 256x64 tiles: 3081 tiles against
# 768 resident work-groups -> 3072 whole, 9 split).
TAIL_SHAPE = (24, 16, 111, 111, 32, 3, 3, 1, 1)


# NCHW patch loader (16-byte runs along W, else per column): output widths
# that do and do not divide by 4 (groups of four columns wrap to the next
# output row or image), strides 1-3 along W, padding on either side, ragged
# Ng, single-pixel outputs.  Integer data, so every output must be exact.
NCHW_EDGES = [
    (2, 3, 7, 9, 5, 3, 3, 1, 1),             # Wo 9: runs cross rows
    (3, 4, 6, 4, 8, 3, 3, 1, (0, 1)),        # Wo 4, padding on both sides
    (1, 8, 5, 18, 16, 1, 3, (1, 1), (0, 2)), # wide rows, pad 2 along W only
    (5, 2, 9, 13, 7, 3, 5, 1, 2),            # Wo 13, N*Ho*Wo odd
    (2, 16, 8, 11, 32, 3, 3, (1, 2), 1),     # stride 2 along W: element path
    (4, 5, 10, 10, 9, 2, 2, (2, 3), (1, 0)), # stride 3 along W
    (3, 6, 3, 3, 12, 3, 3, 1, 0),            # Wo 1
    (2, 7, 4, 5, 6, 3, 2, 1, (1, 0)),        # Wo 4, every group one row
    (1, 32, 14, 14, 64, 3, 3, 1, 1),         # Wo 14 (VGG conv5 blocks)
    (2, 16, 28, 28, 24, 1, 1, 1, 0),         # 1x1, one contiguous plane per channel
]


@pytest.mark.parametrize("case", range(len(NCHW_EDGES)))
def test_nchw_row_vector_loader(case):
    shape = NCHW_EDGES[case]
    say(f"NCHW loader edge {case} shape={shape}")
    x, w, st, pd = make(shape, 700 + case, "NCHW", dist="int")
    acc, _ = oracle.conv2d(x, w, st, pd, "NCHW")
    for plan in (None, "tile=32x64,split=1,via=none", "tile=128x128,split=2,via=none"):
        y = run_gpu(x, w, st, pd, "NCHW", plan=plan)
        assert np.array_equal(y, acc.astype(np.float32)), f"{shape} {plan}"


@pytest.mark.parametrize("layout", ["HWCN", "NCHW"])
@pytest.mark.parametrize("plan", ["tile=256x64,tail=2", "tile=256x64,tail=3", "tile=256x64,tail=5",
                                  "tile=64x256,tail=4", "tile=128x128,kt=32,tail=2"])
def test_tail_split(plan, layout):
    x, w, st, pd = make(TAIL_SHAPE, 85, layout)
    info = mg3m.conv2d_fwd_f32_plan_info(*TAIL_SHAPE, layout, plan)
    say(f"tail split {plan} {layout}: dp_tiles {info['dp_tiles']} tail_tiles {info['tail_tiles']} "
        f"split {info['split']}")
    assert info["dp_tiles"] > 0 and info["tail_tiles"] > 0
    acc, mag = oracle.conv2d(x, w, st, pd, layout)
    y = run_gpu(x, w, st, pd, layout, plan=plan)
    assert_parity(y, acc, mag, f"{TAIL_SHAPE} {plan} {layout}")


def test_tail_split_bit_exact():
    x, w, st, pd = make(TAIL_SHAPE, 86, "HWCN", dist="int")
    acc, _ = oracle.conv2d(x, w, st, pd, "HWCN")
    for plan in ("tile=256x64,tail=3", "tile=256x64,split=4"):
        y = run_gpu(x, w, st, pd, "HWCN", plan=plan)
        assert np.array_equal(y.astype(np.float64), acc), f"{plan}: not bit-exact"


def _rect_grid():
    rng = np.random.Generator(np.random.PCG64(20230705))
    cases = []
    while len(cases) < 16:
        N = int(rng.choice([1, 2, 4, 8]))
        C = int(rng.choice([3, 4, 16, 32]))
        K = int(rng.choice([8, 17, 64]))
        H, W = (int(v) for v in rng.integers(3, 20, 2))
        R, S = (int(v) for v in rng.choice([1, 2, 3, 5], 2))
        sh, sw = (int(v) for v in rng.integers(1, 4, 2))
        ph, pw = (int(v) for v in rng.integers(0, 3, 2))
        if (sh, ph) == (sw, pw) or H + 2 * ph < R or W + 2 * pw < S:
            continue
        cases.append((N, C, H, W, K, R, S, (sh, sw), (ph, pw)))
    return cases


RECT = _rect_grid()


@pytest.mark.parametrize("layout", ["HWCN", "NCHW"])
@pytest.mark.parametrize("case", range(len(RECT)))
def test_rectangular_stride_pad(case, layout):
    """conv2d_fwd_f32_hw: separate vertical / horizontal stride and padding."""
    shape = RECT[case]
    say(f"rectangular {case} {layout} shape={shape}")
    x, w, st, pd = make(shape, 2000 + case, layout)
    acc, mag = oracle.conv2d(x, w, st, pd, layout)
    for plan in (None, "split=3"):
        y = run_gpu(x, w, st, pd, layout, plan=plan)
        assert_parity(y, acc, mag, f"{shape} {layout} {plan}")


@pytest.mark.parametrize("layout", ["HWCN", "NCHW"])
def test_misaligned_pointers(layout):
    """4-byte but not 16-byte aligned buffers take the element-wise paths."""
    shape = (4, 8, 9, 9, 32, 3, 3, 1, 1)
    x, w, st, pd = make(shape, 79, layout)
    acc, mag = oracle.conv2d(x, w, st, pd, layout)
    y = run_gpu(x, w, st, pd, layout, misalign=1)
    assert_parity(y, acc, mag, "misaligned")


@pytest.mark.parametrize("shape", [
    (1, 16, 32, 32, 16, 3, 3, 1, 1),        # the single-layer case
    (2, 32, 14, 14, 64, 3, 3, 1, 1),
    (1, 64, 9, 9, 128, 3, 3, 2, 1),
    (4, 12, 8, 8, 24, 5, 5, 1, 2),
])
@pytest.mark.parametrize("layout", ["HWCN", "NCHW"])
def test_small_integer_bit_exact(shape, layout):
    x, w, st, pd = make(shape, 80, layout, dist="int")
    acc, _ = oracle.conv2d(x, w, st, pd, layout)
    for plan in (None, "split=3"):
        y = run_gpu(x, w, st, pd, layout, plan=plan)
        assert np.array_equal(y.astype(np.float64), acc), f"{shape} {layout} {plan}: not bit-exact"


@pytest.mark.parametrize("shape", [
    (1, 1, 1, 1, 1, 1, 1, 1, 0),            # everything 1
    (1, 2, 3, 3, 2, 2, 2, 1, 3),            # pad >= R: all-zero border outputs
    (2, 3, 7, 7, 5, 2, 2, 4, 0),            # stride > R: skipped input pixels
    (1, 3, 1, 17, 4, 1, 5, 1, 2),           # one input row
    (3, 1, 6, 6, 1, 3, 3, 1, 1),            # C == K == 1
    (1, 4, 5, 5, 200, 1, 1, 1, 0),          # Mg spans several tiles, Ng tiny
])
def test_degenerate_shapes(shape):
    for layout in ("HWCN", "NCHW"):
        x, w, st, pd = make(shape, 81, layout)
        acc, mag = oracle.conv2d(x, w, st, pd, layout)
        y = run_gpu(x, w, st, pd, layout)
        assert_parity(y, acc, mag, f"{shape} {layout}")


def test_guard_bands_and_determinism():
    """Nothing outside y is written; split-K results repeat bit for bit."""
    import torch
    shape = (4, 64, 14, 14, 96, 3, 3, 1, 1)
    x, w, st, pd = make(shape, 82, "HWCN")
    xd, wd = torch.from_numpy(x).cuda(), torch.from_numpy(w).cuda()
    Ho, Wo = mg3m.conv2d_out_dims(14, 14, 3, 3, 1, 1)
    n = Ho * Wo * 96 * 4
    pad = 4096
    outs = []
    for _ in range(2):
        buf = torch.full((n + 2 * pad,), float("nan"), device="cuda")
        y = buf[pad:pad + n].view(Ho, Wo, 96, 4)
        mg3m.conv2d_fwd(xd, wd, st, pd, "HWCN", plan="split=4", out=y)
        torch.cuda.synchronize()
        b = buf.cpu().numpy()
        assert np.isnan(b[:pad]).all() and np.isnan(b[pad + n:]).all(), "write outside y"
        outs.append(b[pad:pad + n].copy())
    assert np.array_equal(outs[0], outs[1])
    acc, mag = oracle.conv2d(x, w, st, pd, "HWCN")
    assert_parity(outs[0].reshape(Ho, Wo, 96, 4), acc, mag, "guard")


@pytest.mark.parametrize("layout,plan", [("HWCN", "split=4"), ("NCHW", "tile=128x128,split=3,via=none"),
                                         ("NCHW", "tile=128x128,split=3,via=hwcn")])
def test_workspace_guard_bands(layout, plan):
    """A caller workspace is written only inside the bytes the plan asks for
    (NCHW: the filter copy, then the partials; run as HWCN: the copies of x,
    w and y, then the partials)."""
    import torch
    shape = (4, 32, 14, 14, 96, 3, 3, 1, 1)
    x, w, st, pd = make(shape, 83, layout)
    N, C, H, W, K, R, S = mg3m.dims_of(x, w, layout)
    need = mg3m.conv2d_fwd_f32_workspace_bytes(N, C, H, W, K, R, S, 1, 1, layout, plan)
    assert need > 0
    pad = 1024
    buf = torch.full((need // 4 + 2 * pad,), float("nan"), device="cuda")
    ws = buf[pad:pad + need // 4]
    Ho, Wo = mg3m.conv2d_out_dims(H, W, R, S, 1, 1)
    y = torch.empty((Ho, Wo, K, N) if layout == "HWCN" else (N, K, Ho, Wo), device="cuda")
    mg3m.conv2d_fwd_f32_ex(to_dev(x), to_dev(w), y, N, C, H, W, K, R, S, 1, 1, layout, ws, need, plan)
    torch.cuda.synchronize()
    b = buf.cpu().numpy()
    assert np.isnan(b[:pad]).all() and np.isnan(b[pad + need // 4:]).all(), "write outside the workspace"
    acc, mag = oracle.conv2d(x, w, st, pd, layout)
    assert_parity(y.cpu().numpy(), acc, mag, f"{layout} {plan}")


def test_injected_launch_failure_leaves_y_untouched(monkeypatch):
    import torch
    shape = (4, 16, 12, 12, 32, 3, 3, 1, 1)
    x, w, st, pd = make(shape, 84, "HWCN")
    y = torch.full((12, 12, 32, 4), float("nan"), device="cuda")
    monkeypatch.setenv("MG3M_TEST_FAIL_LAUNCH", "1")
    for plan in (None, "split=3"):
        with pytest.raises(mg3m.Mg3mError) as ei:
            mg3m.conv2d_fwd(to_dev(x), to_dev(w), st, pd, "HWCN", plan=plan, out=y)
        assert ei.value.status == 8
    torch.cuda.synchronize()
    assert torch.isnan(y).all().item()
    monkeypatch.delenv("MG3M_TEST_FAIL_LAUNCH")
    mg3m.conv2d_fwd(to_dev(x), to_dev(w), st, pd, "HWCN", out=y)        # the stream still works
    acc, mag = oracle.conv2d(x, w, st, pd, "HWCN")
    assert_parity(y.cpu().numpy(), acc, mag, "after injected failure")


def test_vgg_conv9_performance_floor():
    """The hot path keeps at least 60% of the fp32 MFMA peak (94.4 TFLOPS) on
    VGG-16 conv9 (N=64, 512 channels, 28x28), the configuration the
    benchmark's dominant kernel serves."""
    import time
    import torch
    L = workloads.workload("vgg16_n64")[8]
    layer, x, w = workloads.layer_tensors("vgg16_n64", 8, "HWCN")
    xd, wd = torch.from_numpy(x).cuda(), torch.from_numpy(w).cuda()
    y = mg3m.conv2d_fwd(xd, wd, L.stride, L.pad, "HWCN")
    t_end = time.perf_counter() + 0.2
    while time.perf_counter() < t_end:
        mg3m.conv2d_fwd(xd, wd, L.stride, L.pad, "HWCN", out=y)
        torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(10):
        mg3m.conv2d_fwd(xd, wd, L.stride, L.pad, "HWCN", out=y)
    e1.record()
    torch.cuda.synchronize()
    us = e0.elapsed_time(e1) * 1e3 / 10
    Ho, Wo = mg3m.conv2d_out_dims(L.H, L.W, L.R, L.S, L.stride, L.pad)
    tflops = 2.0 * L.N * L.K * L.C * L.R * L.S * Ho * Wo / us / 1e6
    say(f"VGG conv9: {us:.1f} us, {tflops:.1f} TFLOPS")
    assert tflops >= 0.6 * 157.3


def test_non_default_stream():
    import torch
    shape = (8, 32, 16, 16, 64, 3, 3, 1, 1)
    x, w, st, pd = make(shape, 83, "HWCN")
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        xd, wd = torch.from_numpy(x).cuda(), torch.from_numpy(w).cuda()
        y = mg3m.conv2d_fwd(xd, wd, st, pd, "HWCN")
        host = torch.empty(y.shape, dtype=torch.float32, pin_memory=True)
        host.copy_(y, non_blocking=True)
    s.synchronize()
    acc, mag = oracle.conv2d(x, w, st, pd, "HWCN")
    assert_parity(host.numpy(), acc, mag, "stream")


def test_caller_workspace_too_small_is_rejected():
    import torch
    shape = (4, 64, 14, 14, 96, 3, 3, 1, 1)
    x, w, st, pd = make(shape, 84, "HWCN")
    xd, wd = torch.from_numpy(x).cuda(), torch.from_numpy(w).cuda()
    y = torch.full((14, 14, 96, 4), 7.0, device="cuda")
    need = mg3m.conv2d_fwd_f32_workspace_bytes(4, 64, 14, 14, 96, 3, 3, 1, 1, "HWCN", "split=4")
    ws = torch.empty(need // 4 - 1, device="cuda")
    with pytest.raises(mg3m.Mg3mError) as e:
        mg3m.conv2d_fwd_f32_ex(xd, wd, y, 4, 64, 14, 14, 96, 3, 3, 1, 1, "HWCN",
                               ws, ws.numel() * 4, "split=4")
    assert e.value.status == 6
    torch.cuda.synchronize()
    assert (y == 7.0).all().item(), "a rejected call wrote to y"
