"""GPU parity of the fp64-accumulating entry point (conv2d_fwd_f32_acc64)
against the fp64 oracle.

The kernel widens the fp32 operands to fp64, so every product is exact,
accumulates in fp64 and rounds once to fp32 at the store -- the numerics of
the paper's kernel, which converts its staged fp32 tiles to double
(Sec. 4.1.1, Alg. 2).  Each output is therefore within one fp32 rounding of
the exact sum, plus the fp64 summation error of both sides:

    |gpu - acc| <= 2^-24 |acc| + 4 Kg 2^-53 sum|x*w|

With integer data whose partial sums stay below 2^53 every fp64 sum is exact,
so each output must equal the oracle's exact sum rounded to nearest-even fp32,
bit for bit -- also where the sums pass 2^24, which an fp32 accumulator cannot
represent exactly.
"""
import numpy as np
import pytest

import oracle
import workloads
from paper_2307_04941_amd import mg3m
from tests.gpu_util import assert_parity, assert_parity_acc64, make, run_gpu, say

pytestmark = pytest.mark.gpu

TILES64 = ["128x128", "64x256", "256x64", "64x128", "128x64", "64x64,waves=1x1", "32x64", "64x32",
           "64x64,waves=2x2"]

# Shapes spanning several tiles with ragged tails in both output dimensions.
TILE_SHAPES = [
    (4, 32, 13, 13, 72, 3, 3, 1, 1),     # Mg 72, Ng 676, Kg 288
    (4, 16, 9, 9, 300, 3, 3, 1, 1),      # Mg 300 (two 256-row tiles), Ng 324, Kg 144
]

# One shape per loader pair, with the (a, b) modes the selector must pick.
VARIANTS = [
    ((4, 32, 13, 13, 72, 3, 3, 1, 1), "HWCN", "vec_m", "vec_n_tap"),
    ((4, 20, 11, 11, 36, 3, 3, 2, 1), "HWCN", "vec_m", "vec_n"),
    ((1, 12, 15, 15, 24, 3, 3, 1, 1), "HWCN", "vec_m", "vec_c"),
    ((3, 8, 10, 10, 16, 3, 3, 1, 1), "HWCN", "vec_m", "scalar"),
    ((3, 5, 9, 9, 7, 3, 3, 1, 1), "HWCN", "scalar", "scalar"),
    ((2, 4, 9, 9, 16, 3, 3, 1, 1), "NCHW", "vec_k", "vec_w"),
    ((3, 5, 9, 9, 7, 3, 3, 1, 1), "NCHW", "scalar", "vec_w"),
    ((2, 32, 9, 9, 16, 3, 3, 1, 1), "NCHW", "vec_m", "vec_w_tap"),
]


def _plan_fields(shape, layout, plan=None):
    N, C, H, W, K, R, S, st, pd = shape
    (sh, sw), (ph, pw) = mg3m._pair(st), mg3m._pair(pd)
    text = mg3m.conv2d_fwd_f32_acc64_plan_string(N, C, H, W, K, R, S, sh, sw, ph, pw, layout, plan)
    return dict(kv.split("=", 1) for kv in text.split(","))


def _kg(shape):
    N, C, H, W, K, R, S, st, pd = shape
    return C * R * S


def _exact_f32(acc):
    """The exact sum (integer data: acc is exact in fp64) rounded to nearest-even fp32."""
    return np.asarray(acc, np.float64).astype(np.float32)


@pytest.mark.parametrize("layout", ["HWCN", "NCHW"])
@pytest.mark.parametrize("shape", TILE_SHAPES, ids=["ng_ragged", "mg_ragged"])
@pytest.mark.parametrize("tile", TILES64)
def test_every_tile_bit_exact_on_wide_integers(tile, shape, layout):
    say(f"acc64 tile={tile} {layout} shape={shape}")
    x, w, st, pd = make(shape, 300, layout, dist="wideint")
    acc, _ = oracle.conv2d(x, w, st, pd, layout)
    y = run_gpu(x, w, st, pd, layout, plan=f"tile={tile}", acc64=True)
    want = _exact_f32(acc)
    diff = np.flatnonzero(y.reshape(-1).view(np.uint32) != want.reshape(-1).view(np.uint32))
    assert diff.size == 0, (f"{diff.size} outputs differ from the exact sum rounded to fp32; first "
                            f"{diff[0]}: gpu {y.reshape(-1)[diff[0]]!r} want {want.reshape(-1)[diff[0]]!r}")


@pytest.mark.parametrize("case", range(len(VARIANTS)))
def test_every_loader_pair(case):
    shape, layout, am, bm = VARIANTS[case]
    f = _plan_fields(shape, layout)
    assert (f["a"], f["b"]) == (am, bm), f
    assert f["acc"] == "f64"
    say(f"acc64 loaders a={am} b={bm} {layout} shape={shape} tile={f['tile']}")
    x, w, st, pd = make(shape, 310 + case, layout, dist="wideint")
    acc, _ = oracle.conv2d(x, w, st, pd, layout)
    y = run_gpu(x, w, st, pd, layout, acc64=True)
    assert np.array_equal(y.view(np.uint32), _exact_f32(acc).view(np.uint32))
    x, w, st, pd = make(shape, 320 + case, layout)
    acc, mag = oracle.conv2d(x, w, st, pd, layout)
    y = run_gpu(x, w, st, pd, layout, acc64=True)
    worst = assert_parity_acc64(y, acc, mag, _kg(shape), f"{shape} {layout}")
    say(f"  worst ratio to the one-rounding bound {worst:.3g}")


@pytest.mark.parametrize("layout", ["HWCN", "NCHW"])
@pytest.mark.parametrize("tile", TILES64)
def test_every_tile_random_data(tile, layout):
    shape = TILE_SHAPES[0]
    say(f"acc64 random tile={tile} {layout}")
    x, w, st, pd = make(shape, 330, layout)
    acc, mag = oracle.conv2d(x, w, st, pd, layout)
    y = run_gpu(x, w, st, pd, layout, plan=f"tile={tile}", acc64=True)
    assert_parity_acc64(y, acc, mag, _kg(shape), f"tile {tile} {layout}")


# Shape with more tiles than one round of resident work-groups for every
# tested plan, so tail=n leaves whole tiles and split tiles.
SPLIT_SHAPE = (24, 16, 61, 61, 96, 3, 3, 1, 1)
SPLIT_PLANS = ["tile=128x128,split=3", "tile=32x64,split=5", "tile=64x256,tail=4", "tile=256x64,tail=2",
               "tile=64x32,tail=6", "tile=64x64,waves=2x2,split=4", "tile=64x64,waves=2x2,tail=8"]


@pytest.mark.parametrize("layout", ["HWCN", "NCHW"])
@pytest.mark.parametrize("plan", SPLIT_PLANS)
def test_split_reduction_keeps_fp64(plan, layout):
    """Split tiles add fp64 partials in fp64 and round once: still bit-exact
    on wide integers, still within one rounding on random data."""
    f = _plan_fields(SPLIT_SHAPE, layout, plan)
    say(f"acc64 split {plan} {layout}: dp_tiles {f['dp_tiles']} tail_tiles {f['tail_tiles']} "
        f"split {f['split']} ws {f['ws']}")
    assert int(f["tail_tiles"]) > 0 and int(f["split"]) >= 2
    if "tail=" in plan:
        assert int(f["dp_tiles"]) > 0
    x, w, st, pd = make(SPLIT_SHAPE, 390, layout, dist="wideint")
    acc, _ = oracle.conv2d(x, w, st, pd, layout)
    y = run_gpu(x, w, st, pd, layout, plan=plan, acc64=True)
    assert np.array_equal(y.view(np.uint32), _exact_f32(acc).view(np.uint32))
    x, w, st, pd = make(SPLIT_SHAPE, 391, layout)
    acc, mag = oracle.conv2d(x, w, st, pd, layout)
    y = run_gpu(x, w, st, pd, layout, plan=plan, acc64=True)
    assert_parity_acc64(y, acc, mag, _kg(SPLIT_SHAPE), f"{plan} {layout}")


def _rect_cases():
    rng = np.random.Generator(np.random.PCG64(20230706))
    cases = []
    while len(cases) < 8:
        N = int(rng.choice([1, 2, 4]))
        C = int(rng.choice([3, 16, 32]))
        K = int(rng.choice([8, 17, 64]))
        H, W = (int(v) for v in rng.integers(3, 20, 2))
        R, S = (int(v) for v in rng.choice([1, 2, 3, 5], 2))
        sh, sw = (int(v) for v in rng.integers(1, 4, 2))
        ph, pw = (int(v) for v in rng.integers(0, 3, 2))
        if (sh, ph) == (sw, pw) or H + 2 * ph < R or W + 2 * pw < S:
            continue
        cases.append((N, C, H, W, K, R, S, (sh, sw), (ph, pw)))
    return cases


RECT = _rect_cases()


@pytest.mark.parametrize("layout", ["HWCN", "NCHW"])
@pytest.mark.parametrize("case", range(len(RECT)))
def test_rectangular_stride_pad(case, layout):
    shape = RECT[case]
    say(f"acc64 rectangular {case} {layout} shape={shape}")
    x, w, st, pd = make(shape, 340 + case, layout)
    acc, mag = oracle.conv2d(x, w, st, pd, layout)
    y = run_gpu(x, w, st, pd, layout, acc64=True)
    assert_parity_acc64(y, acc, mag, _kg(shape), f"{shape} {layout}")


@pytest.mark.parametrize("shape", [
    (2, 4, 3, 3, 8, 2, 2, 1, 3),          # pad > filter: border outputs see only padding
    (5, 7, 1, 1, 9, 1, 1, 1, 0),          # 1x1 image, 1x1 filter
    (1, 1, 6, 6, 1, 3, 3, 4, 0),          # stride past the filter, one channel in and out
])
@pytest.mark.parametrize("layout", ["HWCN", "NCHW"])
def test_degenerate_shapes(shape, layout):
    say(f"acc64 degenerate {layout} shape={shape}")
    x, w, st, pd = make(shape, 350, layout)
    acc, mag = oracle.conv2d(x, w, st, pd, layout)
    y = run_gpu(x, w, st, pd, layout, acc64=True)
    assert_parity_acc64(y, acc, mag, _kg(shape), f"{shape} {layout}")
    assert np.all(y[mag == 0] == 0)


@pytest.mark.parametrize("layout", ["HWCN", "NCHW"])
def test_misaligned_pointers(layout):
    shape = (4, 8, 9, 9, 32, 3, 3, 1, 1)
    x, w, st, pd = make(shape, 360, layout)
    acc, mag = oracle.conv2d(x, w, st, pd, layout)
    y = run_gpu(x, w, st, pd, layout, misalign=1, acc64=True)
    assert_parity_acc64(y, acc, mag, _kg(shape), "misaligned")


def test_deterministic():
    shape = TILE_SHAPES[0]
    x, w, st, pd = make(shape, 370, "HWCN")
    a = run_gpu(x, w, st, pd, "HWCN", acc64=True)
    b = run_gpu(x, w, st, pd, "HWCN", acc64=True)
    assert np.array_equal(a.view(np.uint32), b.view(np.uint32))


def test_fp32_path_rounds_where_fp64_accumulation_is_exact():
    """On wide integers with Kg = 576 the partial sums pass 2^24: the fp32
    entry point stays inside its 1e-5 bound but misses the correctly rounded
    result somewhere, while the fp64-accumulating one hits it everywhere."""
    shape = (4, 64, 9, 9, 64, 3, 3, 1, 1)
    x, w, st, pd = make(shape, 380, "HWCN", dist="wideint")
    acc, mag = oracle.conv2d(x, w, st, pd, "HWCN")
    want = _exact_f32(acc)
    y64 = run_gpu(x, w, st, pd, "HWCN", acc64=True)
    y32 = run_gpu(x, w, st, pd, "HWCN")
    assert np.array_equal(y64.view(np.uint32), want.view(np.uint32))
    assert_parity(y32, acc, mag, "fp32 path")
    assert np.count_nonzero(y32 != want) > 0


def _pick_layers():
    out = []
    vgg = workloads.workload("vgg16_n64")
    out.append(("vgg16_n64", 1))                                     # 64 -> 64 at 224x224
    out.append(("vgg16_n64", len(vgg) - 1))                          # 512 -> 512 at 14x14
    rn = workloads.workload("resnet50_n32")
    out.append(("resnet50_n32", next(i for i, L in enumerate(rn) if L.C == 512 and L.R == 3)))
    out.append(("alexnet_inception_n128", 0))                        # 11x11, stride 4
    return out


@pytest.mark.parametrize("wl,index", _pick_layers())
def test_full_size_layers_sampled(wl, index):
    import torch
    layer, x, w = workloads.layer_tensors(wl, index, "HWCN")
    shape = (layer.N, layer.C, layer.H, layer.W, layer.K, layer.R, layer.S, layer.stride, layer.pad)
    say(f"acc64 layer {wl}/{layer.name} {shape}: " + ",".join(
        f"{k}={v}" for k, v in _plan_fields(shape, "HWCN").items() if k in ("tile", "grid")))
    xd, wd = torch.from_numpy(x).cuda(), torch.from_numpy(w).cuda()
    y = mg3m.conv2d_fwd(xd, wd, layer.stride, layer.pad, "HWCN", acc64=True)
    torch.cuda.synchronize()
    rng = np.random.Generator(np.random.PCG64(5151 + index))
    per_pix = y.shape[2] * y.shape[3]
    last = y.numel() - per_pix
    idx = np.concatenate([rng.integers(0, per_pix, 2048), last + rng.integers(0, per_pix, 2048),
                          rng.integers(0, y.numel(), 8192)]).astype(np.int64)
    got = y.view(-1)[torch.from_numpy(idx).cuda()].cpu().numpy()
    acc, mag = oracle.conv2d_points(x, w, idx, layer.stride, layer.pad, "HWCN")
    worst = assert_parity_acc64(got, acc, mag, layer.C * layer.R * layer.S, f"{wl}/{layer.name}")
    say(f"  sampled {idx.size} outputs, worst ratio {worst:.3g}")
    del xd, wd, y
    torch.cuda.empty_cache()
