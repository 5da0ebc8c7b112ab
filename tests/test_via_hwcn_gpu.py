"""NCHW calls run as HWCN (plan key via=hwcn; the selector weighs it against
the NCHW kernels): x and the filter are copied to HWCN and [R][S][C][K] in
the workspace, the HWCN kernels write an HWCN copy of y there, and a last
kernel writes y in NCHW, applying any fused output stage.  Small-integer data,
so every output must equal the oracle's exact sum bit for bit (Eq. 1)."""
import numpy as np
import pytest

import oracle
from paper_2307_04941_amd import mg3m
from tests.gpu_util import RTOL, make, run_gpu, say, to_dev

pytestmark = pytest.mark.gpu

TILES = ["128x128", "64x256", "256x64", "64x128", "128x64", "64x64", "32x128", "32x64", "128x32", "64x32",
         "256x128", "128x256", "128x128,kt=32", "16x64", "64x64,kt=32"]

SHAPES = [
    (3, 32, 10, 9, 40, 3, 3, 1, 1),          # one-tap HWCN loaders (into LDS)
    (4, 3, 17, 15, 20, 3, 3, 2, 1),          # three channels: batch-vector loader
    (1, 8, 9, 7, 12, 3, 3, 1, 1),            # N = 1: channel-vector loader
    (2, 5, 7, 6, 9, 2, 3, 1, (1, 0)),        # odd sizes: element-wise loaders
]


def _exact(shape, seed):
    x, w, st, pd = make(shape, seed, "NCHW", dist="int")
    acc, _ = oracle.conv2d(x, w, st, pd, "NCHW")
    return x, w, st, pd, acc.astype(np.float32)


@pytest.mark.parametrize("tile", TILES)
def test_every_tile_via_hwcn(tile):
    for si, shape in enumerate(SHAPES):
        x, w, st, pd, exact = _exact(shape, 880 + si)
        for split in (1, 3):
            plan = f"tile={tile},split={split},via=hwcn"
            st_hw = st if isinstance(st, tuple) else (st, st)
            pd_hw = pd if isinstance(pd, tuple) else (pd, pd)
            N, C, H, W, K, R, S = shape[:7]
            try:
                info = mg3m.conv2d_fwd_f32_plan_info(N, C, H, W, K, R, S, st_hw[0], pd_hw[0], "NCHW", plan) \
                    if st_hw[0] == st_hw[1] and pd_hw[0] == pd_hw[1] else None
            except mg3m.Mg3mError:
                continue                      # the tile does not apply (16x64 needs K mod 32 <= 16)
            if info is not None:
                assert info["via_hwcn"] == 1 and info["layout"] == 0, info
            say(f"via hwcn {shape} {plan}")
            y = run_gpu(x, w, st, pd, "NCHW", plan=plan)
            assert np.array_equal(y, exact), f"{shape} {plan}"


def test_via_hwcn_misaligned_pointers_and_stream_k():
    """Misaligned (4-byte) NCHW buffers: the copies in the workspace are
    aligned, so the HWCN kernels keep their vector loaders; stream-K runs."""
    shape = (4, 64, 13, 11, 68, 3, 3, 1, 1)
    x, w, st, pd, exact = _exact(shape, 890)
    for plan in ("via=hwcn", "tile=128x128,sk=7,via=hwcn", "tile=64x256,persist=1,via=hwcn"):
        y = run_gpu(x, w, st, pd, "NCHW", plan=plan, misalign=1)
        assert np.array_equal(y, exact), plan


@pytest.mark.parametrize("plan", ["tile=64x64,kt=32,via=hwcn", "tile=128x128,split=3,via=hwcn"])
def test_via_hwcn_fused_add_relu(plan):
    """y = relu(conv + add) applied while y is written back to NCHW, also in
    place (add is y)."""
    import torch
    shape = (4, 64, 12, 12, 32, 3, 3, 1, 1)
    x, w, st, pd = make(shape, 892, "NCHW")
    acc, mag = oracle.conv2d(x, w, st, pd, "NCHW")
    add = np.random.Generator(np.random.PCG64(893)).standard_normal(acc.shape).astype(np.float32)
    N, C, H, W, K, R, S = mg3m.dims_of(x, w, "NCHW")
    wsb = mg3m.conv2d_fwd_f32_hw_workspace_bytes(N, C, H, W, K, R, S, 1, 1, 1, 1, "NCHW", plan)
    ws = torch.empty(max(1, wsb // 4), dtype=torch.float32, device="cuda")
    xd, wd = to_dev(x), to_dev(w)
    for inplace in (False, True):
        addd = to_dev(add)
        y = addd if inplace else torch.empty(acc.shape, dtype=torch.float32, device="cuda")
        mg3m.conv2d_fwd_f32_fused(xd, wd, y, addd, 1, N, C, H, W, K, R, S, 1, 1, 1, 1, "NCHW", ws, wsb, plan)
        v = acc + add.astype(np.float64)
        ref = np.maximum(v, 0.0)
        tol = RTOL * mag + 2.0 ** -23 * (np.abs(acc) + np.abs(add))
        assert np.all(np.abs(y.cpu().numpy().astype(np.float64) - ref) <= tol), f"inplace={inplace}"


def test_selector_runs_small_spatial_nchw_layers_as_hwcn():
    """A 14x14, 512-channel NCHW layer (VGG-16's last block, at a smaller
    batch) runs as HWCN in the selector's plan, exactly."""
    shape = (8, 512, 14, 14, 512, 3, 3, 1, 1)
    info = mg3m.conv2d_fwd_f32_plan_info(*shape, "NCHW")
    say(f"selector NCHW {shape}: via_hwcn {info['via_hwcn']} est {info['est_us']:.1f} us")
    assert info["via_hwcn"] == 1, info
    x, w, st, pd, exact = _exact(shape, 895)
    y = run_gpu(x, w, st, pd, "NCHW")
    assert np.array_equal(y, exact)


@pytest.mark.parametrize("shape", [
    (2, 70, 9, 9, 130, 1, 1, 1, 0),          # filter copy: 4-byte loads and stores; 1x1 taps (B = 1)
    (8, 64, 8, 8, 64, 3, 3, 1, 1),           # every copy with 16-byte loads and stores
    (4, 67, 6, 6, 128, 3, 3, 1, 1),          # filter copy: 4-byte loads, 16-byte stores
    (5, 36, 20, 20, 72, 1, 1, 2, 0),         # x copy: 16-byte loads, 4-byte stores (N = 5)
    (3, 130, 5, 7, 66, 3, 3, 1, 1),          # tiles across c with ragged a and j edges
])
def test_layout_change_paths(shape):
    """The layout-change kernel reads in[a][c*B + b] in 64 x 64 tiles, so a
    tile spans several c when B is small; each mix of 16-byte and 4-byte loads
    and stores, ragged edges in a and j, and B = 1 (1x1 filters), exactly."""
    x, w, st, pd, exact = _exact(shape, 900 + shape[1])
    say(f"layout change {shape}")
    y = run_gpu(x, w, st, pd, "NCHW", plan="via=hwcn")
    assert np.array_equal(y, exact), shape
