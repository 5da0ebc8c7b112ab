"""GPU parity at full layer sizes, in the launch configuration the benchmark
times (the selector's plan, HWCN): every layer of every catalogue workload --
the benchmark configurations and the paper's Sec. 5.1 scene sweeps -- and the
network catalogues again in NCHW.  The oracle computes a seeded sample of
outputs one by one: outputs that see the padding (HWCN: the two corner pixels,
all of them up to 4096 per pixel; NCHW: the border rows and columns of 32
(image, channel) planes), plus random ones; every output is also checked to be
finite."""
import numpy as np
import pytest

import oracle
import workloads
from paper_2307_04941_amd import mg3m
from tests.gpu_util import RTOL, say

pytestmark = pytest.mark.gpu

LAYERS = [(wl, i) for wl, (_, layers) in workloads.WORKLOADS.items() for i in range(len(layers))]
CORNER_CAP = 4096


@pytest.mark.parametrize("wl,index", LAYERS, ids=[f"{wl}-{i}" for wl, i in LAYERS])
def test_layer_sampled(wl, index):
    import torch
    layer, x, w = workloads.layer_tensors(wl, index, "HWCN")
    say(f"layer {wl}/{layer.name} N={layer.N} C={layer.C} HW={layer.H} K={layer.K} "
        f"RS={layer.R} s={layer.stride} p={layer.pad}: "
        + mg3m.conv2d_fwd_f32_plan_string(layer.N, layer.C, layer.H, layer.W, layer.K, layer.R,
                                          layer.S, layer.stride, layer.pad, "HWCN"))
    xd, wd = torch.from_numpy(x).cuda(), torch.from_numpy(w).cuda()
    y = mg3m.conv2d_fwd(xd, wd, layer.stride, layer.pad, "HWCN")
    torch.cuda.synchronize()
    assert torch.isfinite(y).all().item(), "non-finite output"
    Ho, Wo, K, N = y.shape
    per_pix = K * N
    rng = np.random.Generator(np.random.PCG64(4242 + index))
    last = (Ho * Wo - 1) * per_pix
    if per_pix <= CORNER_CAP:
        c0, c1 = np.arange(0, per_pix), np.arange(last, last + per_pix)
    else:
        c0 = rng.choice(per_pix, CORNER_CAP, replace=False)
        c1 = last + rng.choice(per_pix, CORNER_CAP, replace=False)
    idx = np.concatenate([c0, c1, rng.integers(0, y.numel(), 8192)]).astype(np.int64)
    got = y.view(-1)[torch.from_numpy(idx).cuda()].cpu().numpy().astype(np.float64)
    acc, mag = oracle.conv2d_points(x, w, idx, layer.stride, layer.pad, "HWCN")
    err = np.abs(got - acc)
    bad = ~(err <= RTOL * mag)
    worst = float(np.max(np.where(mag > 0, err / (RTOL * np.where(mag > 0, mag, 1)), 0)))
    say(f"  sampled {idx.size} outputs, worst ratio {worst:.3g}")
    del xd, wd, y
    torch.cuda.empty_cache()
    assert not bad.any(), f"{int(bad.sum())} sampled outputs outside tolerance (worst {worst:.3g})"


NCHW_LAYERS = [(wl, i) for wl in workloads.CONFIG_WORKLOADS for i in range(len(workloads.workload(wl)))
               if wl != "scene_sweep"]


@pytest.mark.parametrize("wl,index", NCHW_LAYERS, ids=[f"{wl}-{i}" for wl, i in NCHW_LAYERS])
def test_layer_sampled_nchw(wl, index):
    import torch
    layer, x, w = workloads.layer_tensors(wl, index, "NCHW")
    say(f"layer NCHW {wl}/{layer.name} N={layer.N} C={layer.C} HW={layer.H} K={layer.K} "
        f"RS={layer.R} s={layer.stride} p={layer.pad}: "
        + mg3m.conv2d_fwd_f32_plan_string(layer.N, layer.C, layer.H, layer.W, layer.K, layer.R,
                                          layer.S, layer.stride, layer.pad, "NCHW"))
    xd, wd = torch.from_numpy(x).cuda(), torch.from_numpy(w).cuda()
    y = mg3m.conv2d_fwd(xd, wd, layer.stride, layer.pad, "NCHW")
    torch.cuda.synchronize()
    assert torch.isfinite(y).all().item(), "non-finite output"
    N, K, Ho, Wo = y.shape
    rng = np.random.Generator(np.random.PCG64(4343 + index))
    planes = rng.integers(0, N * K, 32)
    border = [(p * Ho + oh) * Wo + ow for p in planes for oh in range(Ho) for ow in range(Wo)
              if oh in (0, Ho - 1) or ow in (0, Wo - 1)]
    idx = np.concatenate([np.asarray(border, np.int64), rng.integers(0, y.numel(), 8192)]).astype(np.int64)
    got = y.view(-1)[torch.from_numpy(idx).cuda()].cpu().numpy().astype(np.float64)
    acc, mag = oracle.conv2d_points(x, w, idx, layer.stride, layer.pad, "NCHW")
    err = np.abs(got - acc)
    bad = ~(err <= RTOL * mag)
    worst = float(np.max(np.where(mag > 0, err / (RTOL * np.where(mag > 0, mag, 1)), 0)))
    say(f"  sampled {idx.size} outputs, worst ratio {worst:.3g}")
    del xd, wd, y
    torch.cuda.empty_cache()
    assert not bad.any(), f"{int(bad.sum())} sampled outputs outside tolerance (worst {worst:.3g})"
