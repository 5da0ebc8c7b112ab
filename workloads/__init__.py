"""Seeded synthetic inputs and the layer catalogues they are shaped after.

This module serves both the tests (oracle side) and the benchmark (GPU side).
It holds no arithmetic of the convolution itself: only layer shapes (as the
architectures define them), seeded random tensors, and layout permutations
(pure data movement).  It does not even compute output sizes.

Inputs stand in for the paper's workloads (Sec. 5): the paper's CNN
experiments use only layer shapes, so seeded uniform / He-normal tensors of
those shapes replace real activations and trained weights.

Random recipe (numpy PCG64): a tensor of n elements, in logical order, is
cut into chunks of 2^22 elements and chunk i is drawn from the stream
``PCG64(seed).jumped(i)`` (chunks are drawn in parallel threads; the values do
not depend on the thread count):
  * x ~ uniform[-1, 1): ``random(float32) * 2 - 1``, drawn in logical
    (N, C, H, W) order, then permuted to the requested layout;
  * w ~ He-normal ``standard_normal(float32) * sqrt(2 / (C*R*S))`` or uniform
    [-1, 1), drawn in logical (K, C, R, S) order, then permuted;
  * small-integer data: x, w drawn uniformly from {-2, ..., 2};
  * seed(x) = 230704941 + 10000 * workload_id + 10 * layer_index,
    seed(w) = seed(x) + 1.
Both layouts of one seed are the same logical tensors.  Layout permutations
are done by torch on the CPU (multi-threaded data movement only).
"""
from __future__ import annotations

import concurrent.futures
import os
from dataclasses import dataclass, asdict
from typing import List

import numpy as np

SEED_BASE = 230704941


@dataclass(frozen=True)
class Layer:
    name: str
    N: int
    C: int
    H: int
    W: int
    K: int
    R: int
    S: int
    stride: int = 1
    pad: int = 0
    mult: int = 1                     # occurrences in the network (aggregates only)
    wdist: str = "uniform"            # "uniform" or "he"

    def as_dict(self):
        return asdict(self)


def _sweep_scenes() -> List[Layer]:
    out = []
    for n in (1, 4, 32, 128):
        for ch in (16, 64, 256):
            hw = 56 if ch <= 64 else 28
            out.append(Layer(f"scene_N{n}_C{ch}", n, ch, hw, hw, ch, 3, 3, 1, 1))
    return out


def _vgg16(n=64) -> List[Layer]:
    spec = [(3, 64, 224), (64, 64, 224), (64, 128, 112), (128, 128, 112),
            (128, 256, 56), (256, 256, 56), (256, 256, 56),
            (256, 512, 28), (512, 512, 28), (512, 512, 28),
            (512, 512, 14), (512, 512, 14), (512, 512, 14)]
    return [Layer(f"vgg16_conv{i + 1}", n, c, hw, hw, k, 3, 3, 1, 1, 1, "he")
            for i, (c, k, hw) in enumerate(spec)]


def _resnet50(n=32) -> List[Layer]:
    # ResNet-50 v1.5 (stride on the 3x3 of the first block of a stage); one entry
    # per unique shape, `mult` = how often it occurs in the 53-conv network.
    L = lambda nm, c, k, hw, r, st, p, m: Layer(f"rn50_{nm}", n, c, hw, hw, k, r, r, st, p, m, "he")
    return [
        L("stem", 3, 64, 224, 7, 2, 3, 1),
        L("c2_1x1a_first", 64, 64, 56, 1, 1, 0, 1),
        L("c2_3x3", 64, 64, 56, 3, 1, 1, 3),
        L("c2_1x1b_ds", 64, 256, 56, 1, 1, 0, 4),
        L("c2_1x1a", 256, 64, 56, 1, 1, 0, 2),
        L("c3_1x1a_first", 256, 128, 56, 1, 1, 0, 1),
        L("c3_3x3_s2", 128, 128, 56, 3, 2, 1, 1),
        L("c3_1x1b", 128, 512, 28, 1, 1, 0, 4),
        L("c3_ds_s2", 256, 512, 56, 1, 2, 0, 1),
        L("c3_1x1a", 512, 128, 28, 1, 1, 0, 3),
        L("c3_3x3", 128, 128, 28, 3, 1, 1, 3),
        L("c4_1x1a_first", 512, 256, 28, 1, 1, 0, 1),
        L("c4_3x3_s2", 256, 256, 28, 3, 2, 1, 1),
        L("c4_1x1b", 256, 1024, 14, 1, 1, 0, 6),
        L("c4_ds_s2", 512, 1024, 28, 1, 2, 0, 1),
        L("c4_1x1a", 1024, 256, 14, 1, 1, 0, 5),
        L("c4_3x3", 256, 256, 14, 3, 1, 1, 5),
        L("c5_1x1a_first", 1024, 512, 14, 1, 1, 0, 1),
        L("c5_3x3_s2", 512, 512, 14, 3, 2, 1, 1),
        L("c5_1x1b", 512, 2048, 7, 1, 1, 0, 3),
        L("c5_ds_s2", 1024, 2048, 14, 1, 2, 0, 1),
        L("c5_1x1a", 2048, 512, 7, 1, 1, 0, 2),
        L("c5_3x3", 512, 512, 7, 3, 1, 1, 2),
    ]


def _alexnet_inception(n=128) -> List[Layer]:
    return [
        Layer("alex_conv1", n, 3, 224, 224, 64, 11, 11, 4, 2),
        Layer("alex_conv2", n, 64, 27, 27, 192, 5, 5, 1, 2),
        Layer("alex_conv3", n, 192, 13, 13, 384, 3, 3, 1, 1),
        Layer("alex_conv4", n, 384, 13, 13, 256, 3, 3, 1, 1),
        Layer("alex_conv5", n, 256, 13, 13, 256, 3, 3, 1, 1),
        Layer("incep3a_1x1", n, 192, 28, 28, 64, 1, 1, 1, 0),
        Layer("incep3a_3x3", n, 96, 28, 28, 128, 3, 3, 1, 1),
        Layer("incep3a_5x5", n, 16, 28, 28, 32, 5, 5, 1, 2),
    ]


# ------------------------------------------------ the paper's scene sweeps
# Sec. 5.1 varies one convolution parameter group at a time; the paper does
# not state the spatial size, the batch of the channel / filter / pad-stride
# sweeps, nor the padding of the filter sweep.  Readings used here: input
# 56x56 when both channel counts are <= 64, else 28x28; B = 128 where B is
# not the swept parameter; 3x3 filters with pad 1 and stride 1 unless swept;
# "same" padding (pad = fltH // 2) in the filter sweep.
CHANNEL_GROUPS = {"small": (16, 32, 48, 64), "medium": (64, 128, 192, 256),
                  "big": (256, 512, 768, 1024)}
IC_EQ_OC = (16, 32, 48, 64, 128, 192, 256, 512, 768, 1024)


def _hw(c, k):
    return 56 if max(c, k) <= 64 else 28


def _channel_scenes(n=128) -> List[Layer]:
    """Sec. 5.1.1: 16 (IC, OC) scenes in each of three channel scales."""
    out = []
    for g, vals in CHANNEL_GROUPS.items():
        for c in vals:
            for k in vals:
                hw = _hw(c, k)
                out.append(Layer(f"{g}_C{c}_K{k}", n, c, hw, hw, k, 3, 3, 1, 1))
    return out


def _batch_sweep() -> List[Layer]:
    """Sec. 5.1.2 (and the scenes of Sec. 5.3, Table 2): B in {64, 128, 256}
    with IC = OC over the channel values of Sec. 5.1.1."""
    return [Layer(f"B{n}_C{c}", n, c, _hw(c, c), _hw(c, c), c, 3, 3, 1, 1)
            for n in (64, 128, 256) for c in IC_EQ_OC]


def _filter_sweep(n=128) -> List[Layer]:
    """Sec. 5.1.3: fltH = fltW in {3, 5, 7, 9, 11} with IC = OC."""
    return [Layer(f"F{r}_C{c}", n, c, _hw(c, c), _hw(c, c), c, r, r, 1, r // 2)
            for r in (3, 5, 7, 9, 11) for c in IC_EQ_OC]


def _padstride_sweep(n=128) -> List[Layer]:
    """Sec. 5.1.4: (pad, stride) in {(0, 1), (1, 1), (0, 2), (1, 2)}, 3x3, IC = OC."""
    return [Layer(f"P{p}S{s}_C{c}", n, c, _hw(c, c), _hw(c, c), c, 3, 3, s, p)
            for (p, s) in ((0, 1), (1, 1), (0, 2), (1, 2)) for c in IC_EQ_OC]


# workload id -> (name, layers); the id enters the seed
WORKLOADS = {
    "single_16x16_32px": (1, [Layer("single", 1, 16, 32, 32, 16, 3, 3, 1, 1)]),
    "scene_sweep": (2, _sweep_scenes()),
    "vgg16_n64": (3, _vgg16()),
    "resnet50_n32": (4, _resnet50()),
    "alexnet_inception_n128": (5, _alexnet_inception()),
    "channel_scenes_n128": (6, _channel_scenes()),
    "batch_sweep": (7, _batch_sweep()),
    "filter_sweep_n128": (8, _filter_sweep()),
    "padstride_sweep_n128": (9, _padstride_sweep()),
}

# the workloads named by the benchmark configurations; the others are the
# paper's Sec. 5.1 / 5.3 scene sweeps
CONFIG_WORKLOADS = ("single_16x16_32px", "scene_sweep", "vgg16_n64", "resnet50_n32",
                    "alexnet_inception_n128")
SWEEP_WORKLOADS = ("channel_scenes_n128", "batch_sweep", "filter_sweep_n128",
                   "padstride_sweep_n128")


def workload(name: str) -> List[Layer]:
    return WORKLOADS[name][1]


def seeds(workload_name: str, layer_index: int):
    wid = WORKLOADS[workload_name][0]
    sx = SEED_BASE + 10000 * wid + 10 * layer_index
    return sx, sx + 1


# ---------------------------------------------------------------- layouts
def _permute(a, order):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a)).permute(*order).contiguous().numpy()


def nchw_to_hwcn(x):      # x[N,C,H,W] -> x[H,W,C,N]
    return _permute(x, (2, 3, 1, 0))


def kcrs_to_rsck(w):      # w[K,C,R,S] -> w[R,S,C,K]
    return _permute(w, (2, 3, 1, 0))


def hwcn_to_nchw(y):      # y[Ho,Wo,K,N] -> y[N,K,Ho,Wo]
    return _permute(y, (3, 2, 0, 1))


def to_layout(x_nchw, w_kcrs, layout: str):
    if layout == "NCHW":
        return np.ascontiguousarray(x_nchw), np.ascontiguousarray(w_kcrs)
    if layout == "HWCN":
        return nchw_to_hwcn(x_nchw), kcrs_to_rsck(w_kcrs)
    raise ValueError(layout)


# ---------------------------------------------------------------- generators
CHUNK = 1 << 22
_THREADS = max(1, min(16, os.cpu_count() or 1))


def _draw(n, seed, fill):
    """n values in logical order; chunk i from PCG64(seed).jumped(i).
    fill(generator, out_view) writes one chunk."""
    out = np.empty(n, np.float32)
    chunks = (n + CHUNK - 1) // CHUNK

    def one(i):
        g = np.random.Generator(np.random.PCG64(seed).jumped(i))
        fill(g, out[i * CHUNK:min(n, (i + 1) * CHUNK)])

    if chunks <= 1:
        for i in range(chunks):
            one(i)
    else:
        with concurrent.futures.ThreadPoolExecutor(min(_THREADS, chunks)) as ex:
            list(ex.map(one, range(chunks)))
    return out


def uniform(shape, seed):
    n = int(np.prod(shape))

    def fill(g, o):
        g.random(out=o, dtype=np.float32)
        o *= np.float32(2)
        o -= np.float32(1)
    return _draw(n, seed, fill).reshape(shape)


def he_normal(shape, fan_in, seed):
    n = int(np.prod(shape))
    scale = np.float32(np.sqrt(2.0 / fan_in))

    def fill(g, o):
        g.standard_normal(out=o, dtype=np.float32)
        o *= scale
    return _draw(n, seed, fill).reshape(shape)


def small_int(shape, seed, lo=-2, hi=2):
    n = int(np.prod(shape))

    def fill(g, o):
        o[:] = g.integers(lo, hi + 1, size=o.size)
    return _draw(n, seed, fill).reshape(shape)


def make_tensors(layer: Layer, seed_x: int, seed_w: int, layout: str = "HWCN", dist: str = None):
    """Logical tensors x[N,C,H,W], w[K,C,R,S] for one layer, returned in `layout`.
    dist: None -> x uniform and w per layer.wdist; "int" -> small integers
    (every partial sum an integer below 2^24); "wideint" -> integers in
    [-2048, 2048] (products up to 2^22, sums past 2^24 but far below 2^53)."""
    xs = (layer.N, layer.C, layer.H, layer.W)
    ws = (layer.K, layer.C, layer.R, layer.S)
    if dist == "int":
        x = small_int(xs, seed_x)
        w = small_int(ws, seed_w)
    elif dist == "wideint":
        x = small_int(xs, seed_x, -2048, 2048)
        w = small_int(ws, seed_w, -2048, 2048)
    else:
        x = uniform(xs, seed_x)
        if layer.wdist == "he":
            w = he_normal(ws, layer.C * layer.R * layer.S, seed_w)
        else:
            w = uniform(ws, seed_w)
    return to_layout(x, w, layout)


def layer_tensors(workload_name: str, index: int, layout: str = "HWCN", dist: str = None):
    layer = workload(workload_name)[index]
    sx, sw = seeds(workload_name, index)
    return layer, *make_tensors(layer, sx, sw, layout, dist)
