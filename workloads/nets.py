"""Layer lists of the convolution stacks of real networks, for the network
executor (mg3m_net_*): the feature extractors of VGG-16 and AlexNet and the
ResNet-50 trunk (the networks of the paper's Sec. 5.2 whose layers the
catalogues in ``workloads`` hold), with ReLU after every convolution, max
pooling between blocks, and ResNet's residual connections.

Each network is a list of dicts (the keys of ``mg3m.Net``); ``filters``
attaches seeded He-normal filters (fan-in C*R*S) as device tensors in the
network's layout.  Everything is synthetic: no trained weights."""
from __future__ import annotations


def _conv(layers, chans, inp, K, R, stride=1, pad=0, relu=1, add=-1):
    layers.append({"op": "conv", "input": inp, "K": K, "R": R, "S": R, "stride": stride, "pad": pad,
                   "relu": relu, "add": add, "C": chans[inp]})
    chans.append(K)
    return len(layers)          # id of the new activation


def _pool(layers, chans, inp, R, stride, pad=0):
    layers.append({"op": "maxpool", "input": inp, "R": R, "S": R, "stride": stride, "pad": pad})
    chans.append(chans[inp])
    return len(layers)


def vgg16_features(C=3):
    """13 3x3 convolutions (pad 1) in five blocks, 2x2 max pooling after each."""
    layers, chans, a = [], [C], 0
    for block, (K, n) in enumerate([(64, 2), (128, 2), (256, 3), (512, 3), (512, 3)]):
        for _ in range(n):
            a = _conv(layers, chans, a, K, 3, 1, 1)
        a = _pool(layers, chans, a, 2, 2)
    return layers


def alexnet_features(C=3):
    """AlexNet's five convolutions with 3x3 stride-2 max pooling after the
    first, second and fifth."""
    layers, chans = [], [C]
    a = _conv(layers, chans, 0, 64, 11, 4, 2)
    a = _pool(layers, chans, a, 3, 2)
    a = _conv(layers, chans, a, 192, 5, 1, 2)
    a = _pool(layers, chans, a, 3, 2)
    a = _conv(layers, chans, a, 384, 3, 1, 1)
    a = _conv(layers, chans, a, 256, 3, 1, 1)
    a = _conv(layers, chans, a, 256, 3, 1, 1)
    _pool(layers, chans, a, 3, 2)
    return layers


def resnet50_trunk(C=3, stages=((64, 3, 1), (128, 4, 2), (256, 6, 2), (512, 3, 2))):
    """7x7 stride-2 stem, 3x3 stride-2 max pooling, then bottleneck blocks
    (1x1 reduce, 3x3 with the stage's stride, 1x1 expand to 4x width, plus the
    shortcut -- a strided 1x1 projection in each stage's first block -- added
    before the final ReLU)."""
    layers, chans = [], [C]
    a = _conv(layers, chans, 0, 64, 7, 2, 3)
    a = _pool(layers, chans, a, 3, 2, 1)
    for width, blocks, stride in stages:
        for b in range(blocks):
            s = stride if b == 0 else 1
            inp = a
            t = _conv(layers, chans, inp, width, 1)
            t = _conv(layers, chans, t, width, 3, s, 1)
            sc = inp
            if b == 0:
                sc = _conv(layers, chans, inp, 4 * width, 1, s, 0, relu=0)
            a = _conv(layers, chans, t, 4 * width, 1, relu=1, add=sc)
    return layers


NETS = {"vgg16": vgg16_features, "alexnet": alexnet_features, "resnet50": resnet50_trunk}


def filters(layers, layout="HWCN", seed=0, device="cuda"):
    """Attach a seeded He-normal filter to every convolution (in place);
    returns the layers.  HWCN filters are [R][S][C][K], NCHW [K][C][R][S]."""
    import math

    import torch
    g = torch.Generator(device="cpu").manual_seed(seed)
    for d in layers:
        if d["op"] != "conv":
            continue
        C, K, R, S = d["C"], d["K"], d["R"], d["S"]
        w = torch.randn((K, C, R, S), generator=g, dtype=torch.float32) * math.sqrt(2.0 / (C * R * S))
        if layout == "HWCN":
            w = w.permute(2, 3, 1, 0)
        d["w"] = w.contiguous().to(device)
    return layers


def conv_flops(layers, input_shape):
    """Multiply-add flops (2 per MAC, padded taps included) of every
    convolution of the chain, and the list of per-layer output shapes (N, C, H, W)."""
    N, C, H, W = input_shape
    shapes = [(N, C, H, W)]
    total = 0.0
    for d in layers:
        n, c, h, w = shapes[d["input"]]
        ho = (h + 2 * d["pad"] - d["R"]) // d["stride"] + 1
        wo = (w + 2 * d["pad"] - d["S"]) // d["stride"] + 1
        if d["op"] == "conv":
            total += 2.0 * n * d["K"] * c * d["R"] * d["S"] * ho * wo
            shapes.append((n, d["K"], ho, wo))
        else:
            shapes.append((n, c, ho, wo))
    return total, shapes
