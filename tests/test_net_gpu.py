"""GPU parity of the pieces around the convolution that the network executor
chains: max pooling (bit-exact against the oracle), the fused output stage
y = relu(conv + add) (the convolution's 1e-5 * sum|x*w| bound plus one fp32
rounding of the addition), and whole chains (mg3m_net_*): every layer checked
against the oracle applied to the layer's own inputs as the GPU produced
them, liveness-packed activations equal to separately kept ones, and HIP-graph
replays equal to eager runs."""
import numpy as np
import pytest

import oracle
import workloads
import workloads.nets as nets
from paper_2307_04941_amd import mg3m
from tests.gpu_util import RTOL, make, say, to_dev

pytestmark = pytest.mark.gpu


def _pool_cases():
    return [
        ((2, 8, 12, 12), 2, 2, 0, "HWCN"),        # VGG-style 2x2/2, vectorised path
        ((4, 16, 13, 13), 3, 2, 0, "HWCN"),       # AlexNet 3x3/2
        ((2, 8, 15, 11), 3, 2, 1, "HWCN"),        # ResNet stem pool, padded
        ((3, 5, 9, 9), 3, 1, 1, "HWCN"),          # C*N not a multiple of 4: element path
        ((2, 8, 12, 12), 2, 2, 0, "NCHW"),
        ((3, 5, 10, 7), 3, 2, 1, "NCHW"),
    ]


@pytest.mark.parametrize("case", range(len(_pool_cases())))
def test_maxpool_bit_exact(case):
    (N, C, H, W), R, st, pd, layout = _pool_cases()[case]
    say(f"maxpool {layout} N={N} C={C} {H}x{W} R={R} s={st} p={pd}")
    rng = np.random.Generator(np.random.PCG64(900 + case))
    xl = rng.standard_normal((N, C, H, W)).astype(np.float32)
    x = xl if layout == "NCHW" else np.ascontiguousarray(np.transpose(xl, (2, 3, 1, 0)))
    y = mg3m.maxpool2d(to_dev(x), R, R, st, pd, layout).cpu().numpy()
    ref = oracle.maxpool2d(x, R, R, st, pd, layout)
    assert np.array_equal(y, ref)


def test_maxpool_misaligned_and_nan():
    import torch
    rng = np.random.Generator(np.random.PCG64(950))
    x = rng.standard_normal((8, 8, 4, 4)).astype(np.float32)          # HWCN, C*N = 16
    x[3, 5, 2, 1] = np.nan
    buf = torch.empty(x.size + 1, dtype=torch.float32, device="cuda")
    buf[1:].copy_(torch.from_numpy(x.reshape(-1)))
    xd = buf[1:].view(x.shape)                                          # 4-byte aligned only
    y = mg3m.maxpool2d(xd, 2, 2, 2, 0, "HWCN").cpu().numpy()
    ref = oracle.maxpool2d(x, 2, 2, 2, 0, "HWCN")
    assert np.array_equal(np.isnan(y), np.isnan(ref)) and np.isnan(y).sum() == 1
    assert np.array_equal(np.nan_to_num(y), np.nan_to_num(ref))


def _fused_ref(acc, mag, add, relu):
    v = acc + (add.astype(np.float64) if add is not None else 0.0)
    ref = np.maximum(v, 0.0) if relu else v
    tol = RTOL * mag + 2.0 ** -23 * (np.abs(acc) + (np.abs(add) if add is not None else 0.0))
    return ref, tol


@pytest.mark.parametrize("layout", ["HWCN", "NCHW"])
@pytest.mark.parametrize("plan,shape", [
    (None, (4, 16, 12, 12, 32, 3, 3, 1, 1)),
    ("tile=128x128,split=3", (4, 16, 12, 12, 32, 3, 3, 1, 1)),      # finished in the split reduction
    (None, (1, 12, 9, 9, 24, 3, 3, 1, 1)),                           # N = 1: 16-byte channel stores
    (None, (8, 16, 14, 14, 16, 3, 3, 1, 1)),                         # K = 16: 16x64 tile, 16x16x4 MFMAs
    ("tile=16x64,split=3", (4, 16, 12, 12, 48, 3, 3, 1, 1)),        # 16x64 pieces, finished in the reduction
])
def test_fused_add_relu(layout, plan, shape):
    import torch
    say(f"fused {layout} {plan} {shape}")
    x, w, st, pd = make(shape, 960, layout)
    acc, mag = oracle.conv2d(x, w, st, pd, layout)
    rng = np.random.Generator(np.random.PCG64(961))
    add = rng.standard_normal(acc.shape).astype(np.float32)
    N, C, H, W, K, R, S = mg3m.dims_of(x, w, layout)
    wsb = mg3m.conv2d_fwd_f32_hw_workspace_bytes(N, C, H, W, K, R, S, 1, 1, 1, 1, layout, plan)
    ws = torch.empty(max(1, (wsb + 3) // 4), dtype=torch.float32, device="cuda")
    xd, wd = to_dev(x), to_dev(w)
    for relu in (0, 1):
        for inplace in (False, True):
            addd = to_dev(add)
            y = addd if inplace else torch.empty(acc.shape, dtype=torch.float32, device="cuda")
            mg3m.conv2d_fwd_f32_fused(xd, wd, y, addd, relu, N, C, H, W, K, R, S, 1, 1, 1, 1, layout,
                                      ws, ws.numel() * 4, plan)
            got = y.cpu().numpy().astype(np.float64)
            ref, tol = _fused_ref(acc, mag, add, relu)
            assert np.all(np.abs(got - ref) <= tol), f"relu={relu} inplace={inplace}"
    # relu without add, and NaN kept by the ReLU
    y = torch.empty(acc.shape, dtype=torch.float32, device="cuda")
    mg3m.conv2d_fwd_f32_fused(xd, wd, y, None, 1, N, C, H, W, K, R, S, 1, 1, 1, 1, layout,
                              ws, ws.numel() * 4, plan)
    ref, tol = _fused_ref(acc, mag, None, 1)
    assert np.all(np.abs(y.cpu().numpy() - ref) <= tol)


@pytest.mark.parametrize("plan,shape", [
    (None, (32, 3, 64, 64, 64, 3, 3, 1, 1)),                        # first-layer shape: the selector's pick
    ("tile=128x128,persist=1", (4, 64, 13, 11, 68, 3, 3, 1, 1)),    # ragged rows and columns, 1-tap loaders
    ("tile=64x256,persist=1", (32, 3, 56, 56, 64, 3, 3, 1, 1)),     # several tiles per work-group
])
def test_fused_add_relu_persistent(plan, shape):
    """The persistent whole-tile kernel's fused output stage: add read and
    ReLU applied in its buffer-store epilogue (HWCN only)."""
    import torch
    info = mg3m.conv2d_fwd_f32_plan_info(*shape, "HWCN", plan)
    assert info["persistent"] == 1, info
    say(f"fused persistent {plan} {shape}: grid {info['grid']} tiles {info['dp_tiles']}")
    x, w, st, pd = make(shape, 962, "HWCN")
    acc, mag = oracle.conv2d(x, w, st, pd, "HWCN")
    rng = np.random.Generator(np.random.PCG64(963))
    add = rng.standard_normal(acc.shape).astype(np.float32)
    N, C, H, W, K, R, S = mg3m.dims_of(x, w, "HWCN")
    ws = torch.empty(1, dtype=torch.float32, device="cuda")
    xd, wd = to_dev(x), to_dev(w)
    for relu in (0, 1):
        for inplace in (False, True):
            addd = to_dev(add)
            y = addd if inplace else torch.empty(acc.shape, dtype=torch.float32, device="cuda")
            mg3m.conv2d_fwd_f32_fused(xd, wd, y, addd, relu, N, C, H, W, K, R, S, 1, 1, 1, 1, "HWCN",
                                      ws, 4, plan)
            got = y.cpu().numpy().astype(np.float64)
            ref, tol = _fused_ref(acc, mag, add, relu)
            assert np.all(np.abs(got - ref) <= tol), f"relu={relu} inplace={inplace}"
    y = torch.empty(acc.shape, dtype=torch.float32, device="cuda")
    mg3m.conv2d_fwd_f32_fused(xd, wd, y, None, 1, N, C, H, W, K, R, S, 1, 1, 1, 1, "HWCN", ws, 4, plan)
    ref, tol = _fused_ref(acc, mag, None, 1)
    assert np.all(np.abs(y.cpu().numpy() - ref) <= tol)


MINI = [
    {"op": "conv", "input": 0, "K": 16, "R": 3, "stride": 1, "pad": 1, "relu": 1},     # 1
    {"op": "conv", "input": 1, "K": 16, "R": 3, "stride": 1, "pad": 1, "relu": 0},     # 2
    {"op": "maxpool", "input": 2, "R": 3, "stride": 2, "pad": 1},                       # 3
    {"op": "conv", "input": 3, "K": 16, "R": 3, "stride": 1, "pad": 1, "relu": 1, "add": 3},  # 4: residual
    {"op": "conv", "input": 4, "K": 32, "R": 1, "stride": 2, "pad": 0, "relu": 1},     # 5
    {"op": "conv", "input": 1, "K": 32, "R": 3, "stride": 4, "pad": 1, "relu": 0},     # 6: branch from 1
    {"op": "conv", "input": 5, "K": 32, "R": 3, "stride": 1, "pad": 1, "relu": 1, "add": 6},  # 7
    {"op": "maxpool", "input": 7, "R": 2, "stride": 2, "pad": 0},                       # 8
]


def _with_channels(layers, C0):
    chans = [C0]
    out = []
    for d in layers:
        d = dict(d)
        if d["op"] == "conv":
            d["C"] = chans[d["input"]]
            d["S"] = d["R"]
            chans.append(d["K"])
        else:
            d["S"] = d["R"]
            chans.append(chans[d["input"]])
        out.append(d)
    return out


def _host(t):
    return t.detach().cpu().numpy()


def _check_chain(net, layers, x_host, y_host, layout, sample=None, seed=0):
    """Every layer against the oracle applied to its own GPU inputs."""
    acts = {0: x_host, len(layers): y_host}
    for i in range(1, len(layers)):
        a = _host(net.activation(i))          # stored activations are HWCN in every network
        acts[i] = a if layout == "HWCN" else np.ascontiguousarray(np.transpose(a, (3, 2, 0, 1)))
    rng = np.random.Generator(np.random.PCG64(seed))
    worst = 0.0
    for i, d in enumerate(layers):
        got, src = acts[i + 1], acts[d["input"]]
        if d["op"] == "maxpool":
            ref = oracle.maxpool2d(src, d["R"], d["S"], d["stride"], d["pad"], layout)
            assert np.array_equal(got, ref), f"layer {i} (maxpool)"
            continue
        w = _host(d["w"])
        add = acts[d["add"]] if d.get("add", -1) >= 0 else None
        if sample is None or got.size <= sample:
            acc, mag = oracle.conv2d(src, w, d["stride"], d["pad"], layout)
            idx = None
        else:
            idx = rng.integers(0, got.size, sample)
            acc, mag = oracle.conv2d_points(src, w, idx, d["stride"], d["pad"], layout)
        g = got.reshape(-1)[idx] if idx is not None else got
        a = (add.reshape(-1)[idx] if idx is not None else add) if add is not None else None
        ref, tol = _fused_ref(acc, mag, a, d.get("relu", 0))
        err = np.abs(g.astype(np.float64) - ref)
        assert np.all(err <= tol), f"layer {i}: {int((err > tol).sum())} outputs out of bound"
        worst = max(worst, float(np.max(np.where(tol > 0, err / np.where(tol > 0, tol, 1), 0))))
    return worst


@pytest.mark.parametrize("layout", ["HWCN", "NCHW"])
def test_mini_chain_every_layer(layout):
    import torch
    layers = nets.filters(_with_channels(MINI, 8), layout, seed=5)
    shape = (4, 8, 19, 17)
    net = mg3m.Net(layers, shape, layout, keep_all=True)
    x = make((4, 8, 19, 17, 1, 1, 1, 1, 0), 970, layout)[0]
    y = net.forward(to_dev(x))
    torch.cuda.synchronize()
    say(f"mini chain {layout}: output {tuple(y.shape)}, arena {net.memory()}")
    worst = _check_chain(net, layers, x, _host(y), layout)
    say(f"  worst ratio to the bound {worst:.3g}")
    net.close()


@pytest.mark.parametrize("layout", ["HWCN", "NCHW"])
def test_packed_arena_equals_kept_activations(layout):
    import torch
    layers = nets.filters(_with_channels(MINI, 8), layout, seed=6)
    x = to_dev(make((4, 8, 19, 17, 1, 1, 1, 1, 0), 971, layout)[0])
    kept = mg3m.Net(layers, (4, 8, 19, 17), layout, keep_all=True)
    packed = mg3m.Net(layers, (4, 8, 19, 17), layout, keep_all=False)
    a, b = kept.forward(x), packed.forward(x)
    torch.cuda.synchronize()
    say(f"arena bytes kept {kept.memory()[0]} packed {packed.memory()[0]}")
    assert packed.memory()[0] < kept.memory()[0]
    assert torch.equal(a, b)
    kept.close()
    packed.close()


def test_graph_replays_equal_eager():
    import torch
    layers = nets.filters(_with_channels(MINI, 8), "HWCN", seed=7)
    net = mg3m.Net(layers, (4, 8, 19, 17), "HWCN")
    x = to_dev(make((4, 8, 19, 17, 1, 1, 1, 1, 0), 972, "HWCN")[0])
    eager = net.forward(x)
    torch.cuda.synchronize()
    s = torch.cuda.Stream()
    out = torch.empty_like(eager)
    with torch.cuda.stream(s):
        for rep in range(3):
            out.fill_(float("nan"))
            net.forward(x, out=out, graph=True, stream=s)
            s.synchronize()
            assert torch.equal(out, eager), f"replay {rep}"
            other = net.forward(x)                         # eager work between replays
            s.synchronize()
            assert torch.equal(other, eager)
        out2 = torch.empty_like(eager)                     # new output: captured again
        net.forward(x, out=out2, graph=True, stream=s)
        s.synchronize()
    assert torch.equal(out2, eager)
    with pytest.raises(mg3m.Mg3mError):
        net.forward(x, out=out, graph=True, stream=0)       # default stream cannot be captured
    net.close()


@pytest.mark.parametrize("name,N", [("vgg16", 2), ("alexnet", 4), ("resnet50", 2)])
def test_real_network_every_layer_sampled(name, N):
    import torch
    layers = nets.filters(nets.NETS[name](), "HWCN", seed=11)
    shape = (N, 3, 224, 224)
    net = mg3m.Net(layers, shape, "HWCN", keep_all=True)
    x = make((N, 3, 224, 224, 1, 1, 1, 1, 0), 980, "HWCN")[0]
    y = net.forward(to_dev(x))
    torch.cuda.synchronize()
    say(f"{name} N={N}: {len(layers)} layers, output {tuple(y.shape)}, arena {net.memory()[0] >> 20} MiB")
    assert torch.isfinite(y).all().item()
    worst = _check_chain(net, layers, x, _host(y), "HWCN", sample=2048, seed=12)
    say(f"  worst ratio to the bound {worst:.3g}")
    net.close()
