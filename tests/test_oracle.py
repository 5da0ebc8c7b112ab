"""Pins of the fp64 CPU oracle (Eq. 1, Sec. 2.1) to things other than itself:
brute force on tiny inputs, library routines, closed forms and invariants.
A plausible mistake in the oracle (flip, wrong pad sign, dropped channel,
transposed operand, swapped stride, wrong magnitude term) fails at least one
of these; tests/test_oracle_mutants.py checks that claim by planting such
mistakes into copies of the oracle source."""
import itertools
import json
import os

import numpy as np
import pytest
import scipy.signal
import torch

import oracle
import workloads
from tests.ref_im2col import im2col_conv_nchw

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rand(shape, seed):
    return workloads.uniform(shape, seed)


def _tiny_grid():
    rng = np.random.Generator(np.random.PCG64(7))
    cases = []
    for N, C, K in [(1, 1, 1), (2, 3, 2), (3, 5, 4), (1, 2, 4), (2, 1, 3)]:
        for H, W in [(1, 1), (2, 5), (5, 7), (7, 2), (5, 5)]:
            for R, S in [(1, 1), (2, 3), (3, 3), (5, 2), (3, 5)]:
                sh, sw = int(rng.integers(1, 4)), int(rng.integers(1, 4))
                ph, pw = int(rng.integers(0, 4)), int(rng.integers(0, 4))
                if H + 2 * ph < R or W + 2 * pw < S:
                    continue
                cases.append((N, C, H, W, K, R, S, sh, sw, ph, pw))
    return cases


def test_bruteforce_im2col_grid():
    """Whole oracle vs a separately written im2col + naive GEMM (fp64)."""
    cases = _tiny_grid()
    assert len(cases) > 80
    for i, (N, C, H, W, K, R, S, sh, sw, ph, pw) in enumerate(cases):
        x = _rand((N, C, H, W), 100 + i)
        w = _rand((K, C, R, S), 200 + i)
        acc, mag = oracle.conv2d(x, w, (sh, sw), (ph, pw), "NCHW")
        ref = im2col_conv_nchw(x.astype(np.float64), w.astype(np.float64), (sh, sw), (ph, pw))
        assert acc.shape == ref.shape, (acc.shape, ref.shape)
        assert np.all(np.abs(acc - ref) <= 1e-12 * mag + 1e-300), (N, C, H, W, K, R, S, sh, sw, ph, pw)


@pytest.mark.parametrize("layout", ["NCHW", "HWCN"])
def test_torch_conv2d_library(layout):
    """Library routine: torch.nn.functional.conv2d on the CPU in float64."""
    rng = np.random.Generator(np.random.PCG64(11))
    for i in range(25):
        N, C, K = (int(v) for v in rng.integers(1, 6, 3))
        H, W = (int(v) for v in rng.integers(3, 17, 2))
        R, S = (int(v) for v in rng.integers(1, 6, 2))
        sh, sw = (int(v) for v in rng.integers(1, 4, 2))
        ph, pw = (int(v) for v in rng.integers(0, 3, 2))
        if H + 2 * ph < R or W + 2 * pw < S:
            continue
        x = _rand((N, C, H, W), 300 + i)
        w = _rand((K, C, R, S), 400 + i)
        ref = torch.nn.functional.conv2d(torch.from_numpy(x).double(), torch.from_numpy(w).double(),
                                         stride=(sh, sw), padding=(ph, pw)).numpy()
        xl, wl = workloads.to_layout(x, w, layout)
        acc, mag = oracle.conv2d(xl, wl, (sh, sw), (ph, pw), layout)
        if layout == "HWCN":
            acc, mag = workloads.hwcn_to_nchw(acc), workloads.hwcn_to_nchw(mag)
        assert acc.shape == ref.shape
        assert np.all(np.abs(acc - ref) <= 1e-12 * mag + 1e-300)


def test_scipy_correlate2d_textbook():
    """Per-channel 2-D cross-correlation (scipy) summed over channels, then
    subsampled by the stride: the textbook reading of Eq. 1."""
    N, C, H, W, K, R, S = 2, 3, 11, 9, 2, 3, 4
    for st, pd in [(1, 0), (1, 1), (2, 1), (3, 2)]:
        x = _rand((N, C, H, W), 500 + st)
        w = _rand((K, C, R, S), 600 + pd)
        acc, mag = oracle.conv2d(x, w, st, pd, "NCHW")
        xp = np.pad(x.astype(np.float64), ((0, 0), (0, 0), (pd, pd), (pd, pd)))
        for b in range(N):
            for k in range(K):
                full = sum(scipy.signal.correlate2d(xp[b, c], w[k, c].astype(np.float64), mode="valid")
                           for c in range(C))
                ref = full[::st, ::st]
                assert ref.shape == acc[b, k].shape
                assert np.all(np.abs(acc[b, k] - ref) <= 1e-12 * mag[b, k] + 1e-300)


@pytest.mark.parametrize("R,S,pad", [(3, 3, 1), (5, 3, 2), (3, 3, 0), (1, 1, 0), (4, 2, 3)])
def test_delta_filter_shift(R, S, pad):
    """w[k,c,r,s] = [k==c][r==r0][s==s0] shifts the input by (r0-pad, s0-pad),
    zero outside; exact."""
    N, C, H, W = 2, 3, 6, 7
    x = _rand((N, C, H, W), 700 + R + S)
    for r0, s0 in itertools.product(range(R), range(S)):
        w = np.zeros((C, C, R, S), np.float32)
        for c in range(C):
            w[c, c, r0, s0] = 1.0
        acc, _ = oracle.conv2d(x, w, 1, pad, "NCHW")
        Ho, Wo = acc.shape[2:]
        ref = np.zeros_like(acc)
        for oh in range(Ho):
            for ow in range(Wo):
                ih, iw = oh + r0 - pad, ow + s0 - pad
                if 0 <= ih < H and 0 <= iw < W:
                    ref[:, :, oh, ow] = x[:, :, ih, iw]
        assert np.array_equal(acc, ref)


def test_linearity_in_x_and_w():
    N, C, H, W, K, R, S = 2, 4, 9, 8, 3, 3, 3
    # dyadic data (multiples of 2**-10) so that a*x1 + b*x2 is exact in fp32
    q = lambda v: (np.round(v * 1024) / 1024).astype(np.float32)
    x1, x2 = q(_rand((N, C, H, W), 801)), q(_rand((N, C, H, W), 802))
    w1, w2 = q(_rand((K, C, R, S), 803)), q(_rand((K, C, R, S), 804))
    a, b = 0.5, -2.0
    ax = (np.float32(a) * x1 + np.float32(b) * x2).astype(np.float32)
    y1, m1 = oracle.conv2d(x1, w1, 2, 1)
    y2, m2 = oracle.conv2d(x2, w1, 2, 1)
    yx, _ = oracle.conv2d(ax, w1, 2, 1)
    tol = 1e-12 * (abs(a) * m1 + abs(b) * m2) * 4
    assert np.all(np.abs(yx - (a * y1 + b * y2)) <= tol)
    aw = (np.float32(a) * w1 + np.float32(b) * w2).astype(np.float32)
    z2, n2 = oracle.conv2d(x1, w2, 2, 1)
    yw, _ = oracle.conv2d(x1, aw, 2, 1)
    tol = 1e-12 * (abs(a) * m1 + abs(b) * n2) * 4
    assert np.all(np.abs(yw - (a * y1 + b * z2)) <= tol)


def test_1x1_is_matmul():
    N, C, H, W, K = 3, 7, 5, 6, 4
    x = _rand((N, C, H, W), 901)
    w = _rand((K, C, 1, 1), 902)
    acc, mag = oracle.conv2d(x, w, 1, 0)
    ref = np.matmul(w.reshape(K, C).astype(np.float64),
                    x.astype(np.float64).reshape(N, C, H * W)).reshape(N, K, H, W)
    assert np.all(np.abs(acc - ref) <= 1e-12 * mag)


def test_ones_input_closed_form():
    """x == 1  =>  y[b,k,oh,ow] = sum of w[k,c,r,s] over taps inside the input."""
    N, C, H, W, K, R, S, st, pd = 2, 3, 7, 6, 2, 3, 5, 2, 2
    x = np.ones((N, C, H, W), np.float32)
    w = _rand((K, C, R, S), 1001)
    acc, mag = oracle.conv2d(x, w, st, pd)
    Ho, Wo = acc.shape[2:]
    for oh in range(Ho):
        for ow in range(Wo):
            rr = [r for r in range(R) if 0 <= oh * st + r - pd < H]
            ss = [s for s in range(S) if 0 <= ow * st + s - pd < W]
            ref = w[:, :, rr][:, :, :, ss].astype(np.float64).sum(axis=(1, 2, 3)) if rr and ss else np.zeros(K)
            for b in range(N):
                assert np.all(np.abs(acc[b, :, oh, ow] - ref) <= 1e-12 * mag[b, :, oh, ow] + 1e-300)


def test_ones_filter_box_sum():
    """w == 1  =>  y is the box sum of the zero-padded input (integral image)."""
    N, C, H, W, K, R, S, st, pd = 2, 3, 9, 8, 2, 3, 2, 1, 1
    x = _rand((N, C, H, W), 1101)
    w = np.ones((K, C, R, S), np.float32)
    acc, mag = oracle.conv2d(x, w, st, pd)
    xs = np.pad(x.astype(np.float64).sum(axis=1), ((0, 0), (pd, pd), (pd, pd)))
    ii = np.zeros((N, xs.shape[1] + 1, xs.shape[2] + 1))
    ii[:, 1:, 1:] = xs.cumsum(1).cumsum(2)
    Ho, Wo = acc.shape[2:]
    for oh in range(Ho):
        for ow in range(Wo):
            t, l = oh * st, ow * st
            box = ii[:, t + R, l + S] - ii[:, t, l + S] - ii[:, t + R, l] + ii[:, t, l]
            for k in range(K):
                assert np.all(np.abs(acc[:, k, oh, ow] - box) <= 1e-12 * mag[:, k, oh, ow] + 1e-12)


@pytest.mark.parametrize("st", [2, 3, 4])
def test_stride_is_subsampling(st):
    N, C, H, W, K, R, S, pd = 2, 3, 13, 11, 2, 3, 5, 2
    x = _rand((N, C, H, W), 1200 + st)
    w = _rand((K, C, R, S), 1300 + st)
    ys, _ = oracle.conv2d(x, w, st, pd)
    y1, _ = oracle.conv2d(x, w, 1, pd)
    assert np.array_equal(ys, y1[:, :, ::st, ::st])


@pytest.mark.parametrize("pd", [1, 2, 4])
def test_pad_is_explicit_zero_padding(pd):
    N, C, H, W, K, R, S = 2, 3, 7, 8, 2, 3, 3
    x = _rand((N, C, H, W), 1400 + pd)
    w = _rand((K, C, R, S), 1500 + pd)
    yp, mp = oracle.conv2d(x, w, 2, pd)
    xz = np.pad(x, ((0, 0), (0, 0), (pd, pd), (pd, pd)))
    y0, m0 = oracle.conv2d(xz, w, 2, 0)
    assert np.array_equal(yp, y0) and np.array_equal(mp, m0)


def test_channel_additivity():
    """Basis of split-K: splitting the input channels sums the partial outputs."""
    N, C, H, W, K, R, S = 2, 7, 8, 8, 3, 3, 3
    x = _rand((N, C, H, W), 1601)
    w = _rand((K, C, R, S), 1602)
    y, m = oracle.conv2d(x, w, 1, 1)
    c1 = 3
    ya, _ = oracle.conv2d(x[:, :c1], w[:, :c1], 1, 1)
    yb, _ = oracle.conv2d(x[:, c1:], w[:, c1:], 1, 1)
    assert np.all(np.abs(y - (ya + yb)) <= 1e-12 * m + 1e-300)


def test_batch_equivariance():
    N, C, H, W, K = 4, 3, 6, 5, 2
    x = _rand((N, C, H, W), 1701)
    w = _rand((K, C, 3, 3), 1702)
    y, _ = oracle.conv2d(x, w, 1, 1)
    perm = np.array([2, 0, 3, 1])
    yp, _ = oracle.conv2d(np.ascontiguousarray(x[perm]), w, 1, 1)
    assert np.array_equal(yp, y[perm])
    y1, _ = oracle.conv2d(np.ascontiguousarray(x[1:2]), w, 1, 1)
    assert np.array_equal(y1[0], y[1])


def test_layout_equivalence():
    N, C, H, W, K, R, S = 3, 4, 7, 9, 5, 3, 2
    x = _rand((N, C, H, W), 1801)
    w = _rand((K, C, R, S), 1802)
    a1, m1 = oracle.conv2d(x, w, (2, 1), (1, 0), "NCHW")
    xh, wh = workloads.to_layout(x, w, "HWCN")
    a2, m2 = oracle.conv2d(xh, wh, (2, 1), (1, 0), "HWCN")
    assert np.array_equal(a1, workloads.hwcn_to_nchw(a2))
    assert np.array_equal(m1, workloads.hwcn_to_nchw(m2))


def test_mag_is_conv_of_magnitudes():
    """mag = sum |x*w| = conv(|x|, |w|) exactly (same taps, same order)."""
    N, C, H, W, K, R, S = 2, 3, 8, 7, 4, 3, 3
    x = _rand((N, C, H, W), 1901)
    w = _rand((K, C, R, S), 1902)
    _, mag = oracle.conv2d(x, w, 2, 1)
    acc_abs, _ = oracle.conv2d(np.abs(x), np.abs(w), 2, 1)
    assert np.array_equal(mag, acc_abs)
    ref = im2col_conv_nchw(np.abs(x).astype(np.float64), np.abs(w).astype(np.float64), (2, 2), (1, 1))
    assert np.all(np.abs(mag - ref) <= 1e-12 * mag + 1e-300)


def test_small_integer_exact():
    """Integer data: the fp64 oracle equals exact int64 arithmetic."""
    N, C, H, W, K, R, S = 2, 5, 7, 6, 3, 3, 3
    x = workloads.small_int((N, C, H, W), 2001)
    w = workloads.small_int((K, C, R, S), 2002)
    acc, _ = oracle.conv2d(x, w, 1, 1)
    ref = im2col_conv_nchw(x.astype(np.int64), w.astype(np.int64), (1, 1), (1, 1), dtype=np.int64)
    assert np.array_equal(acc, ref.astype(np.float64))


@pytest.mark.parametrize("layout", ["NCHW", "HWCN"])
def test_points_match_full(layout):
    N, C, H, W, K, R, S = 3, 4, 9, 7, 5, 3, 3
    x = _rand((N, C, H, W), 2101)
    w = _rand((K, C, R, S), 2102)
    xl, wl = workloads.to_layout(x, w, layout)
    acc, mag = oracle.conv2d(xl, wl, 2, 1, layout)
    rng = np.random.Generator(np.random.PCG64(3))
    idx = rng.integers(0, acc.size, 200)
    pa, pm = oracle.conv2d_points(xl, wl, idx, 2, 1, layout)
    assert np.array_equal(pa, acc.reshape(-1)[idx])
    assert np.array_equal(pm, mag.reshape(-1)[idx])
    with pytest.raises(ValueError):
        oracle.conv2d_points(xl, wl, np.array([acc.size]), 2, 1, layout)


def test_output_sizes_golden():
    """Output sizes of every layer of the benchmark configurations against
    hand-computed values."""
    with open(os.path.join(GOLDEN, "output_sizes.json")) as f:
        gold = json.load(f)["sizes"]
    seen = 0
    for wl_name in workloads.CONFIG_WORKLOADS:
        for L in workloads.workload(wl_name):
            key = f"{wl_name}/{L.name}"
            ho, wo = oracle.out_dims(L.H, L.W, L.R, L.S, L.stride, L.pad)
            assert [ho, wo] == gold[key], key
            seen += 1
    assert seen == len(gold)


def test_output_sizes_of_sweep_layers_by_counting_windows():
    """The Sec. 5.1 sweep layers: output sizes against a count of the window
    positions that fit in the padded input (no floor formula)."""
    def count(size, pad, k, stride):
        n, start = 0, 0
        while start + k <= size + 2 * pad:
            n += 1
            start += stride
        return n
    for wl_name in workloads.SWEEP_WORKLOADS:
        for L in workloads.workload(wl_name):
            expect = (count(L.H, L.pad, L.R, L.stride), count(L.W, L.pad, L.S, L.stride))
            assert oracle.out_dims(L.H, L.W, L.R, L.S, L.stride, L.pad) == expect, L


def test_invalid_shapes_rejected():
    with pytest.raises(ValueError):
        oracle.out_dims(2, 2, 5, 5, 1, 0)
    with pytest.raises(ValueError):
        oracle.out_dims(4, 4, 3, 3, 0, 0)


def test_all_invalid_taps_give_exact_zero():
    """pad >= R: border outputs have no valid tap -> exactly 0 with mag 0."""
    x = _rand((1, 2, 3, 3), 2201)
    w = _rand((2, 2, 2, 2), 2202)
    acc, mag = oracle.conv2d(x, w, 1, 3)
    assert acc[0, :, 0, 0].tolist() == [0.0, 0.0] and mag[0, :, 0, 0].tolist() == [0.0, 0.0]
    ok, _, _, _ = oracle.check(acc.astype(np.float32), acc, mag)
    assert ok
    y = acc.copy()
    y[0, 0, 0, 0] = 1e-30          # zero tolerance where mag == 0
    ok, _, nf, first = oracle.check(y, acc, mag)
    assert not ok and nf == 1 and first == 0
