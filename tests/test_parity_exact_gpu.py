"""Exact GPU parity at every benchmark-configuration layer, at full size.

Eq. 1 (Sec. 2.1) on small-integer data (x, w drawn from {-2, ..., 2}) has an
exact integer result: every product and every partial sum is an integer of
magnitude at most 4 * Kg <= 18432 < 2^24, so fp32 represents each of them
exactly and any summation order, tiling or split of the reduction gives the
same fp32 value.  The GPU output must therefore equal the oracle's exact sum
value for value (signed zeros compare equal), which separates indexing
mistakes from rounding.

For every layer of the five benchmark configurations (the single layer, the
scene sweep, VGG-16, ResNet-50, AlexNet + inception), in the plan the
selector picks, in both layouts: every output whose receptive field meets
the padding (all images and output channels of every border pixel), every
output of the first and last output pixels, and 65536 seeded random outputs.
Both layouts are generated from the same seeds, so they hold the same logical
tensors: the oracle evaluates each logical output once and both results are
compared with it."""
import time

import numpy as np
import pytest

import oracle
import workloads
from paper_2307_04941_amd import mg3m
from tests.gpu_util import say, to_dev

pytestmark = pytest.mark.gpu

LAYERS = [(wl, i) for wl in workloads.CONFIG_WORKLOADS for i in range(len(workloads.workload(wl)))]
N_RANDOM = 65536


def _edge_positions(n_out, n_in, r, s, p):
    """Output rows (or columns) whose window reaches past the input."""
    return [o for o in range(n_out) if o * s - p < 0 or o * s - p + r - 1 >= n_in]


@pytest.mark.parametrize("wl,index", LAYERS, ids=[f"{wl}-{i}" for wl, i in LAYERS])
def test_layer_exact_both_layouts(wl, index):
    import torch
    L, xh, wh = workloads.layer_tensors(wl, index, "HWCN", dist="int")
    _, xn, wn = workloads.layer_tensors(wl, index, "NCHW", dist="int")
    st, pd = L.stride, L.pad
    Ho, Wo = mg3m.conv2d_out_dims(L.H, L.W, L.R, L.S, st, pd)
    K, N = L.K, L.N
    rows = _edge_positions(Ho, L.H, L.R, st, pd)
    cols = _edge_positions(Wo, L.W, L.S, st, pd)
    pix = {oh * Wo + ow for oh in rows for ow in range(Wo)} | {oh * Wo + ow for oh in range(Ho) for ow in cols}
    pix |= {0, Ho * Wo - 1}
    kn = K * N
    rng = np.random.Generator(np.random.PCG64(20231100 + 97 * index + len(wl)))
    border = (np.fromiter(sorted(pix), np.int64)[:, None] * kn + np.arange(kn, dtype=np.int64)[None, :]).ravel()
    idx = np.unique(np.concatenate([border, rng.integers(0, Ho * Wo * kn, N_RANDOM)]))
    # logical (pixel, channel, image) of each HWCN flat index, and its NCHW flat index
    p_, rem = np.divmod(idx, kn)
    k_, b_ = np.divmod(rem, N)
    idx_nchw = (b_ * K + k_) * (Ho * Wo) + p_

    t0 = time.perf_counter()
    acc, _ = oracle.conv2d_points(xh, wh, idx, st, pd, "HWCN")
    t_or = time.perf_counter() - t0
    assert np.all(np.abs(acc) < 2.0**24), "small-integer data must keep every sum exact in fp32"
    exact = acc.astype(np.float32)
    say(f"exact {wl}/{L.name}: {len(pix)} border/corner pixels, {idx.size} outputs, oracle {t_or:.1f} s")

    for layout, x, w, sel in (("HWCN", xh, wh, idx), ("NCHW", xn, wn, idx_nchw)):
        say(f"  {layout}: " + mg3m.conv2d_fwd_f32_plan_string(L.N, L.C, L.H, L.W, L.K, L.R, L.S, st, pd, layout))
        y = mg3m.conv2d_fwd(to_dev(x), to_dev(w), st, pd, layout)
        torch.cuda.synchronize()
        got = y.view(-1)[torch.from_numpy(sel).cuda()].cpu().numpy()
        del y
        bad = got != exact
        if bad.any():
            i = int(np.argmax(bad))
            pytest.fail(f"{layout}: {int(bad.sum())} of {idx.size} outputs differ from the exact sum; first at "
                        f"pixel {p_[i]} channel {k_[i]} image {b_[i]}: gpu {got[i]!r} exact {exact[i]!r}")
    torch.cuda.empty_cache()
