"""Helpers for the GPU parity tests: run the HIP path through the C ABI on
seeded inputs and compare with the fp64 oracle element by element."""
import sys

import numpy as np

import oracle
import workloads
from paper_2307_04941_amd import mg3m

RTOL = 1e-5          # |gpu - oracle| <= 1e-5 * sum |x*w|, per output element


def say(*args):
    print(*args, flush=True)
    sys.stdout.flush()


def to_dev(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def run_gpu(x, w, stride, pad, layout, plan=None, misalign=0, acc64=False):
    """Convolution on the GPU through the C ABI; returns y as numpy.
    misalign: shift every device buffer by this many floats (4-byte aligned,
    not 16-byte aligned) to exercise the element-wise loaders.  acc64: use
    the fp64-accumulating entry point."""
    import torch
    if misalign:
        xb = torch.empty(x.size + misalign, dtype=torch.float32, device="cuda")
        wb = torch.empty(w.size + misalign, dtype=torch.float32, device="cuda")
        xb[misalign:].copy_(torch.from_numpy(x.reshape(-1)))
        wb[misalign:].copy_(torch.from_numpy(w.reshape(-1)))
        xd, wd = xb[misalign:].view(x.shape), wb[misalign:].view(w.shape)
    else:
        xd, wd = to_dev(x), to_dev(w)
    N, C, H, W, K, R, S = mg3m.dims_of(x, w, layout)
    (sh, sw), (ph, pw) = mg3m._pair(stride), mg3m._pair(pad)
    Ho, Wo = mg3m.conv2d_out_dims_hw(H, W, R, S, sh, sw, ph, pw)
    shape = (Ho, Wo, K, N) if layout == "HWCN" else (N, K, Ho, Wo)
    n_out = int(np.prod(shape))
    yb = torch.full((n_out + misalign,), float("nan"), dtype=torch.float32, device="cuda")
    y = yb[misalign:].view(shape)
    mg3m.conv2d_fwd(xd, wd, stride, pad, layout, plan=plan, out=y, acc64=acc64)
    torch.cuda.synchronize()
    return y.cpu().numpy()


def assert_parity(y, acc, mag, what=""):
    ok, worst, nfail, first = oracle.check(y, acc, mag, RTOL)
    assert ok, (f"{what}: {nfail} of {acc.size} outputs outside 1e-5*sum|x*w| "
                f"(worst ratio {worst:.3g}, first flat index {first}: "
                f"gpu {np.asarray(y).reshape(-1)[first]!r} oracle {np.asarray(acc).reshape(-1)[first]!r})")
    return worst


def make(shape, seed, layout, dist=None):
    """shape = (N, C, H, W, K, R, S, stride, pad); stride and pad may be
    (vertical, horizontal) pairs."""
    N, C, H, W, K, R, S, st, pd = shape
    L = workloads.Layer("t", N, C, H, W, K, R, S)
    x, w = workloads.make_tensors(L, seed, seed + 1, layout, dist)
    return x, w, st, pd


def acc64_tolerance(acc, mag, Kg):
    """Bound for the fp64-accumulating path: one rounding of the fp64 sum to
    fp32 (2^-24 relative, round to nearest) plus the fp64 summation error of
    the kernel and of the oracle (each at most Kg * 2^-53 * sum|x*w|, with
    margin)."""
    return np.ldexp(np.abs(acc), -24) * (1 + 2.0**-20) + 4.0 * Kg * 2.0**-53 * mag


def assert_parity_acc64(y, acc, mag, Kg, what=""):
    y = np.asarray(y, np.float64).reshape(-1)
    acc = np.asarray(acc, np.float64).reshape(-1)
    mag = np.asarray(mag, np.float64).reshape(-1)
    err = np.abs(y - acc)
    tol = acc64_tolerance(acc, mag, Kg)
    bad = ~(err <= tol)
    if bad.any():
        i = int(np.argmax(bad))
        raise AssertionError(f"{what}: {int(bad.sum())} of {acc.size} outputs outside one fp32 rounding "
                             f"of the fp64 sum; first flat index {i}: gpu {y[i]!r} oracle {acc[i]!r} "
                             f"tol {tol[i]:.3g}")
    ratio = np.where(tol > 0, err / np.where(tol > 0, tol, 1), 0)
    return float(ratio.max()) if ratio.size else 0.0
