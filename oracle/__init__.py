"""TEST INFRASTRUCTURE ONLY: the fp64 CPU oracle for the forward convolution.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The product (``paper_2307_04941_amd``)
never imports it, and it imports nothing from the product.

The convolution's arithmetic lives in ``direct_conv.c`` (plain C, seven
nested loops of Eq. 1 of the MG3MConv paper, Sec. 2.1, accumulated in fp64);
this module builds that file with gcc and marshals numpy arrays into it.
``maxpool2d`` -- the pooling between the convolution blocks of the networks
the paper runs (Sec. 5.2) -- is written here in numpy, from its definition.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

HWCN = 0
NCHW = 1
LAYOUTS = {"HWCN": HWCN, "NCHW": NCHW}

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "direct_conv.c")
_LIB = os.path.join(_HERE, "libmg3m_oracle.so")
_lib = None


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (OpenMP over output elements only; the
    summation order inside one output is Eq. 1's).  No -ffast-math, so gcc
    keeps the order of every fp64 addition."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        subprocess.run(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c11",
                        "-Wall", "-Wextra", "-o", tmp, _SRC, "-lm"], check=True)
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=True)
        lib = ctypes.CDLL(_LIB)
        i = ctypes.c_int
        p = ctypes.c_void_p
        lib.oracle_out_dims.argtypes = [i, i, i, i, i, i, i, i,
                                        ctypes.POINTER(i), ctypes.POINTER(i)]
        lib.oracle_out_dims.restype = i
        lib.oracle_conv2d_f64.argtypes = [p, p, p, p] + [i] * 12
        lib.oracle_conv2d_f64.restype = i
        lib.oracle_conv2d_points_f64.argtypes = [p, p, p, ctypes.c_int64, p, p] + [i] * 12
        lib.oracle_conv2d_points_f64.restype = i
        _lib = lib
    return _lib


def _pair(v):
    if isinstance(v, (tuple, list)):
        return int(v[0]), int(v[1])
    return int(v), int(v)


def out_dims(H, W, R, S, stride=1, pad=0):
    """(Ho, Wo) by the floor formula; raises ValueError for an empty output."""
    sh, sw = _pair(stride)
    ph, pw = _pair(pad)
    ho, wo = ctypes.c_int(), ctypes.c_int()
    if _load().oracle_out_dims(H, W, R, S, sh, sw, ph, pw, ctypes.byref(ho), ctypes.byref(wo)):
        raise ValueError("invalid convolution shape")
    return ho.value, wo.value


def _dims(x, w, layout):
    if layout == HWCN:
        H, W, C, N = x.shape
        R, S, C2, K = w.shape
    else:
        N, C, H, W = x.shape
        K, C2, R, S = w.shape
    if C != C2:
        raise ValueError("channel mismatch")
    return N, C, H, W, K, R, S


def _out_shape(N, K, Ho, Wo, layout):
    return (Ho, Wo, K, N) if layout == HWCN else (N, K, Ho, Wo)


def conv2d(x: np.ndarray, w: np.ndarray, stride=1, pad=0, layout="NCHW"):
    """Every output of Eq. 1 in fp64.  x, w are float32 arrays in ``layout``
    (NCHW: x[N,C,H,W], w[K,C,R,S]; HWCN: x[H,W,C,N], w[R,S,C,K]).
    Returns (acc, mag), float64 arrays in the layout's output order."""
    lay = LAYOUTS[layout] if isinstance(layout, str) else int(layout)
    x = np.ascontiguousarray(x, dtype=np.float32)
    w = np.ascontiguousarray(w, dtype=np.float32)
    N, C, H, W, K, R, S = _dims(x, w, lay)
    sh, sw = _pair(stride)
    ph, pw = _pair(pad)
    Ho, Wo = out_dims(H, W, R, S, (sh, sw), (ph, pw))
    shape = _out_shape(N, K, Ho, Wo, lay)
    acc = np.empty(shape, np.float64)
    mag = np.empty(shape, np.float64)
    rc = _load().oracle_conv2d_f64(x.ctypes.data, w.ctypes.data, acc.ctypes.data, mag.ctypes.data,
                                   N, C, H, W, K, R, S, sh, sw, ph, pw, lay)
    if rc:
        raise ValueError("oracle rejected the shape")
    return acc, mag


def conv2d_points(x: np.ndarray, w: np.ndarray, idx, stride=1, pad=0, layout="NCHW"):
    """Outputs at the given flat indices of the layout's output array, in fp64.
    Returns (acc, mag), each of shape (len(idx),)."""
    lay = LAYOUTS[layout] if isinstance(layout, str) else int(layout)
    x = np.ascontiguousarray(x, dtype=np.float32)
    w = np.ascontiguousarray(w, dtype=np.float32)
    idx = np.ascontiguousarray(idx, dtype=np.int64)
    N, C, H, W, K, R, S = _dims(x, w, lay)
    sh, sw = _pair(stride)
    ph, pw = _pair(pad)
    acc = np.empty(idx.shape[0], np.float64)
    mag = np.empty(idx.shape[0], np.float64)
    rc = _load().oracle_conv2d_points_f64(x.ctypes.data, w.ctypes.data, idx.ctypes.data,
                                          idx.shape[0], acc.ctypes.data, mag.ctypes.data,
                                          N, C, H, W, K, R, S, sh, sw, ph, pw, lay)
    if rc:
        raise ValueError("oracle rejected the shape or an index")
    return acc, mag


def check(y: np.ndarray, acc: np.ndarray, mag: np.ndarray, rtol: float = 1e-5):
    """Per-element parity test |y - acc| <= rtol * mag, in fp64.
    Returns (ok, worst_ratio, n_fail, first_fail_flat_index)."""
    y = np.asarray(y, dtype=np.float64).reshape(-1)
    acc = np.asarray(acc, dtype=np.float64).reshape(-1)
    mag = np.asarray(mag, dtype=np.float64).reshape(-1)
    err = np.abs(y - acc)
    bound = rtol * mag
    bad = ~(err <= bound)          # NaN in y counts as a failure
    with np.errstate(divide="ignore", invalid="ignore"):
        ratio = np.where(bound > 0, err / np.where(bound > 0, bound, 1.0),
                         np.where(err > 0, np.inf, 0.0))
    n_fail = int(bad.sum())
    first = int(np.argmax(bad)) if n_fail else -1
    worst = float(np.nanmax(ratio)) if ratio.size else 0.0
    if np.isnan(ratio).any():
        worst = float("inf")
    return n_fail == 0, worst, n_fail, first


def maxpool2d(x: np.ndarray, R, S=None, stride=None, pad=0, layout="NCHW"):
    """Max pooling from its definition: y[b,c,oh,ow] = max over the window taps
    (r, s) in [0,R) x [0,S) whose input position ih = oh*sh + r - ph,
    iw = ow*sw + s - pw lies inside the image (padded taps are skipped, never
    read as a value).  Output size by the same floor formula as the
    convolution.  A NaN in a window gives NaN.  stride defaults to the window.
    Returns a float32 array in ``layout`` (NCHW x[N,C,H,W] or HWCN x[H,W,C,N]).
    Parity unpinned by the paper, which prints no pooling example; pinned in
    tests by hand-computed values, brute force and scipy.ndimage."""
    lay = LAYOUTS[layout] if isinstance(layout, str) else int(layout)
    S = R if S is None else S
    sh, sw = _pair((R, S) if stride is None else stride)
    ph, pw = _pair(pad)
    x = np.asarray(x, dtype=np.float32)
    xn = x if lay == NCHW else np.transpose(x, (3, 2, 0, 1))        # -> [N, C, H, W]
    N, C, H, W = xn.shape
    Ho, Wo = (H + 2 * ph - R) // sh + 1, (W + 2 * pw - S) // sw + 1
    if Ho < 1 or Wo < 1:
        raise ValueError("empty pooling output")
    y = np.full((N, C, Ho, Wo), -np.inf, np.float32)
    oh, ow = np.arange(Ho), np.arange(Wo)
    for r in range(R):
        ih = oh * sh + r - ph
        rows = (ih >= 0) & (ih < H)
        for s in range(S):
            iw = ow * sw + s - pw
            cols = (iw >= 0) & (iw < W)
            if not rows.any() or not cols.any():
                continue
            tap = xn[:, :, ih[rows]][:, :, :, iw[cols]]
            cur = y[:, :, rows][:, :, :, cols]
            # NaN-propagating maximum
            new = np.where(np.isnan(tap) | (tap > cur), tap, cur)
            y[np.ix_(np.arange(N), np.arange(C), np.flatnonzero(rows), np.flatnonzero(cols))] = new
    return y if lay == NCHW else np.ascontiguousarray(np.transpose(y, (2, 3, 1, 0)))
