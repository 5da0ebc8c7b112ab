"""Strength of the oracle's pins: plant plausible mistakes into copies of the
oracle's C source (on the CPU, in a temporary directory), and check that the
independent references used by tests/test_oracle.py reject every mutant.
The real oracle must pass the same checks."""
import ctypes
import os
import subprocess

import numpy as np
import pytest
import torch

import workloads
from tests.ref_im2col import im2col_conv_nchw

SRC = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "oracle", "direct_conv.c")

MUTANTS = {
    "filter_flip": ("flt_at(wt, p, oc, ic, fh, fw)", "flt_at(wt, p, oc, ic, p->r - 1 - fh, p->s - 1 - fw)"),
    "pad_sign": ("fh - p->pad_h", "fh + p->pad_h"),
    "stride_w_dropped": ("ow * p->std_w", "ow * p->std_h"),
    "dropped_channel": ("for (int ic = 0; ic < p->c; ++ic)", "for (int ic = 0; ic + 1 < p->c; ++ic)"),
    "transposed_filter_nchw": ("(((int64_t)oc * p->c + c) * p->r + fh)", "(((int64_t)(c % p->k) * p->c + (oc % p->c)) * p->r + fh)"),
    "transposed_filter_hwcn": ("* p->c + c) * p->k + oc;", "* p->c + (oc % p->c)) * p->k + (c % p->k);"),
    "last_row_dropped": ("ih >= p->h", "ih >= p->h - 1"),
    "mag_signed": ("mag += fabs(prod);", "mag += prod;"),
    "ceil_out_size": ("*out_h = eh / std_h + 1;", "*out_h = (eh + std_h - 1) / std_h + 1;"),
    "hwcn_bc_swapped": ("* p->c + c) * p->n + b;", "* p->n + (b % p->n)) * p->c + c;"),
    "wrong_fw_index": ("int iw = ow * p->std_w + fw - p->pad_w;", "int iw = ow * p->std_w + fh % p->s - p->pad_w;"),
}


def _build(tmp, name, src_text):
    c = os.path.join(tmp, f"{name}.c")
    so = os.path.join(tmp, f"lib{name}.so")
    with open(c, "w") as f:
        f.write(src_text)
    subprocess.run(["gcc", "-O1", "-fPIC", "-shared", "-std=c11", "-o", so, c, "-lm"], check=True)
    lib = ctypes.CDLL(so)
    i, p = ctypes.c_int, ctypes.c_void_p
    lib.oracle_conv2d_f64.argtypes = [p, p, p, p] + [i] * 12
    lib.oracle_out_dims.argtypes = [i] * 8 + [ctypes.POINTER(i)] * 2
    return lib


def _run(lib, x, w, st, pd, layout):
    """x, w logical NCHW / KCRS; returns (acc, mag) in logical NCHW or None."""
    N, C, H, W = x.shape
    K, _, R, S = w.shape
    ho, wo = ctypes.c_int(), ctypes.c_int()
    if lib.oracle_out_dims(H, W, R, S, st[0], st[1], pd[0], pd[1], ctypes.byref(ho), ctypes.byref(wo)):
        return None
    xl, wl = workloads.to_layout(x, w, layout)
    shape = (ho.value, wo.value, K, N) if layout == "HWCN" else (N, K, ho.value, wo.value)
    acc, mag = np.empty(shape), np.empty(shape)
    lay = 0 if layout == "HWCN" else 1
    rc = lib.oracle_conv2d_f64(xl.ctypes.data, wl.ctypes.data, acc.ctypes.data, mag.ctypes.data,
                               N, C, H, W, K, R, S, st[0], st[1], pd[0], pd[1], lay)
    if rc:
        return None
    if layout == "HWCN":
        acc, mag = workloads.hwcn_to_nchw(acc), workloads.hwcn_to_nchw(mag)
    return acc, mag


CASES = [  # N, C, H, W, K, R, S, stride(h,w), pad(h,w)
    (2, 3, 7, 6, 4, 3, 2, (2, 1), (2, 1)),
    (1, 2, 5, 8, 3, 3, 3, (1, 2), (1, 1)),
    (3, 4, 6, 5, 2, 2, 3, (1, 1), (0, 2)),
    (2, 3, 9, 7, 2, 5, 3, (3, 2), (2, 1)),
]


def _passes(lib):
    """True iff `lib` agrees with every independent reference on all cases."""
    for i, (N, C, H, W, K, R, S, st, pd) in enumerate(CASES):
        x = workloads.uniform((N, C, H, W), 4000 + i)
        w = workloads.uniform((K, C, R, S), 5000 + i)
        ref = im2col_conv_nchw(x.astype(np.float64), w.astype(np.float64), st, pd)
        tref = torch.nn.functional.conv2d(torch.from_numpy(x).double(), torch.from_numpy(w).double(),
                                          stride=st, padding=pd).numpy()
        mref = im2col_conv_nchw(np.abs(x).astype(np.float64), np.abs(w).astype(np.float64), st, pd)
        for layout in ("NCHW", "HWCN"):
            out = _run(lib, x, w, st, pd, layout)
            if out is None:
                return False
            acc, mag = out
            if acc.shape != ref.shape:
                return False
            tol = 1e-12 * mref + 1e-300
            if not (np.all(np.abs(acc - ref) <= tol) and np.all(np.abs(acc - tref) <= tol)
                    and np.all(np.abs(mag - mref) <= tol)):
                return False
    return True


def test_real_oracle_passes(tmp_path):
    with open(SRC) as f:
        lib = _build(str(tmp_path), "real", f.read())
    assert _passes(lib)


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_rejected(tmp_path, name):
    with open(SRC) as f:
        text = f.read()
    old, new = MUTANTS[name]
    assert text.count(old) >= 1, f"mutation site for {name} not found"
    lib = _build(str(tmp_path), name, text.replace(old, new))
    assert not _passes(lib), f"pins failed to reject mutant {name}"
