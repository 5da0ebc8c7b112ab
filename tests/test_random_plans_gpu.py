"""Seeded random shapes (ragged in every GEMM dimension, odd channel counts,
16 and 48 output channels, strides and pads up to the filter size) in both
layouts, half of them with a random forced tile and split or tail, against
the fp64 oracle element by element."""
import numpy as np
import pytest

import oracle
from tests.gpu_util import RTOL, make, run_gpu, say

pytestmark = pytest.mark.gpu

TILES = ["128x128", "64x256", "256x64", "64x128", "128x64", "64x64", "32x128", "32x64", "128x32", "64x32",
         "256x128", "128x256", "128x128,kt=32", "16x64", "64x64,kt=32"]


def _cases(seed, n):
    rng = np.random.Generator(np.random.PCG64(seed))
    out = []
    while len(out) < n:
        N = int(rng.choice([1, 2, 3, 4, 8, 12]))
        C = int(rng.choice([1, 3, 5, 16, 17, 32, 48, 64]))
        K = int(rng.choice([1, 4, 16, 20, 32, 48, 64, 80, 96]))
        H, W = (int(v) for v in rng.integers(1, 20, 2))
        R, S = int(rng.choice([1, 2, 3, 5])), int(rng.choice([1, 3, 5]))
        st, pd = int(rng.choice([1, 1, 2, 3])), int(rng.choice([0, 1, 2]))
        if H + 2 * pd < R or W + 2 * pd < S:
            continue
        layout = str(rng.choice(["HWCN", "NCHW"]))
        plan = None
        if rng.random() < 0.5:
            sched = str(rng.choice(["split", "tail", "none"]))
            plan = f"tile={rng.choice(TILES)}" + ("" if sched == "none" else f",{sched}={int(rng.integers(2, 9))}")
        out.append(((N, C, H, W, K, R, S, st, pd), layout, plan))
    return out


def test_random_shapes_and_plans():
    failures = []
    for i, (shape, layout, plan) in enumerate(_cases(2307, 400)):
        x, w, st, pd = make(shape, 9000 + i, layout)
        acc, mag = oracle.conv2d(x, w, st, pd, layout)
        try:
            y = run_gpu(x, w, st, pd, layout, plan=plan)
        except RuntimeError as e:
            if "MG3M_ERR_PLAN" in str(e):      # e.g. a tail override on a shape with no left-over tiles
                continue
            raise
        ok, worst, nfail, _ = oracle.check(y, acc, mag, RTOL)
        if not ok:
            failures.append((shape, layout, plan, worst, nfail))
            say(f"random case {i}: {shape} {layout} {plan}: {nfail} outputs outside tolerance")
    assert not failures, failures


def _schedule_cases(seed, n):
    """Random shapes with a random schedule each: persistent tiles, stream-K
    or split tails, whole tiles, the one-tap loaders staged through VGPRs
    (dma=0), and NCHW calls forced to run as HWCN or natively."""
    rng = np.random.Generator(np.random.PCG64(seed))
    out = []
    while len(out) < n:
        N = int(rng.choice([1, 4, 8, 12, 16]))
        C = int(rng.choice([3, 16, 32, 48, 64]))
        K = int(rng.choice([4, 16, 20, 64, 96, 132]))
        H, W = (int(v) for v in rng.integers(3, 24, 2))
        R = S = int(rng.choice([1, 3, 5]))
        st, pd = int(rng.choice([1, 1, 2])), int(rng.choice([0, 1, 2]))
        if H + 2 * pd < R or W + 2 * pd < S:
            continue
        layout = str(rng.choice(["HWCN", "NCHW"]))
        parts = [f"tile={rng.choice([t for t in TILES if t != '16x64'])}"]
        sched = str(rng.choice(["persist", "sk", "split", "tail", "none"]))
        if sched == "persist":
            parts.append(f"persist={int(rng.integers(1, 5))}")
        elif sched == "sk":
            parts.append(f"sk={int(rng.integers(2, 40))}")
        elif sched != "none":
            parts.append(f"{sched}={int(rng.integers(2, 9))}")
        if rng.random() < 0.3:
            parts.append("dma=0")
        if layout == "NCHW":
            parts.append(str(rng.choice(["via=hwcn", "via=none"])))
        out.append(((N, C, H, W, K, R, S, st, pd), layout, ",".join(parts)))
    return out


def test_random_shapes_and_schedules_exact():
    """Small-integer data, so every schedule must reproduce the exact sum bit
    for bit; plans that do not apply to a shape are skipped."""
    ran, failures = 0, []
    for i, (shape, layout, plan) in enumerate(_schedule_cases(4941, 300)):
        x, w, st, pd = make(shape, 12000 + i, layout, dist="int")
        acc, _ = oracle.conv2d(x, w, st, pd, layout)
        try:
            y = run_gpu(x, w, st, pd, layout, plan=plan)
        except RuntimeError as e:
            if "MG3M_ERR_PLAN" in str(e):
                continue
            raise
        ran += 1
        if not np.array_equal(y, acc.astype(np.float32)):
            failures.append((shape, layout, plan))
            say(f"schedule case {i}: {shape} {layout} {plan}: not bit-exact")
    say(f"{ran} of 300 schedule cases applied")
    assert ran >= 150, ran
    assert not failures, failures
