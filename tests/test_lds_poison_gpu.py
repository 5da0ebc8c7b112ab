"""Barrier check on the debug build that poisons every consumed LDS stage
with NaN (python -m paper_2307_04941_amd.build --lds-poison): at the start of
each stage the buffer the previous stage read is overwritten with NaN behind
a barrier before it is staged again, so a read that a missing barrier lets
through shows up as NaN in y.  Small-integer data: every output must still
equal the oracle's exact sum.  Skipped when the debug library is not built."""
import os

import numpy as np
import pytest

import oracle
from paper_2307_04941_amd import build, mg3m
from tests.gpu_util import make, run_gpu, say

pytestmark = pytest.mark.gpu

CASES = [
    ((4, 64, 13, 11, 68, 3, 3, 1, 1), "HWCN", None, False),                      # the selector's plan
    ((16, 64, 28, 28, 128, 3, 3, 1, 1), "HWCN", "tile=128x128,split=1", False),  # whole tiles, loads into LDS
    ((4, 64, 13, 11, 68, 3, 3, 1, 1), "HWCN", "tile=128x128,dma=0", False),      # register-staged
    ((4, 64, 13, 11, 68, 3, 3, 1, 1), "HWCN", "tile=128x128,sk=7", False),       # stream-K pieces
    ((4, 64, 13, 11, 68, 3, 3, 1, 1), "HWCN", "tile=64x64,kt=32,split=3", False),
    ((32, 3, 64, 64, 64, 3, 3, 1, 1), "HWCN", "tile=64x256,persist=1", False),   # persistent, vec-N
    ((4, 64, 13, 11, 68, 3, 3, 1, 1), "HWCN", "tile=128x128,persist=1", False),  # persistent, one-tap into LDS
    ((4, 64, 13, 11, 68, 3, 3, 1, 1), "HWCN", "tile=128x128,persist=1,dma=0", False),  # persistent, staged
    ((8, 64, 9, 7, 68, 1, 1, 1, 0), "HWCN", "tile=64x64,kt=32,persist=1", False),  # persistent, 2 stages/tile
    ((8, 16, 14, 14, 16, 3, 3, 1, 1), "HWCN", "tile=16x64", False),              # 16x16x4 MFMAs
    ((3, 32, 10, 9, 40, 3, 3, 1, 1), "NCHW", "tile=64x64,split=3,via=none", False),   # NCHW tap-major
    ((2, 6, 11, 9, 37, 3, 3, 1, 1), "NCHW", "tile=128x128,via=none", False),          # NCHW element-wise
    ((4, 64, 13, 11, 68, 3, 3, 1, 1), "NCHW", "tile=128x128,sk=7,via=hwcn", False),   # NCHW run as HWCN
    ((4, 64, 13, 11, 68, 3, 3, 1, 1), "HWCN", "tile=128x128,split=3", True),     # fp64 accumulation
]


@pytest.fixture(scope="module")
def poisoned_library():
    if not os.path.exists(build.LIB_LDS_POISON):
        pytest.skip("debug library not built (python -m paper_2307_04941_amd.build --lds-poison)")
    saved = mg3m._lib
    mg3m._lib = None
    try:
        yield mg3m.load_library(build.LIB_LDS_POISON)
    finally:
        mg3m._lib = saved


@pytest.mark.parametrize("case", range(len(CASES)))
def test_poisoned_stages_stay_exact(poisoned_library, case):
    shape, layout, plan, acc64 = CASES[case]
    say(f"lds poison {layout} {shape} {plan} acc64={acc64}")
    x, w, st, pd = make(shape, 990 + case, layout, dist="int")
    acc, _ = oracle.conv2d(x, w, st, pd, layout)
    y = run_gpu(x, w, st, pd, layout, plan=plan, acc64=acc64)
    assert not np.isnan(y).any(), "a poisoned LDS stage reached the output"
    assert np.array_equal(y, acc.astype(np.float32)), f"{shape} {plan}"
