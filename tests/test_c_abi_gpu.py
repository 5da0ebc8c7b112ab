"""The C ABI called from plain C: tests/c_abi_gpu.c, built with gcc against
include/mg3m.h and linked with libmg3m.so and ROCm's HIP runtime (no Python
binding, no torch), run as its own process.  On small-integer data it checks
the plain call on two streams, a forced split plan with a caller workspace
and the entry point that allocates nothing, each bit for bit against Eq. 1
summed in integers, and that rejected calls write nothing."""
import os
import subprocess

import pytest

from paper_2307_04941_amd import build

pytestmark = pytest.mark.gpu


def test_c_program_through_the_abi():
    if not os.path.exists(build.C_ABI_TEST):
        pytest.skip("tests/c_abi_gpu.c not built (paper_2307_04941_amd.build.build_c_abi_test)")
    out = subprocess.run([build.C_ABI_TEST], capture_output=True, text=True, timeout=120)
    print(out.stdout, out.stderr)
    assert out.returncode == 0 and "c abi ok" in out.stdout, out.stderr
