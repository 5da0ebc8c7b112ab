"""Build libmg3m.so (the HIP kernels, the planner and the C ABI) for gfx950.

    python -m paper_2307_04941_amd.build

Compiles in-tree with hipcc; the shared library lands next to this file.
"""
from __future__ import annotations

import concurrent.futures
import os
import subprocess
import sys
import tempfile

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libmg3m.so")
SOURCES = ["conv_hwcn_vecn_tap.hip", "conv_hwcn_vecn.hip", "conv_hwcn_vecc.hip", "conv_hwcn_veca.hip", "conv_hwcn_scalar.hip",
           "conv_nchw.hip", "conv_acc64_hwcn_tap.hip", "conv_acc64_hwcn.hip", "conv_acc64_nchw.hip",
           "conv_launch.hip", "plan.cpp", "abi.cpp"]

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"
# Packed fp32 instructions are switched off for all device code.
COMMON = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
          "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
          "-Wall", "-Wno-unused-result", f"-I{INCLUDE}", f"-I{CSRC}"]


# The fp64-accumulating kernels keep their accumulators in VGPRs: left to
# choose, the compiler carries them across the main loop in VGPRs and copies
# them into AGPRs around every stage's MFMAs.
PER_SOURCE = {s: ["-mllvm", "-amdgpu-mfma-vgpr-form=1"] for s in SOURCES if s.startswith("conv_acc64_")}


def _compile(src: str, obj: str, extra=()):
    cmd = [HIPCC, *COMMON, *PER_SOURCE.get(src, []), *extra, "-c", os.path.join(CSRC, src), "-o", obj]
    p = subprocess.run(cmd, capture_output=True, text=True)
    if p.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{' '.join(cmd)}\n{p.stdout}\n{p.stderr}")
    return obj


def build(verbose: bool = False, extra=()) -> str:
    """Compile every source and link libmg3m.so; returns its path."""
    with tempfile.TemporaryDirectory(prefix="mg3m_build_") as tmp:
        objs = [os.path.join(tmp, s + ".o") for s in SOURCES]
        with concurrent.futures.ThreadPoolExecutor(len(SOURCES)) as ex:
            list(ex.map(lambda so: _compile(so[0], so[1], extra), zip(SOURCES, objs)))
        out_tmp = LIB + ".tmp"
        cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", out_tmp, *objs]
        p = subprocess.run(cmd, capture_output=True, text=True)
        if p.returncode != 0:
            raise RuntimeError(f"link failed:\n{' '.join(cmd)}\n{p.stdout}\n{p.stderr}")
        os.replace(out_tmp, LIB)
    if verbose:
        print(f"built {LIB}")
    return LIB


if __name__ == "__main__":
    build(verbose=True, extra=sys.argv[1:])
