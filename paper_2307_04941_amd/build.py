"""Build libmg3m.so (the HIP kernels, the planner and the C ABI) for gfx950.

    python -m paper_2307_04941_amd.build                 # libmg3m.so
    python -m paper_2307_04941_amd.build --lds-poison    # debug/libmg3m_lds_poison.so

Compiles in-tree with hipcc; the shared library lands next to this file.
"""
from __future__ import annotations

import concurrent.futures
import hashlib
import json
import os
import subprocess
import sys
import tempfile

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libmg3m.so")
SOURCES = ["conv_hwcn_vecn_tap.hip", "conv_hwcn_vecn_tap_dma.hip", "conv_hwcn_vecn_tap_dma_fused.hip", "conv_hwcn_vecn.hip", "conv_hwcn_vecc.hip", "conv_hwcn_veca.hip", "conv_hwcn_scalar.hip",
           "conv_nchw.hip", "conv_acc64_hwcn_tap.hip", "conv_acc64_hwcn.hip", "conv_acc64_nchw.hip",
           "conv_hwcn_vecn_tap_fused.hip", "conv_hwcn_vecn_fused.hip", "conv_hwcn_other_fused.hip",
           "conv_nchw_fused.hip", "conv_nchw_tap.hip", "conv_nchw_tap_fused.hip", "conv_hwcn_persist.hip", "conv_hwcn_persist_fused.hip",
           "conv_launch.hip", "pool.hip", "layout.hip", "plan.cpp", "abi.cpp", "net.cpp", "noalloc.hip", "measure.hip"]

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"
# Packed fp32 instructions are switched off for all device code.
COMMON = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
          "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
          "-Wall", "-Wno-unused-result", f"-I{INCLUDE}", f"-I{CSRC}"]


# The fp64-accumulating kernels keep their accumulators in VGPRs: left to
# choose, the compiler carries them across the main loop in VGPRs and copies
# them into AGPRs around every stage's MFMAs.
# The persistent fp32 kernels likewise: their accumulators stay live across
# the loop over tiles, and in AGPRs the compiler copied all of them to VGPRs
# and back around every stage (180-216 registers instead of 117-155).
PER_SOURCE = {s: ["-mllvm", "-amdgpu-mfma-vgpr-form=1"] for s in SOURCES
              if s.startswith("conv_acc64_") or s.startswith("conv_hwcn_persist")}


def _compile(src: str, obj: str, extra=()):
    cmd = [HIPCC, *COMMON, *PER_SOURCE.get(src, []), *extra, "-c", os.path.join(CSRC, src), "-o", obj]
    p = subprocess.run(cmd, capture_output=True, text=True)
    if p.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{' '.join(cmd)}\n{p.stdout}\n{p.stderr}")
    return obj


LLVM_BIN = "/opt/rocm/llvm/bin"
DIGESTS = os.path.join(PKG, "kernel_digests.json")
# Per kernel (demangled name): registers and LDS as the gfx950 code object's
# metadata states them.  vgpr_count is the whole per-lane register file a wave
# takes (arch VGPRs rounded up to 4, then AGPRs), agpr_count the AGPR part.
RESOURCES = os.path.join(PKG, "kernel_resources.json")
_RESOURCE_KEYS = {".vgpr_count": "vgpr_count", ".agpr_count": "agpr_count", ".sgpr_count": "sgpr_count",
                  ".group_segment_fixed_size": "lds_bytes", ".private_segment_fixed_size": "scratch_bytes"}


def _device_code_object(obj: str, tmp: str) -> str:
    """The gfx950 code object inside a compiled host object (our own build)."""
    base = os.path.join(tmp, os.path.basename(obj))
    fat, co = base + ".fatbin", base + ".gfx950.co"
    subprocess.run([f"{LLVM_BIN}/llvm-objcopy", "--dump-section", f".hip_fatbin={fat}", obj, base + ".junk"],
                   check=True, capture_output=True)
    subprocess.run([f"{LLVM_BIN}/clang-offload-bundler", "--unbundle", "--type=o",
                    f"--targets=hipv4-amdgcn-amd-amdhsa--{ARCH}", f"--input={fat}", f"--output={co}"],
                   check=True, capture_output=True)
    return co


def _kernel_digests(co: str, resources: dict) -> dict:
    """Per kernel (mangled name): sha256 of its instructions (addresses and
    encodings dropped) and of its resource metadata (registers, LDS, ...).
    Also fills resources[mangled name] from that metadata."""
    dis = subprocess.run([f"{LLVM_BIN}/llvm-objdump", "-d", "--no-show-raw-insn", "--no-leading-addr", co],
                         check=True, capture_output=True, text=True).stdout
    code, name = {}, None
    for line in dis.splitlines():
        if line.endswith(">:") and line.startswith("<"):
            name = line[1:-2]
            code[name] = []
        elif name and line.strip():
            code[name].append(line.split("//")[0].split("<")[0].strip())
        elif not line.strip():
            name = None
    notes = subprocess.run([f"{LLVM_BIN}/llvm-readelf", "--notes", co], check=True, capture_output=True,
                           text=True).stdout
    meta, block = {}, []
    for line in notes.splitlines():
        if line.startswith("  - ") and block:
            meta.update(_meta_block(block))
            block = []
        if line.startswith("  - ") or (block and line.startswith("    ")):
            block.append(line.strip())
    if block:
        meta.update(_meta_block(block))
    for k, block in meta.items():
        res = {}
        for line in block:
            key, _, val = line.partition(":")
            if key in _RESOURCE_KEYS:
                res[_RESOURCE_KEYS[key]] = int(val)
            if line.startswith(".private_segment_fixed_size:") and int(line.split(":")[1]) != 0:
                raise RuntimeError(f"kernel {k} uses scratch memory ({line}); keep it in registers")
        resources[k] = res
    out = {}
    for k, lines in code.items():
        h = hashlib.sha256("\n".join(lines).encode() + b"\0" + "\n".join(meta.get(k, [])).encode())
        out[k] = h.hexdigest()[:16]
    return out


def _meta_block(block):
    name = next((l.split(":", 1)[1].strip() for l in block if l.startswith(".name:")), None)
    return {name: block} if name else {}


def write_kernel_digests(objs, tmp) -> dict:
    """kernel_digests.json: demangled kernel name (as rocprofv3 prints it) ->
    digest of its machine code, so that a profile taken on a kernel is reused
    exactly as long as that kernel's code is unchanged.  kernel_resources.json:
    demangled name -> its registers and LDS (the planner's occupancy model is
    checked against these)."""
    digests, resources = {}, {}
    for obj in objs:
        if obj.endswith(".hip.o"):
            digests.update(_kernel_digests(_device_code_object(obj, tmp), resources))
    names = sorted(digests)
    dem = subprocess.run(["c++filt"], input="\n".join(names), capture_output=True, text=True,
                         check=True).stdout.splitlines()
    table = {d: digests[n] for n, d in zip(names, dem)}
    for path, obj in ((DIGESTS, table), (RESOURCES, {d: resources.get(n, {}) for n, d in zip(names, dem)})):
        with open(path + ".tmp", "w") as f:
            json.dump(obj, f, indent=0, sort_keys=True)
        os.replace(path + ".tmp", path)
    return table


# Debug build with every LDS stage poisoned with NaN once consumed (see
# poison_stage in csrc/conv_kernel.h); tests/test_lds_poison_gpu.py runs
# parity cases on it when it is built.
LIB_LDS_POISON = os.path.join(PKG, "debug", "libmg3m_lds_poison.so")


def build(verbose: bool = False, extra=(), lds_poison: bool = False) -> str:
    """Compile every source and link libmg3m.so (or, lds_poison, the debug
    library LIB_LDS_POISON); returns its path."""
    lib = LIB_LDS_POISON if lds_poison else LIB
    if lds_poison:
        extra = (*extra, "-DMG3M_LDS_POISON=1")
        os.makedirs(os.path.dirname(lib), exist_ok=True)
    with tempfile.TemporaryDirectory(prefix="mg3m_build_") as tmp:
        objs = [os.path.join(tmp, s + ".o") for s in SOURCES]
        with concurrent.futures.ThreadPoolExecutor(len(SOURCES)) as ex:
            list(ex.map(lambda so: _compile(so[0], so[1], extra), zip(SOURCES, objs)))
        if not lds_poison:
            write_kernel_digests(objs, tmp)
        out_tmp = lib + ".tmp"
        cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", out_tmp, *objs]
        p = subprocess.run(cmd, capture_output=True, text=True)
        if p.returncode != 0:
            raise RuntimeError(f"link failed:\n{' '.join(cmd)}\n{p.stdout}\n{p.stderr}")
        os.replace(out_tmp, lib)
    if verbose:
        print(f"built {lib}")
    return lib


# tests/c_abi_gpu.c: the C ABI called from plain C (no Python, no torch),
# linked against the built library; tests/test_c_abi_gpu.py runs it.
C_ABI_TEST = os.path.join(PKG, "debug", "c_abi_gpu")


def build_c_abi_test(verbose: bool = False) -> str:
    """Compile tests/c_abi_gpu.c with gcc against include/mg3m.h and link it
    with the built libmg3m.so and ROCm's HIP runtime."""
    os.makedirs(os.path.dirname(C_ABI_TEST), exist_ok=True)
    cmd = ["gcc", "-std=c11", "-O2", "-Wall", "-Wextra", "-D__HIP_PLATFORM_AMD__",
           f"-I{INCLUDE}", "-I/opt/rocm/include", os.path.join(ROOT, "tests", "c_abi_gpu.c"),
           "-o", C_ABI_TEST + ".tmp", f"-L{PKG}", "-lmg3m", "-L/opt/rocm/lib", "-lamdhip64",
           "-Wl,-rpath,$ORIGIN/..", "-Wl,-rpath,/opt/rocm/lib"]
    p = subprocess.run(cmd, capture_output=True, text=True)
    if p.returncode != 0:
        raise RuntimeError(f"gcc failed:\n{' '.join(cmd)}\n{p.stdout}\n{p.stderr}")
    os.replace(C_ABI_TEST + ".tmp", C_ABI_TEST)
    if verbose:
        print(f"built {C_ABI_TEST}")
    return C_ABI_TEST


if __name__ == "__main__":
    args = sys.argv[1:]
    build(verbose=True, extra=[a for a in args if a != "--lds-poison"], lds_poison="--lds-poison" in args)
