"""The planner's occupancy model against the compiled kernels (no GPU needed).

The selector estimates how many work-groups of a tile fit on one compute
unit from the tile's register count and LDS size (the resident waves that
hide memory latency behind the MFMA pipes).  Those numbers live in a table
in mg3m_internal.h; the build writes what the gfx950 code objects actually
use (kernel_resources.json, from each kernel's metadata notes).  This test
fails as soon as the two disagree, so a kernel edit cannot silently skew
the selector."""
import json
import os
import subprocess
import sys
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2307_04941_amd")
RESOURCES = os.path.join(PKG, "kernel_resources.json")
LIB = os.path.join(PKG, "libmg3m.so")

DUMP = r"""
#include <cstdio>
#include "mg3m_internal.h"
int main() {
  using namespace mg3m;
  std::printf("{\"f32\": [");
  for (int i = 0; i < kNumTiles; ++i) {
    const TileDesc& t = kTiles[i];
    std::printf("%s[%d,%d,%d,%d,%d,%d,%d,%d,%d,%d,%d,%d]", i ? "," : "", t.mt, t.nt, t.kt, t.wm, t.wn, t.regs,
                t.m16, t.m16 ? lds_bytes_for64(t) : lds_bytes_for(t), t.forced_only, t.regs_pt[0], t.regs_pt[1],
                t.regs_pt[2]);
  }
  std::printf("], \"f64\": [");
  for (int i = 0; i < kNumTiles64; ++i) {
    const TileDesc& t = kTiles64[i];
    std::printf("%s[%d,%d,%d,%d,%d,%d,%d,%d,%d]", i ? "," : "", t.mt, t.nt, t.kt, t.wm, t.wn, t.regs,
                t.m16, lds_bytes_for64(t), t.forced_only);
  }
  std::printf("]}\n");
  return 0;
}
"""


def tile_tables():
    """The planner's tile tables, read by compiling mg3m_internal.h on the host."""
    with tempfile.TemporaryDirectory() as tmp:
        src, exe = os.path.join(tmp, "dump.cpp"), os.path.join(tmp, "dump")
        with open(src, "w") as f:
            f.write(DUMP)
        subprocess.run(["g++", "-std=c++17", "-O0", "-I", os.path.join(PKG, "csrc"), "-I",
                        os.path.join(ROOT, "include"), src, "-o", exe], check=True)
        return json.loads(subprocess.run([exe], check=True, capture_output=True, text=True).stdout)


@pytest.fixture(scope="module")
def resources():
    if not os.path.exists(RESOURCES) or (os.path.exists(LIB) and os.path.getmtime(RESOURCES) < os.path.getmtime(LIB) - 60):
        sys.path.insert(0, ROOT)
        from paper_2307_04941_amd import build
        build.build()
    with open(RESOURCES) as f:
        return json.load(f)


def tuned_name(kind, t):
    mt, nt, kt, wm, wn, _, m16 = t[:7]
    if kind == "f64":
        return f"void mg3m::conv_igemm_acc64<0, 0, 3, {mt}, {nt}, {kt}, {wm}, {wn}>(mg3m::KArgs)"
    fn = "conv_igemm_f32_m16" if m16 else "conv_igemm_f32"
    return f"void mg3m::{fn}<0, 0, 3, {mt}, {nt}, {kt}, {wm}, {wn}, false>(mg3m::KArgs)"


@pytest.mark.parametrize("kind", ["f32", "f64"])
def test_register_table_matches_build(kind, resources):
    """regs of every tile = .vgpr_count of its tuned (HWCN one-tap) kernel."""
    drift = []
    for i, t in enumerate(tile_tables()[kind]):
        name = tuned_name(kind, t)
        assert name in resources, f"tile {i}: {name} not in the build"
        got = resources[name]["vgpr_count"]
        if got != t[5]:
            drift.append(f"{kind} tile {i} ({t[0]}x{t[1]} kt={t[2]}): table {t[5]}, compiled {got}")
    assert not drift, "register table drifted from the build:\n" + "\n".join(drift)


@pytest.mark.parametrize("kind", ["f32", "f64"])
def test_lds_model_matches_build(kind, resources):
    """The planner's LDS bytes per work-group = the kernel's static LDS."""
    for i, t in enumerate(tile_tables()[kind]):
        got = resources[tuned_name(kind, t)]["lds_bytes"]
        assert got == t[7], f"{kind} tile {i}: model {t[7]} B, compiled {got} B"


def test_persistent_register_table_matches_build(resources):
    """regs_pt of every tile = .vgpr_count of its persistent kernel with the
    batch-vector (kBVecN) and one-tap (kBVecNTap, and its direct-to-LDS form
    kBVecNTapDma) patch loaders."""
    drift = []
    for i, t in enumerate(tile_tables()["f32"]):
        mt, nt, kt, wm, wn, m16 = t[0], t[1], t[2], t[3], t[4], t[6]
        for slot, b_mode in ((0, 0), (1, 3), (2, 6)):
            name = f"void mg3m::conv_igemm_f32_pt<0, 0, {b_mode}, {mt}, {nt}, {kt}, {wm}, {wn}, false>(mg3m::KArgs)"
            got = resources.get(name, {}).get("vgpr_count", 0)
            if m16:
                assert got == 0 and t[9 + slot] == 0, f"tile {i}: the 16-row tile has no persistent kernel"
            elif got != t[9 + slot]:
                drift.append(f"tile {i} ({mt}x{nt} kt={kt}) b_mode {b_mode}: table {t[9 + slot]}, compiled {got}")
    assert not drift, "persistent register table drifted from the build:\n" + "\n".join(drift)


def _resident(regs, waves, lds):
    """Work-groups per CU as the planner counts them (512 registers per lane
    per SIMD in granules of 8, at most 8 waves per SIMD, 160 KB of LDS)."""
    per_simd = min(8, 512 // ((regs + 7) // 8 * 8))
    return min(max(1, 4 * per_simd // waves), max(1, 160 * 1024 // lds))


def test_direct_lds_kernels_keep_the_modelled_occupancy(resources):
    """The selector counts resident work-groups from the register-staged
    kernel's registers; the direct-to-LDS kernel of the same tile (the
    default one-tap path) needs no more registers and must give the same
    count once LDS caps it."""
    for i, t in enumerate(tile_tables()["f32"]):
        mt, nt, kt, wm, wn, regs, m16, lds = t[:8]
        if m16:
            continue
        name = f"void mg3m::conv_igemm_f32<0, 0, 6, {mt}, {nt}, {kt}, {wm}, {wn}, false>(mg3m::KArgs)"
        got = resources[name]
        assert got["vgpr_count"] <= regs and got["lds_bytes"] == lds, (i, got)
        assert _resident(got["vgpr_count"], wm * wn, lds) == _resident(regs, wm * wn, lds), (i, got)


def test_no_kernel_spills_to_scratch(resources):
    """Every kernel keeps its state in registers (no private segment)."""
    spills = [k for k, r in resources.items() if r.get("scratch_bytes", 0) != 0]
    assert not spills, spills
