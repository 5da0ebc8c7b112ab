"""The planner, the C ABI's validation and dispatch path, the network
executor's validation and the CPU oracle, built for the host with
AddressSanitizer and UndefinedBehaviorSanitizer (g++/gcc) and run on a seeded
grid of shapes, plan overrides (fuzzed ones included) and malformed
arguments, with the kernel launchers replaced by stubs that check every
launch's arguments against its plan (tests/host_checks.cpp).  No GPU: HIP
runtime calls fail on such a host, which exercises their error paths."""
import os
import shutil
import subprocess
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2307_04941_amd", "csrc")
ROCM = "/opt/rocm"
SAN = ["-fsanitize=address,undefined", "-fno-omit-frame-pointer", "-fno-sanitize-recover=all"]


@pytest.mark.skipif(shutil.which("g++") is None or not os.path.exists(f"{ROCM}/lib/libamdhip64.so"),
                    reason="needs g++ and the HIP runtime library")
def test_host_code_under_asan_ubsan():
    with tempfile.TemporaryDirectory(prefix="mg3m_san_") as tmp:
        objs = []
        for src in ("plan.cpp", "abi.cpp", "net.cpp"):
            o = os.path.join(tmp, src + ".o")
            subprocess.run(["g++", "-std=c++17", "-O1", "-g", *SAN, "-D__HIP_PLATFORM_AMD__",
                            f"-I{ROCM}/include", f"-I{ROOT}/include", f"-I{CSRC}", "-c",
                            os.path.join(CSRC, src), "-o", o], check=True)
            objs.append(o)
        o = os.path.join(tmp, "host_checks.o")
        subprocess.run(["g++", "-std=c++17", "-O1", "-g", *SAN, "-D__HIP_PLATFORM_AMD__", f"-I{ROCM}/include",
                        f"-I{ROOT}/include", f"-I{CSRC}", "-c", os.path.join(ROOT, "tests", "host_checks.cpp"),
                        "-o", o], check=True)
        objs.append(o)
        o = os.path.join(tmp, "direct_conv.o")
        subprocess.run(["gcc", "-std=c11", "-O1", "-g", *SAN, "-c", os.path.join(ROOT, "oracle", "direct_conv.c"),
                        "-o", o], check=True)
        objs.append(o)
        exe = os.path.join(tmp, "host_checks")
        subprocess.run(["g++", *SAN, *objs, f"-L{ROCM}/lib", "-lamdhip64", f"-Wl,-rpath,{ROCM}/lib", "-o", exe],
                       check=True)
        env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:halt_on_error=1:abort_on_error=0",
                   UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1", HIP_VISIBLE_DEVICES="")
        run = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=600)
        out = run.stdout + run.stderr
        assert run.returncode == 0, out[-4000:]
        assert "all host checks passed" in run.stdout, out[-4000:]
        assert "runtime error" not in out and "AddressSanitizer" not in out, out[-4000:]
