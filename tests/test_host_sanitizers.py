"""The host layer of libsparsp under AddressSanitizer and
UndefinedBehaviorSanitizer, without a GPU.

api.cpp (every argument check of the C ABI) and host_plan.cpp (the chunk
schedule, Eq. 4's placed order, the Eq. 3 count and the routing volumes) are
compiled with the host compiler together with stand-in launchers
(tests/hostcheck/stub_launchers.cpp) and a driver
(tests/hostcheck/abi_host_check.cpp) that replays the rejection cases of
test_abi_cpu.py, the success paths into the launchers, and the host planning
code on real arrays. Any sanitizer report aborts the driver; a wrong status
or a launch on a rejected call makes it exit non-zero.
"""

import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2609_32197_amd", "csrc")
HOSTCHECK = os.path.join(ROOT, "tests", "hostcheck")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")


def test_abi_layer_under_asan_and_ubsan(tmp_path):
    cxx = os.environ.get("CXX") or shutil.which("g++")
    if not cxx or not os.path.exists(os.path.join(ROCM, "include", "hip", "hip_runtime_api.h")):
        pytest.skip("needs g++ and the HIP runtime API headers")
    exe = str(tmp_path / "abi_host_check")
    srcs = [os.path.join(CSRC, "api.cpp"), os.path.join(CSRC, "host_plan.cpp"),
            os.path.join(HOSTCHECK, "stub_launchers.cpp"),
            os.path.join(HOSTCHECK, "abi_host_check.cpp")]
    cmd = [cxx, "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           "-D__HIP_PLATFORM_AMD__", f"-I{os.path.join(ROCM, 'include')}",
           f"-I{os.path.join(ROOT, 'include')}", *srcs, "-o", exe]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-4000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0:halt_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=120)
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-4000:]
    assert "runtime error" not in out and "AddressSanitizer" not in out, out[-4000:]
    assert " 0 failures" in r.stdout
    print(r.stdout.strip().splitlines()[-1])
