"""The host side of the C ABI (schedule construction, argument checks) built
with g++ under AddressSanitizer and UBSan and run on generated graphs.  The
device launchers are replaced by host stand-ins (tests/host/stub_kernels.cpp),
so no GPU is needed; tests/host/schedule_driver.cpp checks that every
schedule covers each row's edges exactly once, numbers its partial-result
slots consistently, honours the output capacity, and that bad arguments are
rejected before any device work."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
ROCM = "/opt/rocm"


def test_host_abi_under_address_and_ub_sanitizers(tmp_path):
    gxx = shutil.which("g++")
    if not gxx or not os.path.exists(os.path.join(ROCM, "include", "hip", "hip_runtime_api.h")) \
            or not os.path.exists(os.path.join(ROCM, "lib", "libamdhip64.so")):
        pytest.skip("needs g++ and the ROCm headers and runtime library")
    exe = str(tmp_path / "schedule_driver")
    csrc = os.path.join(ROOT, "paper_2008_11359_amd", "csrc")
    cmd = [gxx, "-std=c++17", "-O1", "-g", "-fsanitize=address,undefined",
           "-fno-sanitize-recover=all", "-D__HIP_PLATFORM_AMD__",
           "-I" + os.path.join(ROCM, "include"), "-I" + os.path.join(ROOT, "include"), "-I" + csrc,
           os.path.join(csrc, "fg_api.cpp"), os.path.join(ROOT, "tests", "host", "stub_kernels.cpp"),
           os.path.join(ROOT, "tests", "host", "schedule_driver.cpp"),
           "-L" + os.path.join(ROCM, "lib"), "-lamdhip64", "-Wl,-rpath," + os.path.join(ROCM, "lib"),
           "-o", exe]
    subprocess.run(cmd, check=True, timeout=600)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0", UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([exe], env=env, capture_output=True, text=True, timeout=600)
    assert r.returncode == 0, (r.stdout + r.stderr)[-4000:]
    assert r.stdout.startswith("ok "), r.stdout
