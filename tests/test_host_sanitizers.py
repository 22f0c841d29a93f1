"""The C ABI's host layer (csrc/api.cpp) under AddressSanitizer and UndefinedBehaviorSanitizer,
on the CPU: tests/host/host_layer_test.cpp drives every entry point with exact-size buffers
and invalid arguments, and tests/host/stub_launchers.cpp stands in for the kernel launchers
(touching the ends of every range a kernel would address, copying every uploaded table into
its workspace slot).  Built with g++ (host code only), no GPU needed."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2608_27128_amd", "csrc")
HOST = os.path.join(ROOT, "tests", "host")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")


def test_host_layer_under_asan_ubsan(tmp_path):
    gxx = shutil.which("g++")
    if gxx is None or not os.path.exists(os.path.join(ROCM, "include", "hip", "hip_runtime_api.h")):
        pytest.skip("g++ or the HIP headers are missing")
    exe = tmp_path / "host_layer_test"
    cmd = [gxx, "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           "-D__HIP_PLATFORM_AMD__", f"-I{ROCM}/include", f"-I{CSRC}", f"-I{ROOT}/include",
           os.path.join(CSRC, "api.cpp"), os.path.join(HOST, "stub_launchers.cpp"),
           os.path.join(HOST, "host_layer_test.cpp"), "-o", str(exe)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-4000:]
    # the environment is passed on as it is; ASan is told not to insist on coming first in
    # the library list, so a library the environment preloads is left in place
    env = dict(os.environ,
               ASAN_OPTIONS="detect_leaks=1:abort_on_error=0:halt_on_error=1:verify_asan_link_order=0",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([str(exe)], capture_output=True, text=True, env=env, timeout=300)
    assert r.returncode == 0 and "host layer ok" in r.stdout, (r.stdout[-2000:], r.stderr[-6000:])
