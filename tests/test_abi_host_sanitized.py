"""The C ABI's host-side layer (argument validation, workspace layout, dispatch setup) built as
plain host C++ with AddressSanitizer and UndefinedBehaviorSanitizer, the kernel launchers and
the two HIP runtime calls it makes replaced by stand-ins (tests/host_sanitizer/stubs.cpp), and
driven through the validation table, the T = 0 paths, workspace sizes and region offsets at the
workloads and at the stated limits, and valid calls up to their first launch
(tests/host_sanitizer/driver.cpp).  Any sanitizer report aborts the driver."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HERE = os.path.join(ROOT, "tests", "host_sanitizer")
CSRC = os.path.join(ROOT, "paper_2607_18631_amd", "csrc")


@pytest.mark.skipif(shutil.which("g++") is None or not os.path.isdir("/opt/rocm/include"),
                    reason="needs g++ and the ROCm headers")
def test_abi_host_layer_under_asan_ubsan(tmp_path):
    exe = str(tmp_path / "abi_host_sanitized")
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           "-D__HIP_PLATFORM_AMD__", "-I", "/opt/rocm/include", "-I", os.path.join(ROOT, "include"),
           os.path.join(CSRC, "api.cpp"), os.path.join(CSRC, "sizes.cpp"),
           os.path.join(HERE, "stubs.cpp"), os.path.join(HERE, "driver.cpp"), "-o", exe]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-3000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=1:verify_asan_link_order=0",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=120)
    assert r.returncode == 0 and r.stdout.strip().endswith("ALL OK"), r.stdout[-3000:] + r.stderr[-3000:]
