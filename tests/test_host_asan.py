"""The C ABI's host layer (host_api.cpp) under AddressSanitizer and
UndefinedBehaviorSanitizer, on the CPU: built with g++ alone (no device code;
the kernel launchers are stubs that fail), linked into a driver that runs every
entry point's error paths, the host-only helpers and the launch-failure path
(tests/asan/abi_errors.cpp)."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2608_10519_amd", "csrc")
HERE = os.path.join(ROOT, "tests", "asan")


def test_host_layer_error_paths_under_sanitizers(tmp_path):
    if shutil.which("g++") is None or not os.path.isdir("/opt/rocm/include"):
        pytest.skip("g++ or the ROCm headers are not available")
    exe = str(tmp_path / "abi_errors")
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
           "-fno-sanitize-recover=undefined", "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include",
           os.path.join(CSRC, "host_api.cpp"), os.path.join(HERE, "launch_stubs.cpp"),
           os.path.join(HERE, "abi_errors.cpp"), "-L/opt/rocm/lib", "-lamdhip64", "-Wl,-rpath,/opt/rocm/lib",
           "-o", exe]
    b = subprocess.run(cmd, capture_output=True, text=True)
    assert b.returncode == 0, b.stderr[-3000:]
    # a library preloaded into every process would precede the sanitizer's runtime; that order is allowed
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0:exitcode=99:verify_asan_link_order=0",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=120)
    assert r.returncode == 0, (r.stdout + r.stderr)[-4000:]
    assert " 0 failed" in r.stdout and "checks passed" in r.stdout, r.stdout
