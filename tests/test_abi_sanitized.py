"""The host side of the C ABI under AddressSanitizer and
UndefinedBehaviorSanitizer (CPU only).

``csrc/mla_abi.cpp`` is plain C++: it is compiled with g++ and
``-fsanitize=address,undefined`` (no recovery) together with
``abi_host_driver.cpp``, whose stubs stand in for the kernel launchers, and
the driver runs every entry point's host code -- validation of bad and edge
arguments, page geometry, both split planners up to the int32 limit, storage
accounting, dispatch and the argument records handed to the launchers, the
timing hook, the combine and the allocation-free entry point.  Any memory
error or undefined behaviour aborts the driver.
"""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2609_36760_amd", "csrc")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")
def test_host_abi_under_address_and_undefined_behaviour_sanitizers(tmp_path):
    exe = tmp_path / "abi_driver"
    san = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer"]
    cmd = ["g++", "-std=c++17", "-O1", "-g", *san, "-D__HIP_PLATFORM_AMD__",
           "-I", os.path.join(ROCM, "include"), "-I", os.path.join(ROOT, "include"), "-I", CSRC,
           os.path.join(CSRC, "mla_abi.cpp"), os.path.join(ROOT, "tests", "abi_host_driver.cpp"), "-o", str(exe)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=1", UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([str(exe)], capture_output=True, text=True, env=env, timeout=120)
    print(r.stdout, r.stderr)
    assert r.returncode == 0, r.stderr
    assert "all checks passed" in r.stdout
