"""The host side of libawe (the table builder with its self-checks, plane and workspace
sizes, the C ABI's argument checks, the residue set's constants) built with g++ under
AddressSanitizer and UndefinedBehaviorSanitizer, the device launchers replaced by counting
stubs (tests/host_sanitize/launch_stubs.cpp), and driven by tests/host_sanitize/abi_driver.cpp
through every encoding and the error paths.  CPU only: nothing here touches a GPU."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HERE = os.path.join(ROOT, "tests", "host_sanitize")
CSRC = os.path.join(ROOT, "paper_2609_24519_amd", "csrc")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")


def test_host_abi_under_asan_and_ubsan(tmp_path):
    gxx = shutil.which("g++")
    if gxx is None or not os.path.exists(os.path.join(ROCM, "include", "hip", "hip_runtime.h")):
        pytest.skip("needs g++ and the HIP headers")
    exe = str(tmp_path / "abi_driver")
    cmd = [gxx, "-std=c++17", "-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           "-D__HIP_PLATFORM_AMD__", "-I", os.path.join(ROCM, "include"), "-I", os.path.join(ROOT, "include"),
           "-I", CSRC, os.path.join(CSRC, "awe_tables.cpp"), os.path.join(CSRC, "awe_api.cpp"),
           os.path.join(HERE, "launch_stubs.cpp"), os.path.join(HERE, "abi_driver.cpp"),
           "-L", os.path.join(ROCM, "lib"), "-lamdhip64", "-Wl,-rpath," + os.path.join(ROCM, "lib"), "-o", exe]
    b = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True, timeout=600)
    if b.returncode != 0 and ("asan" in b.stdout or "ubsan" in b.stdout):
        pytest.skip("sanitizer runtime not available: " + b.stdout[-300:])
    assert b.returncode == 0, b.stdout[-3000:]
    env = dict(os.environ)
    # the library keeps its tables for the life of the process on purpose; leaks are not the point
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=0"
    env["UBSAN_OPTIONS"] = "print_stacktrace=1"
    r = subprocess.run([exe], stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True, timeout=600, env=env)
    assert r.returncode == 0, r.stdout[-3000:]
    last = r.stdout.strip().splitlines()[-1].split()
    # every encoding id plus every modulus with a scheme; no failed expectation
    assert last[0] == "schemes" and int(last[1]) >= 10 and last[-2:] == ["failures", "0"], r.stdout[-500:]
