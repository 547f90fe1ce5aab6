"""The host side of libawe (the table builder with its self-checks, plane and workspace
sizes, the C ABI's argument checks, the residue set's constants and caches) built with g++
under the host sanitizers, the device launchers replaced by counting stubs
(tests/host_sanitize/launch_stubs.cpp): AddressSanitizer and UndefinedBehaviorSanitizer over
every encoding and error path (tests/host_sanitize/abi_driver.cpp), ThreadSanitizer over
eight threads calling the ABI at once (tests/host_sanitize/abi_threads.cpp).  CPU only:
nothing here touches a GPU."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HERE = os.path.join(ROOT, "tests", "host_sanitize")
CSRC = os.path.join(ROOT, "paper_2609_24519_amd", "csrc")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")


def _build_and_run(tmp_path, driver, sanitize, env_extra):
    gxx = shutil.which("g++")
    if gxx is None or not os.path.exists(os.path.join(ROCM, "include", "hip", "hip_runtime.h")):
        pytest.skip("needs g++ and the HIP headers")
    exe = str(tmp_path / driver.split(".")[0])
    cmd = [gxx, "-std=c++17", "-O1", "-g", "-fsanitize=" + sanitize, "-fno-sanitize-recover=all",
           "-D__HIP_PLATFORM_AMD__", "-I", os.path.join(ROCM, "include"), "-I", os.path.join(ROOT, "include"),
           "-I", CSRC, os.path.join(CSRC, "awe_tables.cpp"), os.path.join(CSRC, "awe_api.cpp"),
           os.path.join(HERE, "launch_stubs.cpp"), os.path.join(HERE, driver),
           "-L", os.path.join(ROCM, "lib"), "-lamdhip64", "-Wl,-rpath," + os.path.join(ROCM, "lib"),
           "-lpthread", "-o", exe]
    b = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True, timeout=600)
    if b.returncode != 0 and ("asan" in b.stdout or "ubsan" in b.stdout or "tsan" in b.stdout):
        pytest.skip("sanitizer runtime not available: " + b.stdout[-300:])
    assert b.returncode == 0, b.stdout[-3000:]
    env = dict(os.environ)
    env.update(env_extra)
    r = subprocess.run([exe], stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True, timeout=600, env=env)
    assert r.returncode == 0, r.stdout[-3000:]
    return r.stdout.strip().splitlines()[-1].split()


def test_host_abi_under_asan_and_ubsan(tmp_path):
    # the library keeps its tables for the life of the process on purpose; leaks are not the point
    last = _build_and_run(tmp_path, "abi_driver.cpp", "address,undefined",
                          {"ASAN_OPTIONS": "detect_leaks=0:abort_on_error=0",
                           "UBSAN_OPTIONS": "print_stacktrace=1"})
    # every encoding id plus every modulus with a scheme; no failed expectation
    assert last[0] == "schemes" and int(last[1]) >= 10 and last[-2:] == ["failures", "0"], last


def test_host_abi_threads_under_tsan(tmp_path):
    last = _build_and_run(tmp_path, "abi_threads.cpp", "thread", {"TSAN_OPTIONS": "halt_on_error=1"})
    assert last == ["threads", "8", "failures", "0"], last
