"""The library's host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only).

Builds the host translation units of libdtp.so (exact and dual-ascent neuron steps,
partitions, encoding, the ABI's host entry points and argument checks) with g++ and the
two sanitizers, together with ``tests/host_sanitizer/driver.cpp``, which stubs out the GPU
launchers and checks every host entry point against brute force on seeded small and
tie-heavy instances.  Any memory error or undefined behaviour aborts the driver.
"""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2609_13846_amd", "csrc")
HOST_SOURCES = ["abi.cpp", "assign.cpp", "encode.cpp", "partitions.cpp"]
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")


def test_host_code_under_sanitizers(tmp_path):
    gxx = shutil.which("g++")
    if gxx is None or not os.path.exists(os.path.join(ROCM, "lib", "libamdhip64.so")):
        pytest.skip("g++ or the HIP runtime library is not available")
    exe = tmp_path / "host_checks"
    cmd = [gxx, "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           "-D__HIP_PLATFORM_AMD__", f"-I{ROCM}/include", f"-I{ROOT}/include", f"-I{CSRC}",
           *[os.path.join(CSRC, f) for f in HOST_SOURCES],
           os.path.join(ROOT, "tests", "host_sanitizer", "driver.cpp"),
           f"-L{ROCM}/lib", "-lamdhip64", "-lpthread", f"-Wl,-rpath,{ROCM}/lib", "-o", str(exe)]
    build = subprocess.run(cmd, capture_output=True, text=True, timeout=600)
    assert build.returncode == 0, build.stderr[-4000:]
    # verify_asan_link_order=0: the sanitizer runtime need not come first among the
    # libraries the environment preloads
    env = dict(os.environ, ASAN_OPTIONS="abort_on_error=1:detect_leaks=1:verify_asan_link_order=0",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    run = subprocess.run([str(exe)], capture_output=True, text=True, timeout=600, env=env)
    assert run.returncode == 0, (run.stdout[-2000:] + run.stderr[-6000:])
    assert "host checks passed" in run.stdout
