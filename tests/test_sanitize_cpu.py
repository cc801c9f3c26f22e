"""The C ABI's host layer under AddressSanitizer and UndefinedBehaviorSanitizer.

csrc/api.cpp is compiled by g++ (host code only, no HIP kernels) with
-fsanitize=address,undefined and linked against launch stand-ins
(tests/sanitize/launch_stubs.cpp) that check the launch arguments the host
layer computes. Every validation case of the ABI and host-logic tests, and
calls that pass validation on the largest and most varied tables, then run
in a child process with the sanitizer runtime preloaded; any report fails
the test."""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _gxx():
    return shutil.which("g++")


@pytest.fixture(scope="module")
def sanitized_lib(tmp_path_factory):
    if not _gxx():
        pytest.skip("g++ not available")
    out = str(tmp_path_factory.mktemp("asan") / "libsaf3r_asan.so")
    cmd = [_gxx(), "-std=c++17", "-g", "-O1", "-fPIC", "-shared",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer",
           "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include", "-I", os.path.join(ROOT, "include"),
           os.path.join(ROOT, "paper_2607_03612_amd", "csrc", "api.cpp"),
           os.path.join(ROOT, "tests", "sanitize", "launch_stubs.cpp"), "-o", out]
    res = subprocess.run(cmd, capture_output=True, text=True)
    assert res.returncode == 0, res.stderr
    return out


def test_abi_host_layer_is_clean_under_sanitizers(sanitized_lib):
    asan = subprocess.run([_gxx(), "-print-file-name=libasan.so"], capture_output=True,
                          text=True).stdout.strip()
    env = dict(os.environ)
    env.update({
        "LD_PRELOAD": asan,
        "ASAN_OPTIONS": "detect_leaks=0:abort_on_error=1:halt_on_error=1",
        "UBSAN_OPTIONS": "halt_on_error=1:print_stacktrace=1",
        "SAF3R_LIBRARY": sanitized_lib,
        "PYTHONPATH": ROOT,
    })
    tests = ["tests/test_abi_cpu.py", "tests/test_host_cpu.py", "tests/sanitize/host_paths.py"]
    res = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider",
                          "-m", "not gpu", *tests], cwd=ROOT, env=env, capture_output=True, text=True,
                         timeout=600)
    report = res.stdout[-4000:] + res.stderr[-4000:]
    assert res.returncode == 0, report
    assert "ERROR: AddressSanitizer" not in report and "runtime error" not in report, report
    assert " passed" in res.stdout
