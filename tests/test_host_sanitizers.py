"""The library's host code under AddressSanitizer and UndefinedBehaviorSanitizer
(CPU only). csrc/validate.cpp -- every argument check and workspace size the
exported calls run before anything is enqueued -- is plain C++ without HIP, so
g++ builds it with both sanitizers beside a driver (sanitize/validate_driver.cpp)
that replays the ABI tests' invalid-argument cases, valid shapes, and the size
functions at the extremes of their int32 arguments. Any out-of-bounds access or
signed overflow aborts the driver."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_host_checks_under_address_and_undefined_behavior_sanitizers(tmp_path):
    gxx = shutil.which("g++")
    if gxx is None:
        pytest.skip("g++ is not available")
    exe = str(tmp_path / "validate_driver")
    build = subprocess.run(
        [gxx, "-std=c++17", "-g", "-O1", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
         "-fno-omit-frame-pointer", "-Wall", "-Werror",
         os.path.join(ROOT, "paper_2606_31519_amd", "csrc", "validate.cpp"),
         os.path.join(ROOT, "tests", "sanitize", "validate_driver.cpp"), "-o", exe],
        stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    assert build.returncode == 0, build.stdout
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    run = subprocess.run([exe], stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True, env=env, timeout=120)
    assert run.returncode == 0 and "all host checks passed" in run.stdout, run.stdout
