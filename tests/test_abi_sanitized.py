"""The host-side argument checks of the attention library under AddressSanitizer and UBSan:
csrc/ts_attn.cpp and csrc/attn_plan.cpp are compiled with g++ (host code only, no device code)
together with tests/abi_san/driver.cpp, which calls every entry point over a grid of extreme
sizes, head counts, head dims, scales and pointer layouts, and tests/abi_san/launch_stubs.cpp,
which stands in for the kernels (device set-up fails, so nothing is ever launched)."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2606_19271_amd", "csrc")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")


def test_abi_checks_are_clean_under_asan_and_ubsan(tmp_path):
    if shutil.which("g++") is None:
        pytest.skip("g++ not available")
    exe = str(tmp_path / "driver")
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-Wall", "-Wextra", "-Werror",
           "-D__HIP_PLATFORM_AMD__", "-I" + os.path.join(ROCM, "include"),
           "-I" + os.path.join(ROOT, "include"), "-I" + CSRC,
           os.path.join(CSRC, "ts_attn.cpp"), os.path.join(CSRC, "attn_plan.cpp"),
           os.path.join(ROOT, "tests", "abi_san", "driver.cpp"),
           os.path.join(ROOT, "tests", "abi_san", "launch_stubs.cpp"),
           "-o", exe, "-L" + os.path.join(ROCM, "lib"), "-lamdhip64",
           "-Wl,-rpath," + os.path.join(ROCM, "lib")]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1", UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([exe], capture_output=True, text=True, timeout=300, env=env)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "failures 0" in r.stdout
