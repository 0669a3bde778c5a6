"""The scheduler's host code under AddressSanitizer and UBSan: csrc/sched.cpp is compiled with
g++ together with tests/sched_san/driver.cpp, a C++ client of include/ts_sched.h that feeds it
random valid and invalid epoch batches and checks every decision (see the driver's header)."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SOURCES = [os.path.join(ROOT, "paper_2606_19271_amd", "csrc", "sched.cpp"),
           os.path.join(ROOT, "tests", "sched_san", "driver.cpp")]


@pytest.fixture(scope="module")
def driver(tmp_path_factory):
    if shutil.which("g++") is None:
        pytest.skip("g++ not available")
    exe = str(tmp_path_factory.mktemp("sched_san") / "driver")
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-ffp-contract=off",
           "-Wall", "-Wextra", "-Werror", "-I" + os.path.join(ROOT, "include")] + SOURCES + ["-o", exe]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    return exe


@pytest.mark.parametrize("seed", [1, 2])
def test_scheduler_is_clean_under_asan_and_ubsan(driver, seed):
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([driver, "30", "100", str(seed)], capture_output=True, text=True,
                       timeout=300, env=env)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "failures 0" in r.stdout
