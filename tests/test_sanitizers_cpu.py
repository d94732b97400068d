"""AddressSanitizer and UndefinedBehaviorSanitizer builds of the CPU parts:
the oracle (gcc) and the C ABI's host-side validation and dispatch (api.hip
with recording stubs in place of the kernel launchers; hipcc with the
sanitizers on the host pass only).  Each driver in tests/sanitize/ exercises
every entry point over every format and flag set and over rejected
arguments; a sanitizer report or a wrong status fails the test."""
import os
import shutil
import subprocess

import pytest

from paper_2603_28765_amd import _build

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HERE = os.path.join(ROOT, "tests", "sanitize")
SAN_ENV = {**os.environ, "ASAN_OPTIONS": "detect_leaks=1:abort_on_error=0",
           "UBSAN_OPTIONS": "print_stacktrace=1:halt_on_error=1"}


def _run(exe):
    r = subprocess.run([exe], capture_output=True, text=True, env=SAN_ENV, timeout=300)
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-4000:]
    assert "ERROR: AddressSanitizer" not in out and "runtime error" not in out, out[-4000:]
    return out


def test_oracle_under_asan_ubsan(tmp_path):
    if not shutil.which("gcc"):
        pytest.skip("gcc not available")
    exe = str(tmp_path / "oracle_driver")
    cmd = ["gcc", "-O1", "-g", "-std=c11", "-ffp-contract=off", "-fsanitize=address,undefined",
           "-fno-sanitize-recover=all", "-fno-omit-frame-pointer",
           os.path.join(HERE, "oracle_driver.c"), os.path.join(ROOT, "oracle", "ifq_oracle.c"),
           "-o", exe, "-lm"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-3000:]
    assert "0 failures" in _run(exe)


def test_abi_host_validation_under_asan_ubsan(tmp_path):
    hipcc = _build.hipcc()
    if not (shutil.which(hipcc) or os.path.exists(hipcc)):
        pytest.skip("hipcc not available")
    exe = str(tmp_path / "abi_host_driver")
    cmd = [hipcc, f"--offload-arch={_build.ARCH}", "-O1", "-g", "-std=c++17",
           "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer",
           "-I", os.path.join(ROOT, "include"), "-I", _build.CSRC,
           os.path.join(_build.CSRC, "api.hip"), os.path.join(HERE, "abi_host_driver.cpp"), "-o", exe]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-3000:]
    out = _run(exe)
    assert " 0 failures" in out and "launches" in out
