"""Host sanitizer builds (CPU only): the oracle and the C-ABI layer's
validation and dispatch code built with AddressSanitizer and
UndefinedBehaviorSanitizer (gcc / g++, host code only) and driven through
valid, invalid and limit-sized arguments (tests/sanitize/)."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HERE = os.path.join(ROOT, "tests", "sanitize")
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-g", "-O1"]


def _run(cmd, env=None, timeout=300):
    res = subprocess.run(cmd, capture_output=True, text=True, timeout=timeout, env=env)
    assert res.returncode == 0, res.stdout[-3000:] + res.stderr[-3000:]
    return res.stdout


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not available")
def test_oracle_under_asan_ubsan(tmp_path):
    exe = str(tmp_path / "oracle_driver")
    _run(["gcc", "-std=c11", *SAN, "-fopenmp", "-ffp-contract=off", os.path.join(HERE, "oracle_driver.c"),
          os.path.join(ROOT, "oracle", "sq_oracle.c"), "-o", exe, "-lm"])
    env = dict(os.environ, OMP_NUM_THREADS="2", ASAN_OPTIONS="detect_leaks=1")
    assert "ORACLE OK" in _run([exe], env=env)


@pytest.mark.skipif(shutil.which("g++") is None or not os.path.isdir("/opt/rocm/include"),
                    reason="g++ or the ROCm headers not available")
def test_abi_validation_under_asan_ubsan(tmp_path):
    exe = str(tmp_path / "abi_driver")
    inc = ["-I", os.path.join(ROOT, "include"), "-I", os.path.join(ROOT, "paper_2609_21704_amd", "csrc"),
           "-I", "/opt/rocm/include", "-D__HIP_PLATFORM_AMD__"]
    _run(["g++", "-std=c++17", *SAN, *inc, os.path.join(HERE, "abi_driver.cpp"), os.path.join(HERE, "abi_stubs.cpp"),
          os.path.join(ROOT, "paper_2609_21704_amd", "csrc", "abi.cpp"), "-o", exe, "-lpthread"])
    assert "ABI OK" in _run([exe], env=dict(os.environ, ASAN_OPTIONS="detect_leaks=1"))
