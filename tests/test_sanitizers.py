"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only).

Builds the oracle and the library's host layer (argument validation and
launch planning, da_api.cpp, with stub kernel launchers) together with small
drivers in tests/sanitize/, with gcc/g++ and -fsanitize=address,undefined, and
runs them: every sanitizer report fails the test.  No GPU code is built here.
"""
from __future__ import annotations

import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HERE = os.path.join(ROOT, "tests", "sanitize")
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer",
       "-g", "-O1"]
ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
           UBSAN_OPTIONS="print_stacktrace=1")


def _run(cmd, **kw):
    return subprocess.run(cmd, capture_output=True, text=True, timeout=600, **kw)


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not found")
def test_oracle_under_sanitizers(tmp_path):
    exe = str(tmp_path / "oracle_driver")
    b = _run(["gcc", "-std=c11", *SAN, os.path.join(HERE, "oracle_driver.c"),
              os.path.join(ROOT, "oracle", "delta_oracle.c"), "-o", exe, "-lm"])
    assert b.returncode == 0, b.stderr
    r = _run([exe], env=ENV)
    assert r.returncode == 0 and "runtime error" not in r.stderr, r.stdout + r.stderr
    assert "oracle driver ok" in r.stdout


ROCM_LIB = "/opt/rocm/lib"


@pytest.mark.skipif(shutil.which("g++") is None or not os.path.exists(ROCM_LIB + "/libamdhip64.so"),
                    reason="g++ or the HIP runtime library not found")
def test_abi_host_layer_under_sanitizers(tmp_path):
    exe = str(tmp_path / "abi_driver")
    csrc = os.path.join(ROOT, "paper_2505_11254_amd", "csrc")
    b = _run(["g++", "-std=c++17", *SAN, "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include",
              "-I" + os.path.join(ROOT, "include"), "-I" + csrc,
              os.path.join(HERE, "abi_driver.cpp"), os.path.join(csrc, "da_api.cpp"),
              "-o", exe, "-L" + ROCM_LIB, "-Wl,-rpath," + ROCM_LIB, "-lamdhip64"])
    assert b.returncode == 0, b.stderr
    r = _run([exe], env=ENV)
    assert r.returncode == 0 and "runtime error" not in r.stderr, r.stdout + r.stderr
    assert "abi driver ok" in r.stdout
