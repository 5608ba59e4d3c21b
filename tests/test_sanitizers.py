"""The CPU oracle and the C ABI's host-side argument checks under the host
compiler's AddressSanitizer and UndefinedBehaviorSanitizer (no GPU).

Two small drivers (tests/sanitize/) are built with gcc / g++ and
-fsanitize=address,undefined: one runs the oracle over edge shapes (n = m,
m = 32 and 64, floored groups, zero and one group, partial 2:4 metadata words,
the categorical sampler at 70 candidates, the threaded entry points, rejected
arguments), the other the argument checks of checks.cpp (every status each
case should get, overflowing sizes and offsets, overlapping ranges, the split
of a launch at Philox block-index boundaries).  Any sanitizer report fails the
run."""
from __future__ import annotations

import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HERE = os.path.join(ROOT, "tests", "sanitize")
CSRC = os.path.join(ROOT, "paper_2608_23048_amd", "csrc")
SAN = ["-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
       "-fno-sanitize-recover=all"]
ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0:halt_on_error=1",
           UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")


def build_and_run(cmd, exe, tmp_path):
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stderr[-4000:]
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=300, env=ENV,
                       cwd=str(tmp_path))
    out = r.stdout + r.stderr
    assert "runtime error" not in out and "AddressSanitizer" not in out and \
        "LeakSanitizer" not in out, out[-4000:]
    assert r.returncode == 0, out[-4000:]
    return out


def test_oracle_under_sanitizers(tmp_path):
    gcc = shutil.which("gcc")
    if not gcc:
        pytest.skip("gcc not available")
    exe = tmp_path / "oracle_driver"
    out = build_and_run([gcc, "-std=c11", *SAN, "-ffp-contract=off", "-Wall", "-Wextra",
                         "-Werror", f"-I{os.path.join(ROOT, 'oracle')}",
                         os.path.join(ROOT, "oracle", "roi_oracle.c"),
                         os.path.join(HERE, "oracle_driver.c"), "-o", str(exe), "-lm",
                         "-lpthread"], exe, tmp_path)
    assert "oracle ok" in out


def test_host_checks_under_sanitizers(tmp_path):
    gxx = shutil.which("g++")
    if not gxx or not os.path.exists("/opt/rocm/include/hip/hip_runtime_api.h"):
        pytest.skip("g++ or the HIP headers not available")
    exe = tmp_path / "checks_driver"
    out = build_and_run([gxx, "-std=c++17", *SAN, "-Wall", "-Wextra", "-Werror",
                         "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include",
                         f"-I{os.path.join(ROOT, 'include')}", f"-I{CSRC}",
                         os.path.join(CSRC, "checks.cpp"), os.path.join(HERE, "checks_driver.cpp"),
                         "-o", str(exe)], exe, tmp_path)
    assert "checks ok" in out
