"""The host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU).

- The CPU oracle (oracle/oracle.c) with a C driver: every bit width, ragged
  lengths, windows, ties, constant and subnormal groups, the range error.
- The library's host code (paper_2607_16248_amd/csrc/kvq_api.cpp: argument
  checks, length bookkeeping, page lists, split plans, workspace sizes,
  export offsets) with host buffers standing in for device memory and no-op
  kernel launches (tests/sanitize/hip), so that every copy the host code
  computes into the arena, the workspace or an export buffer is checked.

Both are built with the system compilers (gcc / g++), never for the GPU.
"""
import os
import re
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN = ["-g", "-O1", "-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer"]
ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0", UBSAN_OPTIONS="print_stacktrace=1",
           OMP_NUM_THREADS="2")


def _run(cmd, **kw):
    r = subprocess.run(cmd, capture_output=True, text=True, **kw)
    assert r.returncode == 0, (cmd[0], r.returncode, r.stdout[-3000:], r.stderr[-3000:])
    return r


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not available")
def test_oracle_under_sanitizers(tmp_path):
    exe = str(tmp_path / "oracle_check")
    _run(["gcc", "-std=c11", "-fopenmp", "-ffp-contract=off"] + SAN +
         ["-I", os.path.join(ROOT, "oracle"), os.path.join(ROOT, "oracle", "oracle.c"),
          os.path.join(ROOT, "tests", "sanitize", "oracle_check.c"), "-o", exe, "-lm"])
    r = _run([exe], env=ENV, timeout=300)
    assert "oracle checks ok" in r.stdout


@pytest.mark.skipif(shutil.which("g++") is None, reason="g++ not available")
def test_host_library_under_sanitizers(tmp_path):
    exe = str(tmp_path / "host_check")
    san = os.path.join(ROOT, "tests", "sanitize")
    _run(["g++", "-std=c++17", "-Wno-return-type-c-linkage"] + SAN +
         ["-I", san, "-I", os.path.join(ROOT, "include"), "-I", os.path.join(ROOT, "paper_2607_16248_amd", "csrc"),
          os.path.join(ROOT, "paper_2607_16248_amd", "csrc", "kvq_api.cpp"), os.path.join(san, "hip_stub.cpp"),
          os.path.join(san, "host_check.cpp"), "-o", exe])
    r = _run([exe], env=ENV, timeout=600)
    assert "host checks ok" in r.stdout
    # the chunk launches' row groups (every head count, n_q up to 64, spare
    # rows) were checked by the launch stand-ins
    assert int(re.search(r"(\d+) chunk row plans checked", r.stdout).group(1)) >= 50, r.stdout
