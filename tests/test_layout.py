"""Host check of the matrix-core code layouts: the bit maps of every width
are bijections with exact inverses, and the decode kernel's operand unpacking
(emulated on the host) returns each code times its fixed weight.  The
byte-exact end-to-end check of the same layouts is the GPU parity suite
(kvq_export against the oracle's canonical image)."""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(os.path.dirname(HERE), "paper_2607_16248_amd", "csrc")


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs a host C++ compiler")
def test_matrix_layouts_on_host(tmp_path):
    exe = tmp_path / "layout_check"
    subprocess.run(["g++", "-std=c++17", "-O1", "-Wall", "-I", CSRC, os.path.join(HERE, "layout_check.cpp"),
                    "-o", str(exe)], check=True)
    out = subprocess.run([str(exe)], capture_output=True, text=True)
    assert out.returncode == 0 and out.stdout.strip() == "ok", out.stdout + out.stderr
