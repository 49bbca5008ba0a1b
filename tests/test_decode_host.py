"""The work-item decode the GEMM kernel and the host share (kernel_params.h:
work_items, decode_item, tile_of), compiled for the host with g++ and checked
over a grid of launch shapes and split settings (tests/decode_check.cpp):
every work position is one (tile, K slice), every tile's K is covered once,
split counters and workspace tiles are distinct and within bounds, and the
tile walk is a bijection."""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "..", "paper_2609_10549_amd", "csrc")


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs a host C++ compiler")
def test_work_item_decode_is_a_bijection(tmp_path):
    exe = tmp_path / "decode_check"
    subprocess.run(["g++", "-std=c++17", "-O1", "-Wall", "-Werror", f"-I{CSRC}", "-o", str(exe),
                    os.path.join(HERE, "decode_check.cpp")], check=True)
    out = subprocess.run([str(exe)], capture_output=True, text=True, timeout=120)
    assert out.returncode == 0, out.stdout + out.stderr
    assert out.stdout.startswith("ok "), out.stdout
    assert int(out.stdout.split()[1]) > 10000
