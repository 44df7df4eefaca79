"""The route kernel's compare-exchange networks (csrc/sort_networks.hpp),
built for the host with g++ and checked exhaustively on 0-1 inputs
(tests/sort_network_check.cpp); the device instantiations are the same
templates.  CPU only."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2602_04870_amd", "csrc")


def test_odd_even_networks_sort_every_01_input(tmp_path):
    gxx = shutil.which("g++")
    if gxx is None:
        pytest.skip("no g++")
    exe = str(tmp_path / "sort_network_check")
    cmd = [gxx, "-std=c++17", "-O1", "-Wall", f"-I{CSRC}",
           os.path.join(ROOT, "tests", "sort_network_check.cpp"), "-o", exe]
    res = subprocess.run(cmd, capture_output=True, text=True, timeout=300)
    assert res.returncode == 0, res.stderr[-4000:]
    res = subprocess.run([exe], capture_output=True, text=True, timeout=300)
    assert res.returncode == 0 and "done 0 failures" in res.stdout, res.stdout[-4000:]
    assert "comparators sort16 63" in res.stdout and "comparators merge16+16 65" in res.stdout
    assert "comparators sort32 191" in res.stdout
