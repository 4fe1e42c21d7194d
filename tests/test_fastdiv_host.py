"""The cache-slot division of the append kernels (slot / block_size) uses
multiply-shift constants from make_fastdiv (Granlund and Montgomery, PLDI
1994, Fig. 4.1).  Compile a host program against the library's header and
check the constants and the kernels' formula against exact division for every
divisor up to 5,000, the powers of two and their neighbours, 2^32 - 1 and
2,000 random divisors, each at about 2,300 dividends (multiples of d and
their predecessors, the extremes, random values).  Runs on the CPU."""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(os.path.dirname(HERE), "paper_2603_28430_amd", "csrc")


def test_fastdiv_constants(tmp_path):
    cxx = shutil.which("g++") or shutil.which("c++")
    if cxx is None:
        pytest.skip("no host C++ compiler")
    exe = tmp_path / "fastdiv_check"
    subprocess.run([cxx, "-O2", "-std=c++17", f"-I{CSRC}", os.path.join(HERE, "native", "fastdiv_check.cpp"),
                    "-o", str(exe)], check=True, capture_output=True, text=True)
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "failures 0" in r.stdout
