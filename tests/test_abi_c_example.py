"""The C ABI used from plain C (tests/native/abi_roundtrip.c): it compiles
against include/isoquant.h with a C compiler (CPU test), and the program
built by __graft_entry__.build() runs init -> quantize -> dequantize -> round
trip on the GPU and checks its own results (GPU test)."""
import os
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
BIN = os.path.join(ROOT, "tests", "native", "abi_roundtrip")


def test_c_example_compiles(tmp_path):
    import __graft_entry__ as g

    if not os.path.exists(os.path.join(ROOT, "paper_2603_28430_amd", "libisoquant.so")):
        pytest.skip("library not built")
    out = g.build_c_example(str(tmp_path / "abi_roundtrip"))
    assert os.path.exists(out)


@pytest.mark.gpu
def test_c_example_runs_on_the_gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    assert os.path.exists(BIN), "tests/native/abi_roundtrip is built by __graft_entry__.build()"
    print("case abi_roundtrip (C program)", flush=True)
    r = subprocess.run([BIN], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "abi_roundtrip ok" in r.stdout
