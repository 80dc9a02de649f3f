"""Two training steps driven from C (tests/c/step_check.c): device memory
from hipMalloc, every stage through the C ABI, no Python runtime in the
process.  The program checks the active set, the remap, finite outputs and
that rows outside both active sets are untouched."""

import os
import subprocess
import sys

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
EXE = os.path.join(HERE, "c", "_bin", "step_check")


@pytest.mark.gpu
def test_two_steps_from_c():
    if not os.path.exists(EXE):
        sys.path.insert(0, os.path.join(HERE, "c"))
        import build_c
        build_c.build()
    print("\nC program: two bf16 steps, B=64 d=128 C=5000 r=0.1", flush=True)
    out = subprocess.run([EXE], capture_output=True, text=True, timeout=120)
    print(out.stdout, out.stderr, flush=True)
    assert out.returncode == 0, out.stderr
    assert "step_check ok" in out.stdout
