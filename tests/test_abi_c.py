"""The C ABI from C: include/pfc.h compiles as strict C99 and a small program
linked against libpfc.so gets the documented results from the host-side
entry points (sizes, capacity, argument checks, status strings).  No GPU."""

import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIBDIR = os.path.join(ROOT, "paper_2010_05222_amd")


@pytest.mark.skipif(shutil.which("gcc") is None, reason="no gcc")
def test_header_compiles_as_c99_and_host_calls_work(tmp_path):
    if not os.path.exists(os.path.join(LIBDIR, "libpfc.so")):
        pytest.skip("libpfc.so not built")
    exe = tmp_path / "abi_check"
    subprocess.run(["gcc", "-std=c99", "-Wall", "-Wextra", "-Werror", "-pedantic",
                    "-I", os.path.join(ROOT, "include"), "-o", str(exe),
                    os.path.join(ROOT, "tests", "c", "abi_check.c"), "-L", LIBDIR, "-lpfc",
                    "-Wl,-rpath," + LIBDIR], check=True, capture_output=True, text=True)
    out = subprocess.run([str(exe)], capture_output=True, text=True, timeout=120)
    assert out.returncode == 0, out.stderr
    assert "abi_check ok" in out.stdout
