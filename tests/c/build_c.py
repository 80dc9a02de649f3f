"""Build the C test programs of tests/c against include/pfc.h and libpfc.so
(host code only, gcc): step_check runs two steps through the C ABI on a GPU.
The binaries go to tests/c/_bin and find libpfc.so through a run path
relative to themselves."""

import os
import shutil
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
BIN = os.path.join(HERE, "_bin")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
PROGRAMS = ["step_check"]


def build():
    gcc = shutil.which("gcc")
    if gcc is None:
        raise RuntimeError("gcc not found: needed for the C test programs")
    os.makedirs(BIN, exist_ok=True)
    out = []
    for name in PROGRAMS:
        exe = os.path.join(BIN, name)
        cmd = [gcc, "-std=c99", "-O2", "-Wall", "-Wextra", "-Werror", "-D__HIP_PLATFORM_AMD__",
               "-I", os.path.join(ROOT, "include"), "-I", os.path.join(ROCM, "include"),
               "-o", exe, os.path.join(HERE, name + ".c"),
               "-L", os.path.join(ROOT, "paper_2010_05222_amd"), "-lpfc",
               "-L", os.path.join(ROCM, "lib"), "-lamdhip64", "-lm",
               "-Wl,-rpath,$ORIGIN/../../../paper_2010_05222_amd",
               "-Wl,-rpath," + os.path.join(ROCM, "lib")]
        res = subprocess.run(cmd, capture_output=True, text=True)
        if res.returncode != 0:
            raise RuntimeError(f"gcc failed on {name}.c:\n{res.stderr}")
        out.append(exe)
    return out


if __name__ == "__main__":
    print("\n".join(build()))
