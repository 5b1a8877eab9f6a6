"""Builds tests/c_abi/jorge_c_driver, the plain C caller of the library, with gcc
(C11, no C++ and no HIP compiler): it links libjorge.so from the package
directory (found at run time through an rpath relative to the binary) and the
HIP runtime."""
from __future__ import annotations

import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
SRC = os.path.join(HERE, "jorge_c_driver.c")
OUT = os.path.join(HERE, "jorge_c_driver")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")


def command(out: str = OUT) -> list[str]:
    return ["gcc", "-std=c11", "-O2", "-Wall", "-Wextra", "-Werror", "-D__HIP_PLATFORM_AMD__",
            "-I", os.path.join(ROOT, "include"), "-I", os.path.join(ROCM, "include"), SRC, "-o", out,
            "-L", os.path.join(ROOT, "paper_2310_12298_amd"), "-ljorge",
            "-L", os.path.join(ROCM, "lib"), "-lamdhip64",
            "-Wl,-rpath,$ORIGIN/../../paper_2310_12298_amd", "-Wl,-rpath," + os.path.join(ROCM, "lib")]


def build_driver(out: str = OUT) -> str:
    """Compiles the driver (libjorge.so must be built first); raises CalledProcessError on failure."""
    res = subprocess.run(command(out), capture_output=True, text=True)
    if res.returncode != 0:
        raise subprocess.CalledProcessError(res.returncode, res.args, res.stdout, res.stderr)
    return out


if __name__ == "__main__":
    print(build_driver())
