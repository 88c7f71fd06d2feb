"""Build the plain-C consumer of the C ABI (abi_driver.c).

It links the GPU library (paper_2510_05361_amd/libmtdao.so), the CPU
oracle (oracle/_liboracle.so, test infrastructure) and the HIP runtime,
with run paths relative to the binary, so the in-tree libraries are the
ones it loads.  Build both libraries first.
"""

from __future__ import annotations

import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
SRC = os.path.join(HERE, "abi_driver.c")
BIN = os.path.join(HERE, "abi_driver")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")


def build() -> str:
    tmp = BIN + ".tmp"
    cmd = ["gcc", "-O2", "-std=c11", "-Wall", "-Wextra", "-D__HIP_PLATFORM_AMD__",
           "-I", os.path.join(ROCM, "include"), "-I", os.path.join(ROOT, "include"),
           "-o", tmp, SRC,
           "-L", os.path.join(ROOT, "paper_2510_05361_amd"), "-lmtdao",
           "-L", os.path.join(ROOT, "oracle"), "-l:_liboracle.so",
           "-L", os.path.join(ROCM, "lib"), "-lamdhip64", "-lm",
           "-Wl,-rpath,$ORIGIN/../../paper_2510_05361_amd", "-Wl,-rpath,$ORIGIN/../../oracle",
           "-Wl,-rpath," + os.path.join(ROCM, "lib")]
    subprocess.run(cmd, check=True)
    os.replace(tmp, BIN)
    return BIN


if __name__ == "__main__":
    print(build())
