"""Build the gfx950 HIP library behind include/mtdao.h.

    python -m paper_2510_05361_amd.build

compiles csrc/mtdao.hip (host code + kernels) with hipcc for gfx950 into
paper_2510_05361_amd/libmtdao.so, and csrc/stream_ref.hip (reference copy /
read / fill kernels used only by the benchmark) into libstream_ref.so.  Packed-fp32 instruction selection is
switched off for the device code.
"""

from __future__ import annotations

import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
SRC = os.path.join(PKG, "csrc", "mtdao.hip")
HEADERS = [os.path.join(PKG, "csrc", "kernels.hpp"), os.path.join(ROOT, "include", "mtdao.h")]
LIB = os.path.join(PKG, "libmtdao.so")
STREAM_SRC = os.path.join(PKG, "csrc", "stream_ref.hip")
STREAM_LIB = os.path.join(PKG, "libstream_ref.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-result", "-Wno-unknown-warning-option",
]


def _compile(src: str, out: str, extra=(), libs=()) -> str:
    tmp = out + ".tmp"
    cmd = [HIPCC, *FLAGS, *extra, "-I", os.path.join(ROOT, "include"), "-o", tmp, src, *libs]
    subprocess.run(cmd, check=True)
    os.replace(tmp, out)
    return out


def build(out: str = LIB, extra=()) -> str:
    """The optimizer library (always) and the benchmark's stream-reference
    kernels (libstream_ref.so)."""
    _compile(STREAM_SRC, STREAM_LIB, extra)
    # roctx ranges (MTDAO_ROCTX=1) come from the rocprofiler-sdk marker library
    return _compile(SRC, out, extra, libs=("-L/opt/rocm/lib", "-lrocprofiler-sdk-roctx", "-Wl,-rpath,/opt/rocm/lib"))


if __name__ == "__main__":
    print(build(extra=sys.argv[1:]))
