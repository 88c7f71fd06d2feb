"""CPU-only sanitizer builds of the host code (no GPU needed to run them):

  libmtdao_san.so   the C ABI (csrc/mtdao.hip) with AddressSanitizer and
                    UndefinedBehaviorSanitizer in its host code only (each
                    -fsanitize= applies to the host pass: -Xarch_host)
  host_abi_check    a plain-C driver of the host paths, linked to it

The driver calls no path that launches a kernel.  Built with the ROCm
clang, whose sanitizer runtime the driver carries.
"""

from __future__ import annotations

import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
CLANG = "/opt/rocm/llvm/bin/clang"
LIB = os.path.join(HERE, "libmtdao_san.so")
BIN = os.path.join(HERE, "host_abi_check")
SAN = ["-fsanitize=address", "-fsanitize=undefined"]


STAMP = os.path.join(HERE, ".build_stamp")


def _inputs_hash() -> str:
    """Hash of everything the two outputs are built from (sources and this
    script), so an unchanged tree reuses them."""
    import hashlib
    h = hashlib.sha256()
    for f in (os.path.join(ROOT, "paper_2510_05361_amd", "csrc", "mtdao.hip"),
              os.path.join(ROOT, "paper_2510_05361_amd", "csrc", "kernels.hpp"),
              os.path.join(ROOT, "include", "mtdao.h"), os.path.join(HERE, "host_abi_check.c"), __file__):
        with open(f, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def build() -> str:
    key = _inputs_hash()
    if os.path.exists(LIB) and os.path.exists(BIN) and os.path.exists(STAMP):
        with open(STAMP) as f:
            if f.read().strip() == key:
                return BIN
    src = os.path.join(ROOT, "paper_2510_05361_amd", "csrc", "mtdao.hip")
    host_san = [a for f in SAN for a in ("-Xarch_host", f)]
    subprocess.run([HIPCC, "--offload-arch=gfx950", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", "-O1", "-g", "-std=c++17", "-fPIC", "-shared",
                    "-fno-omit-frame-pointer", *host_san, "-I", os.path.join(ROOT, "include"),
                    "-o", LIB, src, "-L/opt/rocm/lib", "-lrocprofiler-sdk-roctx", "-Wl,-rpath,/opt/rocm/lib"], check=True)
    subprocess.run([CLANG, "-O1", "-g", "-std=c11", "-fno-omit-frame-pointer", *SAN, "-I",
                    os.path.join(ROOT, "include"), "-o", BIN, os.path.join(HERE, "host_abi_check.c"), LIB,
                    "-Wl,-rpath," + HERE, "-L/opt/rocm/lib", "-lamdhip64", "-Wl,-rpath,/opt/rocm/lib"], check=True)
    with open(STAMP, "w") as f:
        f.write(key + "\n")
    return BIN


if __name__ == "__main__":
    print(build())
