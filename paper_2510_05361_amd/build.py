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


RESOURCES = os.path.join(PKG, "kernel_resources.txt")
_REMARK = "-Rpass-analysis=kernel-resource-usage"
_FIELDS = ("Function Name:", "VGPRs:", "AGPRs:", "ScratchSize [bytes/lane]:", "Occupancy [waves/SIMD]:",
           "LDS Size [bytes/block]:")


def source_hash() -> str:
    """Hash of the device sources the kernels are compiled from."""
    import hashlib
    h = hashlib.sha256()
    for f in [SRC, *HEADERS]:
        with open(f, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def resource_rows(remarks: str):
    """[{name, VGPRs, AGPRs, ScratchSize, Occupancy, LDS}] from hipcc's
    kernel-resource-usage remarks."""
    rows, cur = [], None
    for line in remarks.splitlines():
        if "remark:" not in line:
            continue
        body = line.split("remark:", 1)[1].strip()
        for f in _FIELDS:
            if body.startswith(f):
                val = body[len(f):].split("[-R")[0].strip()
                if f == "Function Name:":
                    cur = {"name": val}
                    rows.append(cur)
                elif cur is not None:
                    cur[f.split()[0].rstrip(":")] = int(val)
    return rows


def _compile(src: str, out: str, extra=(), libs=(), resources: str = "") -> str:
    """hipcc src into out; with ``resources``, also write the register,
    scratch and occupancy figures of every kernel there."""
    tmp = out + ".tmp"
    cmd = [HIPCC, *FLAGS, *extra, "-I", os.path.join(ROOT, "include"), "-o", tmp, src, *libs]
    if resources:
        cmd.append(_REMARK)
    r = subprocess.run(cmd, stderr=subprocess.PIPE, text=True)
    # pass everything that is not a resource remark through
    sys.stderr.write("".join(l + "\n" for l in r.stderr.splitlines() if "kernel-resource-usage" not in l))
    if r.returncode != 0:
        raise subprocess.CalledProcessError(r.returncode, cmd)
    if resources:
        with open(resources, "w") as f:
            f.write(f"# source {source_hash()}\n")
            for row in resource_rows(r.stderr):
                f.write(" ".join(f"{k}={v}" for k, v in row.items()) + "\n")
    os.replace(tmp, out)
    return out


def build(out: str = LIB, extra=()) -> str:
    """The optimizer library (always) and the benchmark's stream-reference
    kernels (libstream_ref.so)."""
    _compile(STREAM_SRC, STREAM_LIB, extra)
    # roctx ranges (MTDAO_ROCTX=1) come from the rocprofiler-sdk marker library
    return _compile(SRC, out, extra, libs=("-L/opt/rocm/lib", "-lrocprofiler-sdk-roctx", "-Wl,-rpath,/opt/rocm/lib"),
                    resources=RESOURCES)


if __name__ == "__main__":
    print(build(extra=sys.argv[1:]))
