"""Register budget of the gfx950 kernels (CPU: reads hipcc's
kernel-resource-usage remarks; no GPU needed).

Every kernel of the library must run without scratch (a spill turns the
HBM-bound passes' register traffic into memory traffic: the fused step
with the device-side update number once spilled 36 bytes per lane and ran
its launch 6% slower), and the wave-per-replica kernels, whose K = 16
workgroups need two resident workgroups per CU, and the local step of each
benchmark workload must keep 8 waves per SIMD.

The figures come from the build (``build.py`` writes them next to the
library with a hash of the sources); when that file is missing or stale the
device code is compiled here alone.
"""

from __future__ import annotations

import os
import subprocess
import tempfile

import pytest

from paper_2510_05361_amd import build

# wave-per-replica kernels (one wavefront per replica row, K <= 16)
WAVE_KERNELS = ("k_local_step_sync_waves", "k_replica_mean_waves", "k_replica_mean_stats",
                "k_sgdm_averaged_momenta_waves")
# local step of each benchmark workload: <form, N, x type, g type, V = 4, ...
WORKLOAD_STEPS = ("k_local_stepILi0ELi3EffLi4E", "k_local_stepILi0ELi2EffLi4E", "k_local_stepILi2ELi2EffLi4E",
                  "k_local_stepILi1ELi2EttLi4E")


def _rows():
    path = build.RESOURCES
    if os.path.exists(path):
        with open(path) as f:
            head = f.readline().strip()
            body = f.read()
        if head == f"# source {build.source_hash()}":
            rows = []
            for line in body.splitlines():
                kv = dict(item.split("=", 1) for item in line.split())
                rows.append({k: (v if k == "name" else int(v)) for k, v in kv.items()})
            return rows
    if not os.path.exists(build.HIPCC):
        pytest.skip("hipcc not available")
    flags = [f for f in build.FLAGS if f not in ("-shared", "-fPIC")]
    with tempfile.TemporaryDirectory() as d:
        cmd = [build.HIPCC, *flags, "--offload-device-only", "-c", "-I", os.path.join(build.ROOT, "include"),
               "-o", os.path.join(d, "k.o"), build.SRC, build._REMARK]
        r = subprocess.run(cmd, stderr=subprocess.PIPE, text=True)
    assert r.returncode == 0, r.stderr[-2000:]
    return build.resource_rows(r.stderr)


@pytest.fixture(scope="module")
def rows():
    out = _rows()
    assert len(out) > 100, "expected the library's kernel instantiations"
    return out


def test_no_kernel_spills(rows):
    spilling = [(r["name"], r["ScratchSize"]) for r in rows if r.get("ScratchSize", 0) != 0]
    assert not spilling, spilling


# The bf16 diagnostics kernel with 16-byte slots (8 elements per lane)
# needs 68 registers: 7 waves per SIMD, which still holds three 8-wave
# workgroups per CU (K = 8); held to 64 it spilled.
EXEMPT = ("k_replica_mean_statsItLi8E",)


def test_wave_per_replica_kernels_keep_eight_waves(rows):
    low = [(r["name"], r["Occupancy"]) for r in rows
           if any(k in r["name"] for k in WAVE_KERNELS) and r["Occupancy"] < 8
           and not any(x in r["name"] for x in EXEMPT)]
    assert not low, low
    assert sum(any(k in r["name"] for k in WAVE_KERNELS) for r in rows) > 20


def test_workload_steps_keep_eight_waves(rows):
    found = [r for r in rows if any(k in r["name"] for k in WORKLOAD_STEPS)]
    assert len(found) >= len(WORKLOAD_STEPS)
    low = [(r["name"], r["Occupancy"], r["VGPRs"]) for r in found if r["Occupancy"] < 8]
    assert not low, low
