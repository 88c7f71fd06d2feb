"""mtdao_sync_stats_static (the diagnostics entry point that allocates
nothing, its scratch a static device array) against mtdao_sync_stats with
a caller buffer: bit-identical diagnostics and averaged states, on two
handles in a row, the second with a smaller input (the static scratch then
holds the first call's contents)."""

import numpy as np
import pytest
import torch

import synth
from gpu_harness import gpu_config, log
from paper_2510_05361_amd import mtdao as abi
from paper_2510_05361_amd.optimizer import MtdaoOptimizer
from synth.device import DeviceInputs

pytestmark = pytest.mark.gpu


def _pair(w, outer=None):
    d = torch.device("cuda:0")
    dev = DeviceInputs(w, d)
    a = MtdaoOptimizer(gpu_config(w, 0, outer), d, x0=dev.x0_row())
    b = MtdaoOptimizer(gpu_config(w, 0, outer), d, x0=dev.x0_row())
    return dev, a, b


def _same(p, q):
    return np.array_equal(np.isnan(p), np.isnan(q)) and np.array_equal(p[~np.isnan(p)], q[~np.isnan(q)])


@pytest.mark.parametrize("outer", [None, (0.7, 0.9)], ids=["plain", "nesterov"])
def test_static_scratch_equals_caller_scratch(outer):
    st = torch.cuda.current_stream().cuda_stream
    cases = [
        synth.small_variant(synth.WORKLOADS["adam_n3_k4_p16m"], 4_000_000, tail=8).replace(
            steps=8, period_x=2, period_u=(4, 4, 8), period_v=8),
        synth.small_variant(synth.WORKLOADS["adopt_n2_k8_p124m_bf16"], 300_000, tail=37).replace(
            steps=6, period_x=3, period_u=(2, 6), period_v=6),
    ]
    for w in cases:
        need = abi.mtdao_stats_scratch_bytes(gpu_config(w, 0, outer))
        assert need <= abi.MTDAO_STATIC_SCRATCH_BYTES
        log(f"case no-alloc {w.name} P={w.numel} K={w.replicas} scratch={need} outer={outer}")
        dev, a, b = _pair(w, outer)
        gdt = torch.bfloat16 if w.grad_dtype == "bf16" else torch.float32
        grads = torch.empty((w.replicas, w.numel), dtype=gdt, device=torch.device("cuda:0"))
        seen = 0
        for s in range(1, w.steps + 1):
            dev.grads_into(s, grads)
            a.step(grads, w.lr, w.adopt_clip_value(s))
            b.step(grads, w.lr, w.adopt_clip_value(s))
            ma, sa = a.sync_stats()
            mb, sb = abi.mtdao_sync_stats_static(b.handle, abi.MTDAO_SYNC_AUTO, st)
            assert ma == mb
            assert _same(sa, sb), (w.name, s)
            seen += bool(ma)
        torch.cuda.synchronize()
        assert seen >= 3
        for p, q in zip(a.states() + ([a.x_outer, a.x_outer_mom] if outer else []),
                        b.states() + ([b.x_outer, b.x_outer_mom] if outer else [])):
            assert torch.equal(p, q)
        a.close()
        b.close()
        del grads
        torch.cuda.empty_cache()
