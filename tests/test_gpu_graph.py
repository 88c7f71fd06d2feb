"""Graph capture of the hot path.

A window of steps -- local steps, the clip-norm pass and the averaging
events of one whole schedule period -- is captured once into a HIP graph
with torch.cuda.graph and replayed.  mtdao_local_step, mtdao_step_sync and
mtdao_sync only enqueue kernel launches on the caller's stream (no
allocation, no host wait, no memset node), so they can be captured.

Kernel arguments are frozen at capture: the per-step scalars and the masks
of the captured steps replay as they were.  A replayed window therefore
equals an eager one when neither depends on the step number -- constant
eta, SGDM or Adam without bias correction, and a window spanning a whole
number of every period -- which is what these tests check, bit for bit,
against eager calls on a second optimizer fed the same gradients, with
eager work and a synchronisation between replays.  The handle's host step
counter advances during capture, not on replay.
"""

import pytest
import torch

import oracle
import synth
from gpu_harness import log
from paper_2510_05361_amd import mtdao as abi
from paper_2510_05361_amd.optimizer import MtdaoOptimizer
from synth.device import DeviceInputs

pytestmark = pytest.mark.gpu

CASES = {
    # fused step+sync, clip-norm pass inside the graph, K=4 (wave-per-replica kernel)
    "sgdm_clip_fused": (synth.small_variant(synth.WORKLOADS["sgdm_n2_k16_p354m_clip"], 40_000, tail=37)
                        .replace(replicas=4, period_x=4, period_u=(2, 4)), True, 4),
    # separate step + sync calls, Adam without bias correction
    "adam_nobc_separate": (synth.small_variant(synth.WORKLOADS["adam_n3_k4_p16m"], 40_000, tail=40)
                           .replace(bias_correction=False, period_x=2, period_u=(4, 4, 4), period_v=4), False, 4),
}


def _window(opt, grads, w, fused, n):
    masks = []
    for _ in range(n):
        if fused:
            masks.append(opt.step_sync(grads, w.lr))
        else:
            opt.step(grads, w.lr)
            masks.append(opt.sync())
    return masks


@pytest.mark.parametrize("case", sorted(CASES))
def test_graph_replay_equals_eager(case):
    w, fused, window = CASES[case]
    log(f"case graph {case} P={w.numel} K={w.replicas} window={window}")
    d = torch.device("cuda:0")
    dev = DeviceInputs(w, d)
    cfg = abi.config_from_workload(w)
    g_opt = MtdaoOptimizer(cfg, d, x0=dev.x0_row())
    e_opt = MtdaoOptimizer(cfg, d, x0=dev.x0_row())
    grads = torch.empty((w.replicas, w.numel), dtype=torch.float32, device=d)
    dev.grads_into(1, grads)
    torch.cuda.synchronize()

    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        captured = _window(g_opt, grads, w, fused, window)
    torch.cuda.synchronize()
    # captured masks are the schedule of steps 1..window, with at least one event of every state
    ocfg = oracle.OracleConfig.from_workload(w)
    want = [oracle.schedule(ocfg, s) for s in range(1, window + 1)]
    assert captured == want
    nst = 1 + w.n_moments + (1 if w.has_v else 0)
    union = 0
    for m in want:
        union |= m
    assert union == (1 << nst) - 1

    for r in range(3):
        dev.grads_into(r + 2, grads)  # eager work between replays
        torch.cuda.synchronize()
        graph.replay()
        eager = _window(e_opt, grads, w, fused, window)
        assert eager == want
        torch.cuda.synchronize()
        for k, (a, b) in enumerate(zip(g_opt.states(), e_opt.states())):
            assert torch.equal(a, b), f"replay {r}: state {k} differs"
        log(f"  replay {r}: all {nst} states bit-identical to eager")
    del graph
    g_opt.close()
    e_opt.close()
