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

With the update count kept on the device (mtdao_step_sync_device, the
window closed by mtdao_device_step_advance), the step-dependent scalars --
eta_t from a schedule table, ADOPT's c_t, Adam's bias corrections -- are
formed in the kernels at every replay, so a window of Adam with bias
correction or of ADOPT replays bit-identical to eager mtdao_step_sync
calls given the same eta_t and c_t, replay after replay.
"""

import numpy as np
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


DEVICE_CASES = {
    # Adam with bias correction, periods 4 / 8 / 16: a window of 16 steps, K = 2 (fused means)
    "adam_bias_corrected": (synth.small_variant(synth.WORKLOADS["adam_n2_k2_p1m"], 60_000, tail=40), 16),
    # ADOPT, bf16 x and g, c_t from a table, K = 8, periods 2 / 4 / 4
    "adopt_bf16_ct": (synth.small_variant(synth.WORKLOADS["adopt_n2_k8_p124m_bf16"], 30_000, tail=8)
                      .replace(period_x=2, period_u=(4, 4), period_v=4), 4),
    # clipped SGDM, K = 16 (wave-per-replica fused kernel), clip-norm pass inside the graph
    "sgdm_clip_k16": (synth.small_variant(synth.WORKLOADS["sgdm_n2_k16_p354m_clip"], 40_000, tail=37)
                      .replace(period_x=4, period_u=(2, 4)), 4),
    # Adam N = 3 with bias correction, K = 4: six streams, so the fused kernel forms the
    # device-side scalars once per workgroup before its loads (the other cases form them after)
    "adam_n3_k4_early_scalars": (synth.small_variant(synth.WORKLOADS["adam_n3_k4_p16m"], 40_000, tail=13)
                                 .replace(period_x=2, period_u=(4, 4, 4), period_v=4), 4),
    # Algorithm 4's order (moments averaged inside the step), K = 5
    "sgdm_momenta_in_step": (synth.small_variant(synth.WORKLOADS["sgdm_n2_k16_p354m_clip"], 30_000, tail=8)
                             .replace(replicas=5, period_x=4, period_u=(2, 4)), 4,
                             {"sync_order": abi.MTDAO_SYNC_MOMENTA_IN_STEP}),
    # K = 17: the thread-per-column fused kernel
    "adam_k17": (synth.small_variant(synth.WORKLOADS["adam_n2_k2_p1m"], 20_000, tail=8)
                 .replace(replicas=17, period_x=4, period_u=(8, 8), period_v=8), 8),
    # Nesterov OuterOpt at every x averaging (the outer step of each replayed s runs once)
    "adam_nesterov": (synth.small_variant(synth.WORKLOADS["adam_n2_k2_p1m"], 30_000, tail=12)
                      .replace(replicas=4, period_x=2, period_u=(4, 4), period_v=4), 4,
                      {"outer_opt": abi.MTDAO_OUTER_NESTEROV, "outer_lr": 0.7, "outer_momentum": 0.9}),
    # one worker: the plain step over the row's two halves, an outer step only at x events
    "adam_k1_nesterov": (synth.small_variant(synth.WORKLOADS["adam_n2_k2_p1m"], 30_000, tail=12)
                         .replace(replicas=1, period_x=2, period_u=(4, 4), period_v=4), 4,
                         {"outer_opt": abi.MTDAO_OUTER_NESTEROV, "outer_lr": 0.7, "outer_momentum": 0.9}),
}


@pytest.mark.parametrize("case", sorted(DEVICE_CASES))
def test_graph_device_step_equals_eager(case):
    w, window, *extra = DEVICE_CASES[case]
    replays = 3
    n_total = 1 + window * (replays + 1)
    log(f"case graph device step {case} P={w.numel} K={w.replicas} window={window}")
    d = torch.device("cuda:0")
    dev = DeviceInputs(w, d)
    cfg = abi.config_from_workload(w, **(extra[0] if extra else {}))
    g_opt = MtdaoOptimizer(cfg, d, x0=dev.x0_row())
    e_opt = MtdaoOptimizer(cfg, d, x0=dev.x0_row())
    gdt = torch.bfloat16 if w.grad_dtype == "bf16" else torch.float32
    grads = torch.empty((w.replicas, w.numel), dtype=gdt, device=d)
    # a decaying eta_t schedule and ADOPT's c_t, indexed by s - 1
    lr = np.array([w.lr * (1.0 - 0.5 * k / n_total) for k in range(n_total)], dtype=np.float32)
    clip = np.array([w.adopt_clip_value(k + 1) for k in range(n_total)], dtype=np.float32)
    lr_t, clip_t = torch.from_numpy(lr).to(d), torch.from_numpy(clip).to(d)
    use_clip = w.form == "adopt"
    # update 1 on the host path on both (ADOPT's first update sets v only)
    dev.grads_into(1, grads)
    g_opt.step_sync(grads, float(lr[0]), float(clip[0]))
    e_opt.step_sync(grads, float(lr[0]), float(clip[0]))
    g_opt.device_step(lr_t, clip_t if use_clip else None)
    torch.cuda.synchronize()

    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        captured = [g_opt.step_sync_device(grads) for _ in range(window)]
        g_opt.device_step_advance()
    torch.cuda.synchronize()
    ocfg = oracle.OracleConfig.from_workload(w)
    assert captured == [oracle.schedule(ocfg, s) for s in range(2, window + 2)]
    s = 1
    for r in range(replays):
        dev.grads_into(r + 2, grads)  # eager work between replays
        torch.cuda.synchronize()
        graph.replay()
        for _ in range(window):
            s += 1
            e_opt.step_sync(grads, float(lr[s - 1]), float(clip[s - 1]) if use_clip else 0.0)
        torch.cuda.synchronize()
        for k, (a, b) in enumerate(zip(g_opt.states(), e_opt.states())):
            assert torch.equal(a, b), f"replay {r}: state {k} differs"
        if g_opt.x_outer is not None:
            assert torch.equal(g_opt.x_outer, e_opt.x_outer) and torch.equal(g_opt.x_outer_mom, e_opt.x_outer_mom)
        assert int(g_opt._dstep[0].item()) == s
        log(f"  replay {r}: steps up to {s}, every state bit-identical to eager")
    del graph
    g_opt.close()
    e_opt.close()
