"""GPU path (C ABI, gfx950 kernels) against the CPU oracle.

Small variants of every workload run their full step sequence and are
compared on every element; the full-size workloads run in the launch
configuration the benchmark times and are compared on a deterministic
element sample (each element's trajectory depends only on its own inputs
and on the per-worker clip norms, which the oracle takes over full rows).
The applied sync mask of every step must equal the oracle's bit for bit.
"""

import math

import numpy as np
import pytest
import torch

import oracle
import synth
from gpu_harness import (OracleResult, XAbsMax, compare, free, gather_state, log, run_gpu, run_oracle,
                         run_oracle_parallel)
from paper_2510_05361_amd import mtdao as abi
from paper_2510_05361_amd.optimizer import MtdaoOptimizer
from synth.device import DeviceInputs

pytestmark = pytest.mark.gpu

NAMES = list(synth.WORKLOADS)


def _steps(w, start=0):
    return list(range(start + 1, w.steps + 1))


def _aligned_tail(name: str, target: int, tail: int) -> int:
    """A tail of at least ``tail`` elements that makes the row length a
    multiple of 8 (16-byte slots for fp32 and bf16 rows) when ``tail`` is
    even, and odd (the one-element path) when ``tail`` is odd."""
    base = synth.small_variant(synth.WORKLOADS[name], target).numel
    if tail % 2:
        return tail + (base + tail + 1) % 2
    return tail + (-(base + tail)) % 8


@pytest.mark.parametrize("tail", [40, 37], ids=["aligned_tail", "odd_tail"])
@pytest.mark.parametrize("name", NAMES)
def test_small_variant_full_compare(name, tail):
    """~60k elements per replica (tens of tiles) plus a ragged tail; the
    aligned tail makes the row length a multiple of 8 (the 16-byte slots of
    every kernel), the odd tail takes the one-element path."""
    w = synth.small_variant(synth.WORKLOADS[name], 60_000, tail=_aligned_tail(name, 60_000, tail))
    assert w.numel % 8 == 0 if tail % 2 == 0 else w.numel % 2 == 1
    log(f"case small {w.name} P={w.numel} K={w.replicas} T={w.steps}")
    g = run_gpu(w, _steps(w))
    o = run_oracle(w, _steps(w))
    assert g.masks == o.masks
    assert any(g.masks)
    compare(w, g.opt, o, w.name)
    free(g)


FULL_EVERY_ELEMENT = ("adam_n2_k2_p1m", "adam_n3_k4_p16m", "adopt_n2_k8_p124m_bf16")


@pytest.mark.timeout(900)
@pytest.mark.parametrize("name", NAMES)
def test_full_size(name):
    """Every workload at its full size for all its steps, through
    mtdao_step_sync (the call and launch configuration the benchmark
    times).  The 1M, 16.8M and 124M-parameter workloads are compared on
    every element of every replica, and their separate calls
    (mtdao_local_step + mtdao_sync) must give the same states bit for bit;
    the 1.31B and 354M ones on a sample of more than 2^20 elements per
    replica: 2^20 strided columns (the unbiased subset the rms floor is
    taken over), the first and last 64 elements of every tensor and the
    columns around the flat-index and byte-offset boundaries 2^29..2^33."""
    w = synth.WORKLOADS[name]
    every = name in FULL_EVERY_ELEMENT
    idx = None if every else synth.sample_indices(w)
    log(f"case full {w.name} P={w.numel} K={w.replicas} T={w.steps} "
        f"compared={'all' if idx is None else idx.size} columns")
    g = run_gpu(w, _steps(w), fused=True)
    log("  gpu done")
    if every:
        sep = run_gpu(w, _steps(w))
        assert sep.masks == g.masks
        for p, q in zip(sep.opt.states(), g.opt.states()):
            assert torch.equal(p, q)
        free(sep)
    o = run_oracle_parallel(w, _steps(w), idx, rms_cols=None if every else synth.strided_mask(w, idx))
    assert g.masks == o.masks
    compare(w, g.opt, o, f"full-{w.name}")
    free(g)


@pytest.mark.parametrize("name", ["adam_n3_k4_p1311m", "sgdm_n2_k16_p354m_clip"])
def test_full_size_every_element_written(name):
    """Write coverage of the full-size launches, on every element of every
    replica: SGDM with N = 1, beta = 0, omega = 1, lr = 1 and no clip makes
    one update u = g and x = x0 - g exactly (one fp32 rounding, as torch's
    subtraction), so the plain step (tile placement, replica-pair windows)
    must leave exactly those values; then the standalone mean of x and u
    and a fused step with x and u due must leave every row equal to
    S^0 + (sum_{m>=1} (S^m - S^0)) / K formed in fp64 in replica order and
    rounded once (K = 4 and 16 make 1/K exact), computed here with torch."""
    base = synth.WORKLOADS[name]
    w = base.replace(form="sgdm", beta1=(0.0,), omega=(1.0,), lr=1.0, clip_rho=0.0, period_x=0, period_u=(0,),
                     period_v=0, steps=2)
    K, P = w.replicas, w.numel
    log(f"case coverage {name} P={P} K={K}")
    d = torch.device("cuda:0")
    dev = DeviceInputs(w, d)
    opt = MtdaoOptimizer(abi.config_from_workload(w), d, x0=dev.x0_row())
    grads = torch.empty((K, P), dtype=torch.float32, device=d)
    x0 = dev.x0_row()
    dev.grads_into(1, grads)
    opt.step(grads, 1.0)
    torch.cuda.synchronize()
    for m in range(K):
        assert torch.equal(opt.x[m], x0 - grads[m]), m
        assert torch.equal(opt.u[0][m], grads[m]), m

    def assert_rows_are_mean(t, rows, what):
        # rows(m, lo, hi) -> the pre-average fp32 values of row m, columns [lo, hi)
        step = 1 << 28
        for lo in range(0, P, step):
            hi = min(P, lo + step)
            s0 = rows(0, lo, hi).double()
            acc = torch.zeros_like(s0)
            for m in range(1, K):
                acc += rows(m, lo, hi).double() - s0
            want = (s0 + acc * (1.0 / K)).float()
            for m in range(K):
                assert torch.equal(t[m, lo:hi], want), (what, m, lo)

    before_x, before_u = opt.x.clone(), opt.u[0].clone()
    assert opt.sync(0b11) == 0b11
    torch.cuda.synchronize()
    assert_rows_are_mean(opt.x, lambda m, lo, hi: before_x[m, lo:hi], "mean x")
    assert_rows_are_mean(opt.u[0], lambda m, lo, hi: before_u[m, lo:hi], "mean u")
    del before_x, before_u
    xbar = opt.x[0].clone()
    dev.grads_into(2, grads)
    assert opt.step_sync(grads, 1.0, 0.0, 0b11) == 0b11
    torch.cuda.synchronize()
    assert_rows_are_mean(opt.x, lambda m, lo, hi: xbar[lo:hi] - grads[m, lo:hi], "fused x")
    assert_rows_are_mean(opt.u[0], lambda m, lo, hi: grads[m, lo:hi], "fused u")
    opt.close()
    del opt, grads, x0, xbar
    torch.cuda.empty_cache()


EDGE = {
    "one_replica": dict(replicas=1),
    "four_moments": dict(beta1=(0.0, 0.5, 0.9, 0.999), omega=(0.1, 0.2, 0.3, 0.4),
                         period_u=(1, 3, 0, 5)),
    "no_moment_weight": dict(omega=(0.0, 0.0)),
    "all_moment_weight": dict(omega=(0.25, 0.75)),
    "zero_betas": dict(beta1=(0.0, 0.0)),
    "all_periods_one": dict(period_x=1, period_u=(1, 1), period_v=1),
    "never_sync": dict(period_x=0, period_u=(0, 0), period_v=0),
}


@pytest.mark.parametrize("form", ["adam", "adopt", "sgdm"])
@pytest.mark.parametrize("edge", list(EDGE))
def test_edge_cases(form, edge):
    base = {"adam": "adam_n2_k2_p1m", "adopt": "adopt_n2_k8_p124m_bf16",
            "sgdm": "sgdm_n2_k16_p354m_clip"}[form]
    w = synth.small_variant(synth.WORKLOADS[base], 9_000, tail=12)
    kw = dict(steps=min(w.steps, 24), replicas=min(w.replicas, 4))
    kw.update(EDGE[edge])
    w = w.replace(**kw)
    if edge == "four_moments" and form == "sgdm":
        w = w.replace(omega=(0.1, 0.2, 0.3, 0.3))
    log(f"case edge {edge} {form} P={w.numel} K={w.replicas}")
    g = run_gpu(w, _steps(w))
    o = run_oracle(w, _steps(w))
    assert g.masks == o.masks
    compare(w, g.opt, o, f"{edge}-{form}")
    if edge == "all_periods_one":
        for t in g.opt.states():
            assert torch.equal(t, t[0:1].expand_as(t)), "replicas differ after an every-step sync"
    free(g)


@pytest.mark.parametrize("variant", ["adopt_cur", "f32_params_bf16_grads", "bf16_params_f32_grads",
                                     "adam_with_clip", "start_step_offset", "adam_no_bias_correction",
                                     "sgdm_clip_bf16_grads", "adopt_no_clamp"])
def test_variants(variant):
    if variant == "adam_no_bias_correction":
        w = synth.small_variant(synth.WORKLOADS["adam_n3_k4_p16m"], 30_000, tail=8).replace(
            bias_correction=False, steps=40)
    elif variant == "sgdm_clip_bf16_grads":
        w = synth.small_variant(synth.WORKLOADS["sgdm_n2_k16_p354m_clip"], 30_000, tail=16).replace(
            grad_dtype="bf16", replicas=5, steps=40)
    elif variant == "adopt_no_clamp":
        w = synth.small_variant(synth.WORKLOADS["adopt_n2_k8_p124m_bf16"], 30_000, tail=8).replace(
            adopt_clip="off", steps=40)
    elif variant == "adopt_cur":
        w = synth.small_variant(synth.WORKLOADS["adopt_n2_k8_p124m_bf16"], 30_000, tail=8).replace(
            adopt_order="cur", steps=40)
    elif variant == "f32_params_bf16_grads":
        w = synth.small_variant(synth.WORKLOADS["adam_n3_k4_p16m"], 30_000, tail=8).replace(
            grad_dtype="bf16", steps=40)
    elif variant == "bf16_params_f32_grads":
        w = synth.small_variant(synth.WORKLOADS["adopt_n2_k8_p124m_bf16"], 30_000, tail=16).replace(
            grad_dtype="f32", steps=40)
    elif variant == "adam_with_clip":
        w = synth.small_variant(synth.WORKLOADS["adam_n3_k4_p16m"], 30_000, tail=4).replace(
            clip_rho=0.05, steps=40)
    else:
        w = synth.small_variant(synth.WORKLOADS["adam_n2_k2_p1m"], 30_000).replace(steps=40)
    log(f"case variant {variant}")
    start = 1000 if variant == "start_step_offset" else 0
    g = run_gpu(w, list(range(start + 1, start + w.steps + 1)), start_step=start)
    o = run_oracle(w, list(range(start + 1, start + w.steps + 1)))
    assert g.masks == o.masks
    compare(w, g.opt, o, variant)
    free(g)


def test_zero_gradient_replica_and_zero_gradients():
    """A worker whose gradient is all zero has norm 0 and clip factor 1."""
    w = synth.small_variant(synth.WORKLOADS["sgdm_n2_k16_p354m_clip"], 20_000).replace(
        replicas=3, steps=6)
    d = torch.device("cuda:0")
    dev = DeviceInputs(w, d)
    cfg = abi.config_from_workload(w)
    opt = MtdaoOptimizer(cfg, d, x0=dev.x0_row())
    ocfg = oracle.OracleConfig.from_workload(w)
    ost = oracle.new_state(ocfg, synth.host_x0_row(w), w.replicas)
    track = XAbsMax(ost)
    grads = torch.empty((w.replicas, w.numel), dtype=torch.float32, device=d)
    for s in range(1, w.steps + 1):
        dev.grads_into(s, grads)
        grads[1].zero_()
        if s == 3:
            grads.zero_()
        hg = grads.cpu().numpy()  # built by torch from the seeded pool, not by the library
        hg2 = synth.host_grad_rows(w, s)
        hg2[1] = 0
        if s == 3:
            hg2[:] = 0
        assert np.array_equal(hg, hg2)
        opt.step(grads, w.lr)
        m = opt.sync()
        oracle.run(ocfg, ost, lambda s_: hg2, [s], lambda s_: w.lr)
        track.update(ost)
        assert m == oracle.schedule(ocfg, s)
    torch.cuda.synchronize()
    compare(w, opt, OracleResult(ost, [], None, x_absmax=[track.a], steps=w.steps), "zero-grad")
    opt.close()


def test_resume_is_bit_identical():
    """Checkpoint/resume: read every state with mtdao_read_state, destroy,
    re-init with init_states=1 and start_step=s, continue: bit-identical to
    an uninterrupted run (bias correction and schedule depend only on s)."""
    w = synth.small_variant(synth.WORKLOADS["adam_n3_k4_p16m"], 40_000, tail=8).replace(steps=70)
    d = torch.device("cuda:0")
    dev = DeviceInputs(w, d)
    full = run_gpu(w, _steps(w), dev=dev)
    cut = 37
    a = run_gpu(w.replace(steps=cut), list(range(1, cut + 1)), dev=dev)
    K, P = w.replicas, w.numel
    host = []
    for sid, t in enumerate(a.opt.states()):
        rows = np.empty((K, P), dtype=np.float32)
        for m in range(K):
            abi.mtdao_read_state(a.opt.handle, sid, m, 0, P, rows[m], torch.cuda.current_stream().cuda_stream)
        assert np.array_equal(rows, t.cpu().numpy())
        host.append(rows)
    assert abi.mtdao_step_count(a.opt.handle) == cut
    a.opt.close()
    del a
    torch.cuda.empty_cache()
    tx = torch.from_numpy(host[0]).to(d)
    tu = [torch.from_numpy(h).to(d) for h in host[1:1 + w.n_moments]]
    tv = torch.from_numpy(host[-1]).to(d)
    cfg = abi.config_from_workload(w, start_step=cut)
    opt = MtdaoOptimizer(cfg, d, resume=True, x=tx, u=tu, v=tv)
    b = run_gpu(w, list(range(cut + 1, w.steps + 1)), dev=dev, opt=opt)
    assert full.masks[cut:] == b.masks
    for p, q in zip(full.opt.states(), b.opt.states()):
        assert torch.equal(p, q)
    free(full, b)


def test_sync_idempotent_and_explicit_masks():
    w = synth.small_variant(synth.WORKLOADS["adopt_n2_k8_p124m_bf16"], 30_000, tail=8).replace(
        steps=5, period_x=0, period_u=(0, 0), period_v=0)
    g = run_gpu(w, _steps(w))
    o = run_oracle(w, _steps(w))
    ocfg = oracle.OracleConfig.from_workload(w)
    for mask in [0b0010, 0b1001, 0b1111]:
        assert g.opt.sync(mask) == mask
        before = [t.clone() for t in g.opt.states()]
        assert g.opt.sync(mask) == mask  # averaging identical rows is an exact no-op
        torch.cuda.synchronize()
        for p, q in zip(before, g.opt.states()):
            assert torch.equal(p, q)
        oracle.sync(ocfg, o.state, mask)
        compare(w, g.opt, o, f"mask{mask:04b}")
    free(g)


@pytest.mark.parametrize("tail", [40, 37], ids=["aligned_tail", "odd_tail"])
@pytest.mark.parametrize("base,K", [("adam_n3_k4_p16m", 6), ("adam_n3_k4_p16m", 10), ("adopt_n2_k8_p124m_bf16", 12),
                                    ("adam_n3_k4_p16m", 14), ("adopt_n2_k8_p124m_bf16", 10)],
                         ids=["fp32_k6", "fp32_k10", "bf16x_k12", "fp32_k14", "bf16x_k10"])
def test_mean_wave_shapes(base, K, tail):
    """The replica mean with one row per wave (K = 6) and two rows per wave
    (even K >= 8: 5 to 7 waves, so the column-to-wave assignment wraps for
    the 4 fp32 and 8 bf16 columns of a lane) against the oracle on every
    element, and bit-identical to the diagnostics pass, which averages with
    one wave per row."""
    w = synth.small_variant(synth.WORKLOADS[base], 20_000, tail=_aligned_tail(base, 20_000, tail))
    w = w.replace(replicas=K, steps=3, period_x=0, period_u=(0,) * w.n_moments, period_v=0)
    log(f"case mean shapes {w.name} P={w.numel} K={K}")
    a = run_gpu(w, _steps(w))
    b = run_gpu(w, _steps(w))
    o = run_oracle(w, _steps(w))
    full = (1 << (w.n_moments + 2)) - 1
    assert a.opt.sync(full) == full
    mb, _ = b.opt.sync_stats(full)
    assert mb == full
    oracle.sync(oracle.OracleConfig.from_workload(w), o.state, full)
    torch.cuda.synchronize()
    for p, q in zip(a.opt.states(), b.opt.states()):
        assert torch.equal(p, q)
    compare(w, a.opt, o, f"mean-K{K}")
    free(a, b)


def test_deterministic():
    """Two runs of the clipped SGDM workload are bit-identical (fixed-order
    norm reduction, no atomics)."""
    w = synth.small_variant(synth.WORKLOADS["sgdm_n2_k16_p354m_clip"], 200_000).replace(steps=20)
    a = run_gpu(w, _steps(w))
    b = run_gpu(w, _steps(w))
    for p, q in zip(a.opt.states(), b.opt.states()):
        assert torch.equal(p, q)
    free(a, b)


GUARD_CASES = {
    # clipped SGDM, separate step and sync: the norm pass, the clip finalize, the mean
    "sgdm_k5_clip_separate": (synth.small_variant(synth.WORKLOADS["sgdm_n2_k16_p354m_clip"], 30_000, tail=37)
                              .replace(replicas=5, steps=40, period_x=3, period_u=(2, 5)), {}, False, False),
    # Adam N = 3, fused step + sync with the Nesterov OuterOpt, then the diagnostics of every state
    "adam_n3_k4_fused_nesterov_stats": (synth.small_variant(synth.WORKLOADS["adam_n3_k4_p16m"], 30_000, tail=13)
                                        .replace(steps=24, period_x=2, period_u=(4, 4, 8), period_v=8),
                                        {"outer_opt": abi.MTDAO_OUTER_NESTEROV, "outer_lr": 0.7,
                                         "outer_momentum": 0.9}, True, True),
    # ADOPT with bf16 x and g, fused, then the diagnostics (the bf16 x launch included)
    "adopt_bf16_k8_fused_stats": (synth.small_variant(synth.WORKLOADS["adopt_n2_k8_p124m_bf16"], 30_000, tail=8)
                                  .replace(steps=16, period_x=2, period_u=(4, 4), period_v=4), {}, True, True),
    # Algorithm 4's order
    "sgdm_k5_momenta_in_step": (synth.small_variant(synth.WORKLOADS["sgdm_n2_k16_p354m_clip"], 30_000, tail=5)
                                .replace(replicas=5, steps=24, period_x=3, period_u=(2, 4)),
                                {"sync_order": abi.MTDAO_SYNC_MOMENTA_IN_STEP}, True, False),
    # K = 17: the thread-per-column fused kernel and mean
    "adam_k17_fused": (synth.small_variant(synth.WORKLOADS["adam_n2_k2_p1m"], 20_000, tail=8)
                       .replace(replicas=17, steps=16, period_x=2, period_u=(4, 4), period_v=8), {}, True, False),
}


@pytest.mark.parametrize("case", sorted(GUARD_CASES))
def test_guard_bands_untouched(case):
    """Canary regions around every buffer the library is given (states,
    gradients, workspace, the outer parameters and momentum, the
    diagnostics scratch) keep their contents through init, steps, syncs and
    the diagnostics: no kernel writes outside its buffers."""
    w, kw, fused, stats = GUARD_CASES[case]
    log(f"case guard bands {case} K={w.replicas} P={w.numel}")
    d = torch.device("cuda:0")
    K, P, pad = w.replicas, w.numel, 4096
    cfg = abi.config_from_workload(w, **kw)
    st = torch.cuda.current_stream().cuda_stream
    canary32 = float.fromhex("0x1.5555p-3")
    guards = []

    def guarded(n, dtype):
        fill = 0xA5 if dtype == torch.uint8 else canary32
        big = torch.full((n + 2 * pad,), fill, dtype=dtype, device=d)
        guards.append((big, n, big[0].clone()))
        return big[pad:pad + n]

    xdt = torch.bfloat16 if w.param_dtype == "bf16" else torch.float32
    gdt = torch.bfloat16 if w.grad_dtype == "bf16" else torch.float32
    x = guarded(K * P, xdt).view(K, P)
    u = [guarded(K * P, torch.float32).view(K, P) for _ in range(w.n_moments)]
    v = guarded(K * P, torch.float32).view(K, P) if w.form != "sgdm" else None
    grads = guarded(K * P, gdt).view(K, P)
    nesterov = kw.get("outer_opt") == abi.MTDAO_OUTER_NESTEROV
    xo = guarded(P, torch.float32) if nesterov else None
    mom = guarded(P, torch.float32) if nesterov else None
    dev = DeviceInputs(w, d)
    x[0].copy_(dev.x0_row().to(xdt))
    ws_bytes = abi.mtdao_workspace_bytes(cfg)
    ws = guarded(max(ws_bytes, 256), torch.uint8)
    bufs = abi.make_buffers(x.data_ptr(), [t.data_ptr() for t in u], v.data_ptr() if v is not None else None, False,
                            xo.data_ptr() if nesterov else None, mom.data_ptr() if nesterov else None)
    h = abi.mtdao_init(cfg, bufs, ws.data_ptr(), ws_bytes, st)
    try:
        for s_ in range(1, w.steps + 1):
            dev.grads_into(s_, grads)
            if fused:
                abi.mtdao_step_sync(h, grads.data_ptr(), w.lr, w.adopt_clip_value(s_), abi.MTDAO_SYNC_AUTO, st)
            else:
                abi.mtdao_local_step(h, grads.data_ptr(), w.lr, w.adopt_clip_value(s_), st)
                abi.mtdao_sync(h, abi.MTDAO_SYNC_AUTO, st)
        if stats:
            nbytes = abi.mtdao_stats_scratch_bytes(cfg)
            scratch = guarded(nbytes, torch.uint8)
            nstates = 2 + w.n_moments - (1 if w.form == "sgdm" else 0)
            abi.mtdao_sync_stats(h, (1 << nstates) - 1, scratch.data_ptr(), nbytes, st)
        torch.cuda.synchronize()
        for k, (big, n, fill) in enumerate(guards):
            assert torch.all(big[:pad] == fill) and torch.all(big[pad + n:] == fill), f"guard {k} written"
    finally:
        abi.mtdao_destroy(h)


def test_row_longer_than_2_pow_31():
    """One replica row of 2^31 + 1000 fp32 elements (64-bit indexing, ragged
    end): SGDM N=1, sampled around the 2^31 boundary and the end."""
    P = (1 << 31) + 1000
    w = synth.Workload(name="sgdm_long_row", replicas=1, form="sgdm", beta1=(0.9,), omega=(0.5,),
                       beta2=0.0, eps=0.0, lr=1e-2, clip_rho=0.0, adopt_order="prev", adopt_clip="off",
                       period_x=0, period_u=(0,), period_v=0, steps=3, param_dtype="f32",
                       grad_dtype="f32", tensors=(synth.TensorSpec("flat", P, "matrix"),),
                       grad_dist="normal", grad_std=1e-2, seed_g=1009)
    idx = np.unique(np.concatenate([np.arange(0, 64), np.arange((1 << 31) - 64, (1 << 31) + 64),
                                    np.arange(P - 64, P), np.arange(0, P, P // 4096)])).astype(np.int64)
    log(f"case long row P={P}")
    g = run_gpu(w, _steps(w))
    o = run_oracle(w, _steps(w), idx)
    compare(w, g.opt, o, "long-row")
    free(g)


# ------------------------------------------------------------ fused step + sync


def _run_fused(w, steps, start_step=0, masks=None, dev=None):
    d = torch.device("cuda:0")
    dev = dev or DeviceInputs(w, d)
    opt = MtdaoOptimizer(abi.config_from_workload(w, start_step=start_step), d, x0=dev.x0_row())
    gdt = torch.bfloat16 if w.grad_dtype == "bf16" else torch.float32
    grads = torch.empty((w.replicas, w.numel), dtype=gdt, device=d)
    applied = []
    for k, s in enumerate(steps):
        dev.grads_into(s, grads)
        m = abi.MTDAO_SYNC_AUTO if masks is None else masks[k]
        applied.append(opt.step_sync(grads, w.lr, w.adopt_clip_value(s), m))
    torch.cuda.synchronize()
    return opt, applied


@pytest.mark.parametrize("tail", [40, 37], ids=["aligned_tail", "odd_tail"])
@pytest.mark.parametrize("name", NAMES)
def test_step_sync_bit_identical_to_separate_calls(name, tail):
    """mtdao_step_sync (one fused pass) == mtdao_local_step + mtdao_sync, bit
    for bit, over every workload's full step sequence."""
    w = synth.small_variant(synth.WORKLOADS[name], 60_000, tail=_aligned_tail(name, 60_000, tail))
    log(f"case fused {w.name} P={w.numel} K={w.replicas}")
    sep = run_gpu(w, _steps(w))
    fused, applied = _run_fused(w, _steps(w))
    assert applied == sep.masks and any(applied)
    for p, q in zip(sep.opt.states(), fused.states()):
        assert torch.equal(p, q)
    fused.close()
    free(sep)


@pytest.mark.parametrize("form", ["adam", "adopt", "sgdm"])
def test_step_sync_explicit_masks_and_first_step(form):
    """Explicit masks (including every state at step 1, where ADOPT only
    initialises v), K=1 and random per-step masks: fused == separate, and
    both match the oracle."""
    base = {"adam": "adam_n3_k4_p16m", "adopt": "adopt_n2_k8_p124m_bf16", "sgdm": "sgdm_n2_k16_p354m_clip"}[form]
    w = synth.small_variant(synth.WORKLOADS[base], 20_000, tail=8).replace(steps=12, replicas=3)
    nst = 1 + w.n_moments + (1 if w.has_v else 0)
    rng = np.random.default_rng(5)
    masks = [(1 << nst) - 1] + [int(rng.integers(0, 1 << nst)) for _ in range(w.steps - 1)]
    fused, applied = _run_fused(w, _steps(w), masks=masks)
    assert applied == masks
    sep = run_gpu(w.replace(period_x=0, period_u=(0,) * w.n_moments, period_v=0), [])
    d = torch.device("cuda:0")
    dev = DeviceInputs(w, d)
    gdt = torch.bfloat16 if w.grad_dtype == "bf16" else torch.float32
    grads = torch.empty((w.replicas, w.numel), dtype=gdt, device=d)
    for s, m in zip(_steps(w), masks):
        dev.grads_into(s, grads)
        sep.opt.step(grads, w.lr, w.adopt_clip_value(s))
        assert sep.opt.sync(m) == m
    torch.cuda.synchronize()
    for p, q in zip(sep.opt.states(), fused.states()):
        assert torch.equal(p, q)
    ocfg = oracle.OracleConfig.from_workload(w)
    ost = oracle.new_state(ocfg, synth.host_x0_row(w), w.replicas)
    track = XAbsMax(ost)
    from gpu_harness import oracle_clip_scales
    for s in _steps(w):
        oracle.run(ocfg, ost, lambda s_: synth.host_grad_rows(w, s_), [s], lambda s_: w.lr,
                   w.adopt_clip_value, scales=lambda s_, g: oracle_clip_scales(w, s_),
                   masks=lambda s_: masks[s_ - 1])
        track.update(ost)
    compare(w, fused, OracleResult(ost, masks, None, x_absmax=[track.a]), f"explicit-{form}")
    fused.close()
    free(sep)


def test_step_sync_full_size_bench_workload():
    """The 1.31B-parameter K=4 workload through the fused entry point over a
    window that contains x-, u- and v-averaging (steps 249..256 after a
    resume at 248 from seeded per-worker states), sampled against the
    oracle from the same states."""
    w = synth.WORKLOADS["adam_n3_k4_p1311m"]
    start = 248
    d = torch.device("cuda:0")
    dev = DeviceInputs(w, d)
    K, P = w.replicas, w.numel
    x = torch.empty((K, P), dtype=torch.float32, device=d)
    dev.pool_rows_into(11, 0.02, x)
    u = [torch.empty((K, P), dtype=torch.float32, device=d) for _ in range(3)]
    for j, t in enumerate(u):
        dev.pool_rows_into(12 + j, 1e-3, t)
    v = torch.empty((K, P), dtype=torch.float32, device=d)
    dev.pool_rows_into(15, 1e-6, v, absolute=True)
    opt = MtdaoOptimizer(abi.config_from_workload(w, start_step=start), d, resume=True, x=x, u=u, v=v)
    grads = torch.empty((K, P), dtype=torch.float32, device=d)
    applied = []
    for s in range(start + 1, w.steps + 1):
        dev.grads_into(s, grads)
        applied.append(opt.step_sync(grads, w.lr))
    torch.cuda.synchronize()
    idx = synth.sample_indices(w)
    o = run_oracle_parallel(
        w, range(start + 1, w.steps + 1), idx, rms_cols=synth.strided_mask(w, idx),
        init=lambda c: oracle.OracleState(synth.host_pool_rows(w, 11, 0.02, c),
                                          [synth.host_pool_rows(w, 12 + j, 1e-3, c) for j in range(3)],
                                          synth.host_pool_rows(w, 15, 1e-6, c, absolute=True)))
    assert applied == o.masks == [0] * 7 + [0b11111]
    compare(w, opt, o, "fused-full")
    opt.close()
    del x, u, v, grads
    torch.cuda.empty_cache()


# ------------------------------------------------------------ probabilistic variant (Algorithm 4)


def _run_prob_gpu(w, steps, masks, dev=None):
    d = torch.device("cuda:0")
    dev = dev or DeviceInputs(w, d)
    cfg = abi.config_from_workload(w, sync_order=abi.MTDAO_SYNC_MOMENTA_IN_STEP)
    opt = MtdaoOptimizer(cfg, d, x0=dev.x0_row())
    gdt = torch.bfloat16 if w.grad_dtype == "bf16" else torch.float32
    grads = torch.empty((w.replicas, w.numel), dtype=gdt, device=d)
    applied = []
    for s, m in zip(steps, masks):
        dev.grads_into(s, grads)
        applied.append(opt.step_sync(grads, w.lr, 0.0, m))
    torch.cuda.synchronize()
    return opt, applied


def _prob_workload(name, **kw):
    w = synth.WORKLOADS["sgdm_n2_k16_p354m_clip"]
    # Algorithm 4: sum of omega = 1, the gradient entering as a beta = 0 momentum
    w = w.replace(beta1=(0.0, 0.99), omega=(0.3, 0.7), clip_rho=0.0, period_x=0, period_u=(0, 0), **kw)
    return w if name == "full" else synth.small_variant(w, 60_000, tail=37 if name == "odd" else 40)


@pytest.mark.parametrize("size", ["aligned", "odd", "full", "k17", "bf16"])
def test_probabilistic_sync_against_oracle(size):
    """Bernoulli averaging events (p_x = 1/16, p_u = 1/4, 1/32; drawn on the
    host) through mtdao_step_sync with the averaged-momenta order, against
    the oracle's Algorithm 4 on the same events.  K = 16 runs the
    wave-per-replica kernel, K = 17 the thread-per-column one; "bf16" takes
    bf16 parameters and gradients."""
    extra = {"k17": {"replicas": 17}, "bf16": {"param_dtype": "bf16", "grad_dtype": "bf16"}}.get(size, {})
    w = _prob_workload(size, steps=40 if size == "full" else 64, **extra)
    masks = synth.bernoulli_masks(123, w.steps, 2, 1 / 16, (1 / 4, 1 / 32))
    assert any(m & 0b010 for m in masks) and any(m & 1 for m in masks)
    log(f"case prob {size} P={w.numel} K={w.replicas} masks={sum(1 for m in masks if m)}")
    opt, applied = _run_prob_gpu(w, _steps(w), masks)
    assert applied == masks
    idx = synth.sample_indices(w) if size == "full" else None
    ocfg = oracle.OracleConfig.from_workload(w)
    ost = oracle.new_state(ocfg, synth.host_x0_row(w, idx), w.replicas)
    track = XAbsMax(ost)
    for s in _steps(w):
        oracle.run_probabilistic(ocfg, ost, lambda s_: synth.host_grad_rows(w, s_, idx), [s],
                                 lambda s_: w.lr, lambda s_: masks[s_ - 1])
        track.update(ost)
    compare(w, opt, OracleResult(ost, masks, idx, rms_cols=None if idx is None else synth.strided_mask(w, idx),
                                 x_absmax=[track.a]), f"prob-{size}")
    opt.close()
    torch.cuda.empty_cache()


def test_probabilistic_order_x_only_equals_standard_order():
    """With only x events the two orders coincide bit for bit; with every
    moment averaged at every step all replicas stay identical."""
    w = _prob_workload("aligned", steps=20, replicas=5)
    masks = [1 if s % 3 == 0 else 0 for s in _steps(w)]
    a, _ = _run_prob_gpu(w, _steps(w), masks)
    b, _ = _run_fused(w, _steps(w), masks=masks)
    for p, q in zip(a.states(), b.states()):
        assert torch.equal(p, q)
    c, _ = _run_prob_gpu(w, _steps(w), [0b110] * w.steps)
    assert torch.equal(c.x, c.x[0:1].expand_as(c.x))
    for o in (a, b, c):
        o.close()


# ------------------------------------------------------------ Nesterov OuterOpt

NESTEROV = (0.7, 0.9)


@pytest.mark.parametrize("name", ["adam_n3_k4_p16m", "adopt_n2_k8_p124m_bf16", "sgdm_n2_k16_p354m_clip"])
@pytest.mark.parametrize("fused", [False, True], ids=["separate", "fused"])
def test_outer_nesterov_against_oracle(name, fused):
    """Nesterov OuterOpt at every averaging event of x, through the separate
    and the fused entry points, against the oracle (x, moments, outer
    parameters and outer momentum)."""
    w = synth.small_variant(synth.WORKLOADS[name], 40_000, tail=8)
    w = w.replace(steps=min(w.steps, 96), period_x=max(2, w.period_x // 8))
    log(f"case nesterov {w.name} fused={fused} period_x={w.period_x}")
    g = run_gpu(w, _steps(w), outer=NESTEROV, fused=fused)
    o = run_oracle(w, _steps(w), outer=NESTEROV)
    assert g.masks == o.masks and sum(m & 1 for m in g.masks) >= 4
    compare(w, g.opt, o, f"nesterov-{name}-{fused}")
    assert torch.equal(g.opt.x, g.opt.x[0:1].expand_as(g.opt.x)) or (g.masks[-1] & 1) == 0
    free(g)


def test_outer_nesterov_fused_bit_identical_and_resume():
    w = synth.small_variant(synth.WORKLOADS["adam_n3_k4_p16m"], 40_000, tail=8).replace(
        steps=70, period_x=8)
    d = torch.device("cuda:0")
    dev = DeviceInputs(w, d)
    a = run_gpu(w, _steps(w), outer=NESTEROV, dev=dev)
    b = run_gpu(w, _steps(w), outer=NESTEROV, dev=dev, fused=True)
    assert a.masks == b.masks
    for p, q in zip(a.opt.states() + [a.opt.x_outer, a.opt.x_outer_mom],
                    b.opt.states() + [b.opt.x_outer, b.opt.x_outer_mom]):
        assert torch.equal(p, q)
    # resume: read the outer states through mtdao_read_state, restart at s = 40
    cut = 40
    c = run_gpu(w, list(range(1, cut + 1)), outer=NESTEROV, dev=dev)
    st = torch.cuda.current_stream().cuda_stream
    xo = np.empty(w.numel, dtype=np.float32)
    xm = np.empty(w.numel, dtype=np.float32)
    abi.mtdao_read_state(c.opt.handle, abi.MTDAO_STATE_X_OUTER, 0, 0, w.numel, xo, st)
    abi.mtdao_read_state(c.opt.handle, abi.MTDAO_STATE_OUTER_MOM, 0, 0, w.numel, xm, st)
    assert np.array_equal(xo, c.opt.x_outer.cpu().numpy()) and np.array_equal(xm, c.opt.x_outer_mom.cpu().numpy())
    with pytest.raises(abi.MtdaoError):
        abi.mtdao_read_state(c.opt.handle, abi.MTDAO_STATE_X_OUTER, 1, 0, 4, xo, st)
    from gpu_harness import gpu_config
    opt = MtdaoOptimizer(gpu_config(w, cut, NESTEROV), d, resume=True, x=c.opt.x.clone(),
                         u=[t.clone() for t in c.opt.u], v=c.opt.v.clone(),
                         x_outer=torch.from_numpy(xo).to(d), x_outer_mom=torch.from_numpy(xm).to(d))
    r = run_gpu(w, list(range(cut + 1, w.steps + 1)), dev=dev, opt=opt)
    for p, q in zip(a.opt.states() + [a.opt.x_outer, a.opt.x_outer_mom],
                    r.opt.states() + [r.opt.x_outer, r.opt.x_outer_mom]):
        assert torch.equal(p, q)
    free(a, b, c, r)


@pytest.mark.parametrize("name,K", [("adam_n3_k4_p16m", 4), ("adopt_n2_k8_p124m_bf16", 8), ("adam_n3_k4_p16m", 1)],
                         ids=["fp32_k4", "bf16x_k8", "fp32_k1"])
@pytest.mark.parametrize("fused", [False, True], ids=["separate", "fused"])
def test_outer_nesterov_repeated_averaging_changes_nothing(name, K, fused):
    """Under the Nesterov OuterOpt the outer step runs once per step s: after
    the averaging of x at s (fused or separate), a second mtdao_sync, a
    mtdao_sync_stats and a third mtdao_sync at the same s leave x, the outer
    parameters and the outer momentum bit for bit as they were, and the
    states still equal the oracle's (which takes one outer step per event).
    The repeated diagnostics of x are those of pseudo-gradients that are
    all zero (fp32) or the rounding residual x_outer - bf16(x_outer)."""
    w = synth.small_variant(synth.WORKLOADS[name], 20_000, tail=8).replace(replicas=K, steps=8, period_x=4)
    log(f"case nesterov repeat {w.name} K={K} fused={fused}")
    g = run_gpu(w, _steps(w), outer=NESTEROV, fused=fused)
    assert g.masks[-1] & 1
    keep = [t.clone() for t in g.opt.states() + [g.opt.x_outer, g.opt.x_outer_mom]]
    assert g.opt.sync(1) == 1
    mask, stats = g.opt.sync_stats(1) if K <= 16 else (1, None)
    assert mask == 1
    assert g.opt.sync(abi.MTDAO_SYNC_AUTO) & 1
    torch.cuda.synchronize()
    for p, q in zip(keep, g.opt.states() + [g.opt.x_outer, g.opt.x_outer_mom]):
        assert torch.equal(p, q)
    if w.param_dtype == "f32":
        assert stats[0][abi.MTDAO_STAT_MEAN_SQ] == 0.0 and stats[0][abi.MTDAO_STAT_VARIANCE] == 0.0
    o = run_oracle(w, _steps(w), outer=NESTEROV)
    compare(w, g.opt, o, f"nesterov-repeat-{name}-{K}-{fused}")
    free(g)


def test_outer_nesterov_unit_lr_is_averaging():
    """outer_lr = 1, momentum 0 restarts every worker from the mean."""
    w = synth.small_variant(synth.WORKLOADS["sgdm_n2_k16_p354m_clip"], 30_000).replace(steps=48)
    a = run_gpu(w, _steps(w))
    b = run_gpu(w, _steps(w), outer=(1.0, 0.0))
    from gpu_harness import rel_err
    for p, q in zip(a.opt.states(), b.opt.states()):
        assert rel_err(q.cpu().numpy(), p.cpu().numpy()) < 1e-6
    free(a, b)


def test_outer_nesterov_full_size_bench_workload():
    """The 1.31B-parameter K=4 workload with the Nesterov OuterOpt through
    the fused entry point over 128 steps (x averaged at 64 and 128),
    sampled against the oracle."""
    w = synth.WORKLOADS["adam_n3_k4_p1311m"].replace(steps=128)
    idx = synth.sample_indices(w)
    g = run_gpu(w, _steps(w), outer=NESTEROV, fused=True)
    o = run_oracle_parallel(w, _steps(w), idx, outer=NESTEROV, rms_cols=synth.strided_mask(w, idx))
    assert g.masks == o.masks
    # the outer rows are [P]; they are compared on the same columns
    compare(w, g.opt, o, "nesterov-full")
    free(g)


# ------------------------------------------------------------ averaging diagnostics


def _stats_case(name, outer=None, steps=None, tail=8):
    w = synth.small_variant(synth.WORKLOADS[name], 50_000, tail=tail)
    w = w.replace(replicas=min(w.replicas, 16), steps=steps or w.steps)
    return w


@pytest.mark.parametrize("name,outer,tail", [("adam_n3_k4_p16m", None, 8), ("adopt_n2_k8_p124m_bf16", None, 8),
                                             ("sgdm_n2_k16_p354m_clip", None, 8), ("adam_n3_k4_p16m", (0.7, 0.9), 8),
                                             ("adopt_n2_k8_p124m_bf16", (0.7, 0.9), 8), ("adam_n3_k4_p16m", None, 37),
                                             ("adopt_n2_k8_p124m_bf16", (0.7, 0.9), 37)],
                         ids=["adam", "adopt_bf16", "sgdm_k16", "adam_nesterov", "adopt_bf16_nesterov", "adam_odd",
                              "adopt_bf16_nesterov_odd"])
def test_sync_stats_against_oracle(name, outer, tail):
    """mtdao_sync_stats: averaged states bit-identical to mtdao_sync, and the
    diagnostics of every averaged state equal the oracle's on the same
    pre-average values (fp32: 1e-5 relative; bf16 x: rounding flips of x
    shift the worker differences by a bf16 ulp, bound 2e-3).  An odd tail
    takes the one-element-per-lane path."""
    w = _stats_case(name, tail=tail)
    w = w.replace(period_x=4, period_u=(6,) * w.n_moments, period_v=8, steps=24)
    log(f"case stats {w.name} K={w.replicas} outer={outer}")
    d = torch.device("cuda:0")
    dev = DeviceInputs(w, d)
    from gpu_harness import gpu_config, oracle_cfg
    a = MtdaoOptimizer(gpu_config(w, 0, outer), d, x0=dev.x0_row())
    b = MtdaoOptimizer(gpu_config(w, 0, outer), d, x0=dev.x0_row())
    ocfg = oracle_cfg(w, outer)
    ost = oracle.new_state(ocfg, synth.host_x0_row(w), w.replicas)
    track = XAbsMax(ost)
    gdt = torch.bfloat16 if w.grad_dtype == "bf16" else torch.float32
    grads = torch.empty((w.replicas, w.numel), dtype=gdt, device=d)
    checked = 0
    for s in _steps(w):
        dev.grads_into(s, grads)
        a.step(grads, w.lr, w.adopt_clip_value(s))
        b.step(grads, w.lr, w.adopt_clip_value(s))
        ma = a.sync()
        mb, stats = b.sync_stats()
        oracle.local_step(ocfg, ost, synth.host_grad_rows(w, s), s, w.lr, w.adopt_clip_value(s),
                          oracle.clip_scales(ocfg, synth.host_grad_rows(w, s)))
        track.update(ost)
        ostats = oracle.sync_stats(ocfg, ost, oracle.schedule(ocfg, s))
        track.update(ost)
        assert ma == mb == oracle.schedule(ocfg, s)
        for sid in range(abi.MTDAO_MAX_N + 2):
            if sid not in ostats:
                assert np.all(np.isnan(stats[sid])), (s, sid)
                continue
            K = w.replicas
            got = np.concatenate([stats[sid][:3], stats[sid][4:4 + K], stats[sid][20:20 + K]])
            want = np.concatenate([ostats[sid][:3], ostats[sid][4:4 + K], ostats[sid][4 + K:4 + 2 * K]])
            tol = 2e-3 if (sid == 0 and w.param_dtype == "bf16") else 1e-5
            scale = np.maximum(np.abs(want), np.abs(want).max() * 1e-6)
            err = np.max(np.abs(got - want) / scale)
            assert err <= tol, (s, sid, err, got[:3], want[:3])
            checked += 1
    torch.cuda.synchronize()
    assert checked >= 6
    for p, q in zip(a.states(), b.states()):
        assert torch.equal(p, q)
    if outer is not None:
        assert torch.equal(a.x_outer, b.x_outer) and torch.equal(a.x_outer_mom, b.x_outer_mom)
    compare(w, b, OracleResult(ost, [], None, x_absmax=[track.a], steps=w.steps), f"stats-{name}")
    a.close()
    b.close()


@pytest.mark.parametrize("outer", [None, (0.7, 0.9)], ids=["plain", "nesterov"])
def test_sync_stats_full_size_multi_chunk(outer):
    """mtdao_sync_stats on the full 16.8M-parameter K=4 workload, where the
    workgroup sums span several chunks of both reduction levels: every
    state's diagnostics against the oracle on all elements, and the averaged
    states bit-identical to mtdao_sync."""
    w = synth.WORKLOADS["adam_n3_k4_p16m"].replace(steps=4, period_x=2, period_u=(2, 4, 4), period_v=4)
    log(f"case stats full P={w.numel} K={w.replicas} outer={outer}")
    d = torch.device("cuda:0")
    dev = DeviceInputs(w, d)
    from gpu_harness import gpu_config, oracle_cfg
    a = MtdaoOptimizer(gpu_config(w, 0, outer), d, x0=dev.x0_row())
    b = MtdaoOptimizer(gpu_config(w, 0, outer), d, x0=dev.x0_row())
    ocfg = oracle_cfg(w, outer)
    ost = oracle.new_state(ocfg, synth.host_x0_row(w), w.replicas)
    grads = torch.empty((w.replicas, w.numel), dtype=torch.float32, device=d)
    K = w.replicas
    checked = 0
    for s in _steps(w):
        dev.grads_into(s, grads)
        a.step(grads, w.lr)
        b.step(grads, w.lr)
        ma = a.sync()
        mb, stats = b.sync_stats()
        g = synth.host_grad_rows(w, s)
        oracle.local_step(ocfg, ost, g, s, w.lr, 0.0, None)
        ostats = oracle.sync_stats(ocfg, ost, oracle.schedule(ocfg, s))
        assert ma == mb == oracle.schedule(ocfg, s)
        for sid, want_row in ostats.items():
            got = np.concatenate([stats[sid][:3], stats[sid][4:4 + K], stats[sid][20:20 + K]])
            want = np.concatenate([want_row[:3], want_row[4:4 + K], want_row[4 + K:4 + 2 * K]])
            scale = np.maximum(np.abs(want), np.abs(want).max() * 1e-6)
            err = np.max(np.abs(got - want) / scale)
            assert err <= 1e-5, (s, sid, err)
            checked += 1
    torch.cuda.synchronize()
    assert checked >= 6
    for p, q in zip(a.states(), b.states()):
        assert torch.equal(p, q)
    a.close()
    b.close()
    torch.cuda.empty_cache()


@pytest.mark.parametrize("fused", [False, True], ids=["separate", "fused"])
def test_outer_nesterov_single_replica(fused):
    """K = 1: averaging is the identity, but the Nesterov outer step still
    moves the outer parameters and restarts the worker from them."""
    w = synth.small_variant(synth.WORKLOADS["adam_n3_k4_p16m"], 20_000, tail=4).replace(
        replicas=1, steps=24, period_x=3)
    g = run_gpu(w, _steps(w), outer=NESTEROV, fused=fused)
    o = run_oracle(w, _steps(w), outer=NESTEROV)
    assert g.masks == o.masks
    compare(w, g.opt, o, f"nesterov-k1-{fused}")
    avg = run_gpu(w, _steps(w), fused=fused)
    assert not torch.equal(avg.opt.x, g.opt.x), "the outer step must act at K = 1"
    free(g, avg)


# ------------------------------------------------------------ degenerate sizes


@pytest.mark.parametrize("P,K", [(1, 3), (3, 2), (63, 5), (64, 4), (1029, 17), (200, 1024)],
                         ids=["one_element", "three", "below_a_wave", "one_wave", "k17_thread_fused", "k_max"])
@pytest.mark.parametrize("form", ["adam", "adopt", "sgdm"])
def test_degenerate_sizes(P, K, form):
    """Tiny rows (one element, shorter than a wavefront), K = 17 (the fused
    kernel that walks the replicas per thread) and K = MTDAO_MAX_REPLICAS:
    separate and fused entry points against the oracle, bit-identical to
    each other."""
    base = {"adam": "adam_n3_k4_p16m", "adopt": "adopt_n2_k8_p124m_bf16", "sgdm": "sgdm_n2_k16_p354m_clip"}[form]
    w = synth.WORKLOADS[base].replace(tensors=(synth.TensorSpec("t", P, "matrix"),), replicas=K, steps=10,
                                      period_x=2, period_u=(3,) * synth.WORKLOADS[base].n_moments, period_v=5)
    g = run_gpu(w, _steps(w))
    f = run_gpu(w, _steps(w), fused=True)
    o = run_oracle(w, _steps(w))
    assert g.masks == f.masks == o.masks
    compare(w, g.opt, o, f"tiny-{form}-{P}-{K}")
    for p, q in zip(g.opt.states(), f.opt.states()):
        assert torch.equal(p, q)
    free(g, f)


# ------------------------------------------------------------ seeded random configurations

def _random_workload(seed: int):
    """A small configuration drawn from seed: form, N, betas, omegas (the
    gradient weight 1 - sum omega sometimes exactly 0), K (1 to 17), storage
    types, ADOPT order, bias correction, clip, periods (0 = never, 1 =
    every step) and a ragged row tail."""
    rng = np.random.Generator(np.random.PCG64(9000 + seed))
    form = ["adam", "adopt", "sgdm"][seed % 3]
    base = {"adam": "adam_n3_k4_p16m", "adopt": "adopt_n2_k8_p124m_bf16", "sgdm": "sgdm_n2_k16_p354m_clip"}[form]
    n = int(rng.integers(1, 5))
    beta1 = tuple(float(b) for b in np.sort(rng.choice([0.0, 0.5, 0.9, 0.95, 0.99, 0.995, 0.999], n, replace=False)))
    total = 1.0 if rng.random() < 0.25 else float(rng.uniform(0.3, 0.95))
    wts = rng.uniform(0.1, 1.0, n)
    omega = tuple(float(np.float32(total * x / wts.sum())) for x in wts)
    periods = [0, 1, 2, 3, 5]
    kw = dict(replicas=int(rng.choice([1, 2, 3, 5, 8, 12, 16, 17])), beta1=beta1, omega=omega, steps=12,
              param_dtype=str(rng.choice(["f32", "bf16"])), grad_dtype=str(rng.choice(["f32", "bf16"])),
              period_x=int(rng.choice(periods)), period_u=tuple(int(rng.choice(periods)) for _ in range(n)),
              period_v=int(rng.choice(periods)), start_step=0)
    if form == "adopt":
        kw.update(adopt_order=str(rng.choice(["prev", "cur"])), clip_rho=0.0)
    else:
        kw.update(clip_rho=float(rng.choice([0.0, 1.0])))
    if form == "adam":
        kw.update(bias_correction=bool(rng.random() < 0.7))
    kw.pop("start_step")
    tail = int(rng.choice([0, 1, 7, 37, 40]))
    w = synth.small_variant(synth.WORKLOADS[base], int(rng.integers(3_000, 20_000)), tail=tail)
    fused = bool(rng.random() < 0.5)
    outer = None
    if kw["period_x"] > 0 and rng.random() < 0.3:
        # lr (1 + mu) / (1 - mu) <= 15.2 stays within the bf16 outer bound
        outer = (float(np.float32(rng.uniform(0.5, 0.8))), float(np.float32(rng.choice([0.0, 0.5, 0.9]))))
    return w.replace(**kw), fused, outer


@pytest.mark.parametrize("seed", range(48))
def test_random_configs(seed):
    """Seeded random small configurations (some with the Nesterov OuterOpt)
    through the separate or the fused entry points, every element against
    the oracle and the applied masks bit for bit."""
    w, fused, outer = _random_workload(seed)
    log(f"case random {seed} {w.form} N={w.n_moments} K={w.replicas} P={w.numel} x={w.param_dtype} "
        f"g={w.grad_dtype} periods={w.period_x}/{w.period_u}/{w.period_v} clip={w.clip_rho} fused={fused} "
        f"outer={outer}")
    g = run_gpu(w, _steps(w), fused=fused, outer=outer)
    o = run_oracle(w, _steps(w), outer=outer)
    assert g.masks == o.masks
    compare(w, g.opt, o, f"random{seed}")
    free(g)


@pytest.mark.parametrize("seed", range(16))
def test_random_probabilistic(seed):
    """Algorithm 4 on seeded random SGDM configurations: N, betas (beta_1 = 0
    in half of them, the gradient as a momentum), omegas, K (2 to 17),
    storage types, clip, and Bernoulli events with drawn probabilities,
    through mtdao_step_sync against the oracle's Algorithm 4."""
    rng = np.random.Generator(np.random.PCG64(7000 + seed))
    n = int(rng.integers(1, 5))
    beta1 = tuple(float(b) for b in np.sort(rng.choice([0.5, 0.9, 0.95, 0.99, 0.999], n, replace=False)))
    if rng.random() < 0.5:
        beta1 = (0.0,) + beta1[1:]
    total = 1.0 if rng.random() < 0.5 else float(rng.uniform(0.4, 0.95))
    wts = rng.uniform(0.1, 1.0, n)
    omega = tuple(float(np.float32(total * x / wts.sum())) for x in wts)
    w = synth.small_variant(synth.WORKLOADS["sgdm_n2_k16_p354m_clip"], int(rng.integers(3_000, 20_000)),
                            tail=int(rng.choice([0, 1, 7, 37, 40])))
    w = w.replace(replicas=int(rng.choice([2, 3, 5, 8, 12, 16, 17])), beta1=beta1, omega=omega, steps=24,
                  period_x=0, period_u=(0,) * n, clip_rho=float(rng.choice([0.0, 1.0])),
                  param_dtype=str(rng.choice(["f32", "bf16"])), grad_dtype=str(rng.choice(["f32", "bf16"])))
    p_x = float(rng.choice([0.0, 0.1, 0.3]))
    p_u = tuple(float(rng.choice([0.05, 0.25, 0.5, 1.0])) for _ in range(n))
    masks = synth.bernoulli_masks(7100 + seed, w.steps, n, p_x, p_u)
    log(f"case random prob {seed} N={n} K={w.replicas} P={w.numel} x={w.param_dtype} g={w.grad_dtype} "
        f"beta={beta1} clip={w.clip_rho} events={sum(1 for m in masks if m)}")
    opt, applied = _run_prob_gpu(w, _steps(w), masks)
    assert applied == masks
    ocfg = oracle.OracleConfig.from_workload(w)
    ost = oracle.new_state(ocfg, synth.host_x0_row(w), w.replicas)
    track = XAbsMax(ost)
    for s in _steps(w):
        oracle.run_probabilistic(ocfg, ost, lambda s_: synth.host_grad_rows(w, s_), [s],
                                 lambda s_: w.lr, lambda s_: masks[s_ - 1])
        track.update(ost)
    compare(w, opt, OracleResult(ost, masks, None, x_absmax=[track.a]), f"random-prob{seed}")
    opt.close()
    torch.cuda.empty_cache()


@pytest.mark.parametrize("seed", range(16))
def test_random_sync_stats(seed):
    """mtdao_sync_stats on seeded random configurations (K up to 16, some
    with the Nesterov OuterOpt): after a few local steps every state is
    averaged with its diagnostics; the diagnostics against the oracle's and
    the averaged states bit-identical to mtdao_sync."""
    w, _, outer = _random_workload(100 + seed)
    w = w.replace(replicas=min(w.replicas, 16), steps=5, period_x=0, period_u=(0,) * w.n_moments, period_v=0)
    log(f"case random stats {seed} {w.form} N={w.n_moments} K={w.replicas} P={w.numel} x={w.param_dtype} "
        f"outer={outer}")
    from gpu_harness import gpu_config, oracle_cfg
    d = torch.device("cuda:0")
    dev = DeviceInputs(w, d)
    a = MtdaoOptimizer(gpu_config(w, 0, outer), d, x0=dev.x0_row())
    b = MtdaoOptimizer(gpu_config(w, 0, outer), d, x0=dev.x0_row())
    ocfg = oracle_cfg(w, outer)
    ost = oracle.new_state(ocfg, synth.host_x0_row(w), w.replicas)
    gdt = torch.bfloat16 if w.grad_dtype == "bf16" else torch.float32
    grads = torch.empty((w.replicas, w.numel), dtype=gdt, device=d)
    for s in _steps(w):
        dev.grads_into(s, grads)
        a.step(grads, w.lr, w.adopt_clip_value(s))
        b.step(grads, w.lr, w.adopt_clip_value(s))
        g = synth.host_grad_rows(w, s)
        oracle.local_step(ocfg, ost, g, s, w.lr, w.adopt_clip_value(s), oracle.clip_scales(ocfg, g))
    full = (1 << (w.n_moments + (2 if w.has_v else 1))) - 1
    assert a.sync(full) == full
    mb, stats = b.sync_stats(full)
    assert mb == full
    ostats = oracle.sync_stats(ocfg, ost, full)
    K = w.replicas
    for sid, want_row in ostats.items():
        got = np.concatenate([stats[sid][:3], stats[sid][4:4 + K], stats[sid][20:20 + K]])
        want = np.concatenate([want_row[:3], want_row[4:4 + K], want_row[4 + K:4 + 2 * K]])
        tol = 2e-3 if (sid == 0 and w.param_dtype == "bf16") else 1e-5
        scale = np.maximum(np.abs(want), np.abs(want).max() * 1e-6)
        err = np.max(np.abs(got - want) / scale)
        assert err <= tol, (sid, err, got[:3], want[:3])
    torch.cuda.synchronize()
    for p, q in zip(a.states(), b.states()):
        assert torch.equal(p, q)
    if outer is not None:
        assert torch.equal(a.x_outer, b.x_outer) and torch.equal(a.x_outer_mom, b.x_outer_mom)
    a.close()
    b.close()
    torch.cuda.empty_cache()


@pytest.mark.parametrize("name,k,fused", [("adam_n3_k4_p16m", 5, False), ("adam_n3_k4_p16m", -3, True),
                                          ("adopt_n2_k8_p124m_bf16", 4, False), ("adopt_n2_k8_p124m_bf16", -2, True)],
                         ids=["adam_up", "adam_down_fused", "adopt_bf16_up", "adopt_bf16_down_fused"])
def test_power_of_two_gradient_scale_invariance(name, k, fused):
    """With eps = 0, scaling every gradient by 2^k leaves the Adam and ADOPT
    trajectories of x unchanged bit for bit on the GPU (averaging events
    included): v scales by 4^k, Adam's u by 2^k, ADOPT's u not at all,
    because a power-of-two scale commutes with every fp32 rounding, the
    square root and the division.  No oracle is involved."""
    w = synth.small_variant(synth.WORKLOADS[name], 30_000, tail=8)
    w = w.replace(eps=0.0, steps=24, period_x=4, period_u=(6,) * w.n_moments, period_v=8)
    log(f"case scale {w.name} k={k} fused={fused}")
    d = torch.device("cuda:0")
    dev = DeviceInputs(w, d)
    gdt = torch.bfloat16 if w.grad_dtype == "bf16" else torch.float32
    grads = torch.empty((w.replicas, w.numel), dtype=gdt, device=d)
    opts = []
    for scale in (1.0, 2.0 ** k):
        opt = MtdaoOptimizer(abi.config_from_workload(w), d, x0=dev.x0_row())
        for s in _steps(w):
            dev.grads_into(s, grads)
            grads.mul_(scale)
            if fused:
                opt.step_sync(grads, w.lr, w.adopt_clip_value(s))
            else:
                opt.step(grads, w.lr, w.adopt_clip_value(s))
                opt.sync()
        opts.append(opt)
    torch.cuda.synchronize()
    a, b = opts
    assert torch.equal(a.x, b.x)
    u_scale = 2.0 ** k if w.form == "adam" else 1.0
    for ua, ub in zip(a.u, b.u):
        assert torch.equal(ua * u_scale, ub)
    assert torch.equal(a.v * 4.0 ** k, b.v)
    a.close()
    b.close()


@pytest.mark.parametrize("name", ["adam_n3_k4_p16m", "adopt_n2_k8_p124m_bf16", "sgdm_n2_k16_p354m_clip"])
def test_identical_workers_equal_one_worker(name):
    """K workers that all receive worker 0's gradient follow, bit for bit,
    the trajectory of a single worker: averaging identical rows is an exact
    no-op, the clip norms agree, and the K = 1 launch shapes (half-row
    windows, no averaging) compute the same per-element arithmetic as the
    replica-pair windows and the averaging kernels.  No oracle is involved."""
    w = synth.small_variant(synth.WORKLOADS[name], 30_000, tail=37)
    w = w.replace(replicas=6, steps=20, period_x=3, period_u=(4,) * w.n_moments, period_v=5)
    log(f"case identical workers {w.name}")
    d = torch.device("cuda:0")
    dev = DeviceInputs(w, d)
    gdt = torch.bfloat16 if w.grad_dtype == "bf16" else torch.float32
    grads = torch.empty((w.replicas, w.numel), dtype=gdt, device=d)
    many = MtdaoOptimizer(abi.config_from_workload(w), d, x0=dev.x0_row())
    one = MtdaoOptimizer(abi.config_from_workload(w.replace(replicas=1)), d, x0=dev.x0_row())
    for s in _steps(w):
        dev.grads_into(s, grads)
        grads[1:] = grads[0:1]
        many.step_sync(grads, w.lr, w.adopt_clip_value(s))
        one.step(grads[0:1].contiguous(), w.lr, w.adopt_clip_value(s))
        one.sync()
    torch.cuda.synchronize()
    for a, b in zip(many.states(), one.states()):
        assert torch.equal(a, b.expand_as(a))
    many.close()
    one.close()


@pytest.mark.parametrize("name", ["adam_n3_k4_p16m", "sgdm_n2_k16_p354m_clip"])
def test_worker_permutation_permutes_states(name):
    """Without averaging, permuting the workers' gradients permutes every
    state bit for bit (each worker's update depends on its own row and its
    own clip norm only).  No oracle is involved."""
    w = synth.small_variant(synth.WORKLOADS[name], 30_000, tail=8)
    w = w.replace(replicas=5, steps=12, period_x=0, period_u=(0,) * w.n_moments, period_v=0)
    log(f"case permutation {w.name}")
    d = torch.device("cuda:0")
    dev = DeviceInputs(w, d)
    perm = torch.tensor([3, 0, 4, 1, 2], device=d)
    grads = torch.empty((w.replicas, w.numel), dtype=torch.float32, device=d)
    a = MtdaoOptimizer(abi.config_from_workload(w), d, x0=dev.x0_row())
    b = MtdaoOptimizer(abi.config_from_workload(w), d, x0=dev.x0_row())
    for s in _steps(w):
        dev.grads_into(s, grads)
        a.step(grads, w.lr)
        b.step(grads[perm].contiguous(), w.lr)
    torch.cuda.synchronize()
    for p, q in zip(a.states(), b.states()):
        assert torch.equal(p[perm], q)
    a.close()
    b.close()


@pytest.mark.parametrize("name,steps", [("adam_n3_k4_p16m", 512), ("adopt_n2_k8_p124m_bf16", 512),
                                        ("sgdm_n2_k16_p354m_clip", 512)])
def test_long_run_within_tolerance(name, steps):
    """A long run (512 local steps with every state averaged on its period)
    against the oracle on every element: the per-step fp32 differences do
    not accumulate beyond the tolerances (the EMAs forget old errors, x
    gathers about sqrt(T) 1e-7 of its update size, bf16 flips stay rare)."""
    w = synth.small_variant(synth.WORKLOADS[name], 6_000, tail=37)
    w = w.replace(steps=steps, replicas=min(w.replicas, 6), period_x=16, period_u=(32,) * w.n_moments, period_v=64)
    log(f"case long {w.name} T={w.steps} K={w.replicas} P={w.numel}")
    g = run_gpu(w, _steps(w), fused=True)
    o = run_oracle(w, _steps(w))
    assert g.masks == o.masks
    compare(w, g.opt, o, f"long-{name}")
    free(g)


@pytest.mark.parametrize("name", ["adam_n3_k4_p16m", "adopt_n2_k8_p124m_bf16", "sgdm_n2_k16_p354m_clip"])
def test_tuned_layout_same_results(name):
    """The tuned arena layout only moves buffers: steps and averaging events
    over it give bit-identical states to the packed layout, the chosen order
    is a permutation of the [K][P] buffers, and the tuning passes left no
    trace in the states (each optimizer starts from x_0 and zero moments)."""
    w = synth.small_variant(synth.WORKLOADS[name], 40_000, tail=12)
    w = w.replace(steps=20, period_x=4, period_u=(8,) * w.n_moments, period_v=16 if w.form != "sgdm" else 0)
    log(f"case tuned-layout {w.name} K={w.replicas} P={w.numel}")
    d = torch.device("cuda:0")
    dev = DeviceInputs(w, d)
    a = MtdaoOptimizer(abi.config_from_workload(w), d, x0=dev.x0_row(), grad_buffer=True)
    b = MtdaoOptimizer(abi.config_from_workload(w), d, x0=dev.x0_row(), grad_buffer=True, layout="tuned")
    n_rows = 3 + w.n_moments - (1 if w.form == "sgdm" else 0)
    assert sorted(b.layout_order) == list(range(n_rows))
    assert b.layout_report["candidates"] == min(24, math.factorial(n_rows))
    for s in _steps(w):
        dev.grads_into(s, a.grad)
        b.grad.copy_(a.grad)
        assert a.step_sync(a.grad, w.lr, w.adopt_clip_value(s)) == b.step_sync(b.grad, w.lr, w.adopt_clip_value(s))
    torch.cuda.synchronize()
    for p, q in zip(a.states(), b.states()):
        assert torch.equal(p, q)
    a.close()
    b.close()
