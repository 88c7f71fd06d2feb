#!/usr/bin/env python3
"""Benchmark of the MT-DAO hot path on one MI355X.

One step = one pass of the whole hot path over one batch of synthetic
gradients: the per-replica clip norm (when the workload clips), the fused
local step of every replica, and the replica-mean of every state the
schedule makes due at that step -- one mtdao_step_sync call, which folds
the averaging into the step's pass on steps where states are due.  Inputs
(states and one filled gradient buffer) are resident in HBM before the timed
region.  The default run times 256 consecutive steps of the 1.31B-parameter,
K=4, Adam N=3 fp32 workload.  The window is centred on the step at which
every state is due together (s = 256 for that workload), so it holds that
averaging event at any --steps, and at 256 steps the amortised share of
every state's events (x: 4, each u^j: 2, v: 1).

Prints ONE JSON line.  Extra objects:
  step / sync       element-updates/s and GB/s of each part, % of HBM peak
                    (step: mean and median of the timed launches with nothing
                    due; sync: the standalone averaging pass per state, median
                    of 20 launches outside the timed region)
  step_sync_fused   the fused step + averaging: the window's launches with
                    due states, and 10 launches each with x due and with
                    every state due, outside the window
  achievable        plain copy / read / write kernels, and a bare stream
                    with the step's exact access mix on the same buffers
  device            the device the line was measured on
  roofline          dominant kernel (the local step): algorithmic bytes per
                    launch / mean launch time from HIP events on its stream
  cpu_baseline      the CPU oracle, unchanged, on a bounded sample of the same
                    workload: all cores of the job's share (value) and one
                    thread (single_thread)
"""

from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "param-element updates/s (x K workers) + achieved HBM GB/s % peak, step & sync"
HBM_PEAK_GBS = 8000.0
DEFAULT_WORKLOAD = "adam_n3_k4_p1311m"
KERNEL_SRCS = [os.path.join(ROOT, "paper_2510_05361_amd", "csrc", f) for f in ("kernels.hpp", "mtdao.hip")]
STREAM_LIB = os.path.join(ROOT, "paper_2510_05361_amd", "libstream_ref.so")


def step_bytes_per_element(w) -> int:
    """Algorithmic HBM bytes of one element-update of the local step: read
    and write x, u^1..u^N, v; read g (plus one more read of g for the
    clip norm)."""
    p = 2 if w.param_dtype == "bf16" else 4
    pg = 2 if w.grad_dtype == "bf16" else 4
    b = 2 * p + pg + 8 * w.n_moments + (8 if w.has_v else 0)
    return b


def norm_bytes_per_element(w) -> int:
    if w.clip_rho > 0 and w.form != "adopt":
        return 2 if w.grad_dtype == "bf16" else 4
    return 0


def kernel_hash() -> str:
    """Hash of the kernel source and its launch configuration (kernels.hpp
    and mtdao.hip with comments removed and white space collapsed, so that
    a change of wording leaves it alone and a change of code does not)."""
    import re

    h = hashlib.sha256()
    for p in KERNEL_SRCS:
        with open(p, encoding="utf-8") as f:
            text = f.read()
        text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
        text = re.sub(r"//[^\n]*", " ", text)
        h.update(" ".join(text.split()).encode())
    return h.hexdigest()[:16]


def stream_lib():
    import ctypes

    L = ctypes.CDLL(STREAM_LIB)
    for n in ("stream_ref_copy", "stream_ref_read"):
        getattr(L, n).argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p]
        getattr(L, n).restype = ctypes.c_int32
    L.stream_ref_fill.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p]
    L.stream_ref_fill.restype = ctypes.c_int32
    L.stream_ref_step_mix.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.POINTER(ctypes.c_void_p),
                                      ctypes.c_int32, ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32,
                                      ctypes.c_int64, ctypes.c_int32, ctypes.c_void_p]
    L.stream_ref_step_mix.restype = ctypes.c_int32
    return L


def same_mix(opt, grads, w, stream, reps: int = 10) -> float:
    """Seconds per launch of a bare stream with the local step's exact access
    mix (reads g, x, u^j, v; writes x, u^j, v back unchanged) on the
    optimizer's own buffers, with the step kernel's tile placement and
    windows, preceded by a plain read of g when the workload clips (the norm
    pass): the ceiling the step is measured against."""
    import ctypes

    import torch

    L = stream_lib()
    u = (ctypes.c_void_p * len(opt.u))(*[t.data_ptr() for t in opt.u])
    args = (opt.x.data_ptr(), grads.data_ptr(), u, len(opt.u), opt.v.data_ptr() if opt.v is not None else None,
            int(w.param_dtype == "bf16"), int(w.grad_dtype == "bf16"), w.numel, w.replicas, stream.cuda_stream)

    # a clipping step also reads g once more for its norm: the ceiling then
    # adds a plain read of the gradient rows
    clip = norm_bytes_per_element(w) > 0
    sink = torch.empty(4, dtype=torch.float32, device=grads.device)
    g_n4 = w.replicas * w.numel * (2 if w.grad_dtype == "bf16" else 4) // 16

    def launch():
        if clip:
            r = L.stream_ref_read(grads.data_ptr(), sink.data_ptr(), g_n4, stream.cuda_stream)
            if r != 0:
                raise RuntimeError(f"stream_ref_read: HIP error {r}")
        r = L.stream_ref_step_mix(*args)
        if r != 0:
            raise RuntimeError(f"stream_ref_step_mix: HIP error {r}")

    ms = _event_times(launch, reps, stream)
    torch.cuda.synchronize()
    return _median(ms) / 1e3


def _median(xs):
    ys = sorted(xs)
    n = len(ys)
    return ys[n // 2] if n % 2 else 0.5 * (ys[n // 2 - 1] + ys[n // 2])


def achievable(nbytes: int = 8 << 30, reps: int = 5):
    """HBM bandwidth of plain streaming kernels on this device (copy: read
    + write, read only, write only), the practical ceilings of each mix."""
    import torch

    L = stream_lib()
    n4 = nbytes // 16
    a = torch.ones(n4 * 4, dtype=torch.float32, device="cuda:0")
    b = torch.empty_like(a)
    st = torch.cuda.current_stream()
    out = {}
    for name, fn, moved in (("copy", lambda: L.stream_ref_copy(a.data_ptr(), b.data_ptr(), n4, st.cuda_stream), 2 * nbytes),
                            ("read", lambda: L.stream_ref_read(a.data_ptr(), b.data_ptr(), n4, st.cuda_stream), nbytes),
                            ("write", lambda: L.stream_ref_fill(b.data_ptr(), n4, st.cuda_stream), nbytes)):
        fn()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(st)
        for _ in range(reps):
            fn()
        e1.record(st)
        torch.cuda.synchronize()
        t = e0.elapsed_time(e1) / reps / 1e3
        out[name + "_GBps"] = moved / t / 1e9
    del a, b
    torch.cuda.empty_cache()
    return out


def load_traffic(workload: str, launch_bytes: float):
    """HBM traffic of the local-step kernel from committed rocprofv3 --pmc
    counters (FETCH_SIZE and WRITE_SIZE per dispatch, scaled by the same
    counters' reading for a plain copy of known size); None when absent or
    taken on another version of the kernel source."""
    path = os.path.join(ROOT, "profiles", f"traffic_k_local_step_{workload}.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        t = json.load(f)
    if t.get("kernel_source_sha256_16") != kernel_hash():
        return None
    return float(t["traffic_bytes_per_launch"])


def _oracle_steps(w, idx, target_s: float, ready=None):
    """Local steps of the oracle, as it is, on the elements ``idx`` of every
    replica until ~target_s of wall time: (steps, seconds, seconds of one
    replica mean of one state on the slice).  ``ready`` (if given) is called
    once the inputs are built, before the clock starts."""
    import numpy as np

    import oracle
    import synth

    cfg = oracle.OracleConfig.from_workload(w)
    st = oracle.new_state(cfg, synth.host_x0_row(w, idx), w.replicas)
    g = synth.host_grad_rows(w, 1, idx)
    scale = np.ones(w.replicas) if w.clip_rho > 0 and w.form != "adopt" else None
    if ready is not None:
        ready()
    steps, t0 = 0, time.perf_counter()
    while True:
        s = steps + 2
        if scale is not None:
            for m in range(w.replicas):
                oracle.sumsq(g[m], w.grad_dtype)
        oracle.local_step(cfg, st, g, s, w.lr, w.adopt_clip_value(s), scale)
        steps += 1
        el = time.perf_counter() - t0
        if el >= target_s or steps >= 1000:
            break
    t1 = time.perf_counter()
    oracle.replica_mean(st.u[0], "f32")
    return steps, el, time.perf_counter() - t1


def cpu_baseline(w, target_s: float = 10.0, parallel_s: float = 2.0):
    """The CPU oracle, as it is, on a sample of the same workload: a slice of
    2^20 elements per replica (every replica), timed for local steps plus
    one replica mean of one state, the sync cost amortised by the schedule.

    Two legs: one thread (~target_s), then one thread per host core of this
    job's share (up to 16), each running the unchanged oracle on its own
    disjoint 2^20-element slice for ~parallel_s (the C oracle releases the
    GIL).  ``value`` is the all-cores rate."""
    import threading

    import numpy as np

    n = min(w.numel, 1 << 20)
    syncs_per_step = (1.0 / w.period_x if w.period_x else 0.0) + sum(
        1.0 / h for h in w.period_u if h) + (1.0 / w.period_v if (w.has_v and w.period_v) else 0.0)

    def rate(steps, el, t_mean):
        return w.replicas * n / (el / steps + syncs_per_step * t_mean)

    steps1, el1, mean1 = _oracle_steps(w, np.arange(n, dtype=np.int64), target_s)
    single = rate(steps1, el1, mean1)

    threads = max(1, min(16, os.cpu_count() or 1, int(os.environ.get("OMP_NUM_THREADS", "16") or 16)))
    results = [None] * threads
    start = threading.Barrier(threads)

    def work(i):
        idx = (np.arange(n, dtype=np.int64) + i * n) % w.numel
        results[i] = _oracle_steps(w, idx, parallel_s, start.wait)

    pool = [threading.Thread(target=work, args=(i,)) for i in range(threads)]
    for t in pool:
        t.start()
    for t in pool:
        t.join()
    par = sum(rate(*r) for r in results)
    stepsp = sum(r[0] for r in results)

    cpu = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    cpu = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    eb = step_bytes_per_element(w) + norm_bytes_per_element(w)
    clip = ", clip norms included" if (w.clip_rho > 0 and w.form != "adopt") else ""
    return {
        "value": par,
        "unit": "element-updates/s",
        "cores": threads,
        "kind": "oracle",
        "GBps_algorithmic": par * eb / 1e9,
        "single_thread": {"value": single, "cores": 1, "steps": steps1, "seconds": round(el1, 2)},
        "cpu_model": cpu,
        "host_cpus": os.cpu_count(),
        "sample": (f"{n} elements x {w.replicas} replicas of {w.name} per thread ({threads} threads on "
                   f"disjoint slices, {stepsp} local steps in ~{parallel_s:.0f} s{clip}) + one replica "
                   f"mean per thread, sync amortised at {syncs_per_step:.4f} state-syncs/step; "
                   f"single-thread leg: {steps1} steps in {el1:.1f} s"),
    }


def calibrate_copy(nbytes: int, reps: int) -> None:
    """A plain device copy of known size (the stream-reference copy kernel):
    the reference reading of FETCH_SIZE / WRITE_SIZE under rocprofv3 --pmc."""
    import torch

    L = stream_lib()
    n4 = nbytes // 16
    a = torch.ones(n4 * 4, dtype=torch.float32, device="cuda:0")
    b = torch.empty_like(a)
    st = torch.cuda.current_stream()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(reps):
        L.stream_ref_copy(a.data_ptr(), b.data_ptr(), n4, st.cuda_stream)
    torch.cuda.synchronize()
    dt = (time.perf_counter() - t0) / reps
    print(json.dumps({"copy_bytes_each_way": n4 * 16, "reps": reps, "ms": dt * 1e3,
                      "GBps_read_plus_write": 2 * n4 * 16 / dt / 1e9}), flush=True)


def _event_times(fn, reps: int, stream) -> list:
    """Milliseconds of each of ``reps`` calls of fn (which enqueues on
    ``stream``), HIP events around each call; one untimed call first."""
    import torch

    fn()
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(reps)]
    for a, b in evs:
        a.record(stream)
        fn()
        b.record(stream)
    torch.cuda.synchronize()
    return [a.elapsed_time(b) for a, b in evs]


def layout_json(opt, layout):
    """Where the [K][P] buffers sit in the optimizer's allocation."""
    names = ["x"] + (["g"] if opt.grad is not None else []) + [f"u{j + 1}" for j in range(opt.N)] \
        + (["v"] if opt.has_v else [])
    out = {"mode": layout, "order": [names[i] for i in opt.layout_order] if opt.layout_order else None}
    r = opt.layout_report
    if r is not None:
        out.update({"candidates": r["candidates"], "packed_ms": r["packed_ms"], "best_ms": r["best_ms"],
                    "worst_ms": r["worst_ms"],
                    "note": "one timed pass of the local step per candidate order, over zeroed buffers"})
    return out


def device_info() -> dict:
    import torch

    p = torch.cuda.get_device_properties(0)
    return {"name": p.name, "gcnArchName": getattr(p, "gcnArchName", None),
            "compute_units": p.multi_processor_count, "memory_GB": round(p.total_memory / 1e9, 1)}


def _time_calls(fn, reps: int, stream) -> float:
    """Mean seconds per call of fn (enqueues on ``stream``), HIP events
    around each call; one untimed call first."""
    import torch

    fn()
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(reps)]
    for a, b in evs:
        a.record(stream)
        fn()
        b.record(stream)
    torch.cuda.synchronize()
    return sum(a.elapsed_time(b) for a, b in evs) / reps / 1e3


def _part(name: str, seconds: float, nbytes: float, kernel: str, copy_gbs: float) -> dict:
    gbs = nbytes / seconds / 1e9
    return {"part": name, "kernel": kernel, "mean_launch_ms": seconds * 1e3, "algorithmic_bytes": nbytes,
            "GBps": gbs, "pct_hbm_peak": 100 * gbs / HBM_PEAK_GBS, "pct_of_plain_copy": 100 * gbs / copy_gbs}


def measure_row(args) -> int:
    """Launch time and bandwidth of the kernels behind one of the paths
    beyond the plain step, at full size (one JSON line):
      outer  Nesterov OuterOpt at an x averaging event: the standalone mean
             of x with the outer step, and the fused step + x mean + outer
             step (bench workload, outer lr 0.7, momentum 0.9)
      stats  mtdao_sync_stats of every state (bench workload): the mean
             plus the averaging diagnostics, one call, host wait included
      prob   Algorithm 4's step with averaged momenta (SGDM, K = 16,
             beta = (0, 0.99), omega = (0.3, 0.7), no clip): every momentum
             due, and momenta and x due
    Each part is reported against its algorithmic bytes and next to the
    plain local step of the same buffers."""
    import torch

    import synth
    from paper_2510_05361_amd import mtdao as abi
    from paper_2510_05361_amd.optimizer import MtdaoOptimizer
    from synth.device import DeviceInputs

    d = torch.device("cuda:0")
    if args.row == "prob":
        w = synth.WORKLOADS["sgdm_n2_k16_p354m_clip"].replace(beta1=(0.0, 0.99), omega=(0.3, 0.7), clip_rho=0.0,
                                                              period_x=0, period_u=(0, 0))
        cfg = abi.config_from_workload(w, sync_order=abi.MTDAO_SYNC_MOMENTA_IN_STEP)
    elif args.row == "outer":
        w = synth.WORKLOADS[args.workload]
        cfg = abi.config_from_workload(w, outer_opt=abi.MTDAO_OUTER_NESTEROV, outer_lr=0.7, outer_momentum=0.9)
    else:
        w = synth.WORKLOADS[args.workload]
        cfg = abi.config_from_workload(w)
    K, P = w.replicas, w.numel
    print(f"bench --row {args.row}: {w.name} K={K} P={P}", file=sys.stderr, flush=True)
    dev = DeviceInputs(w, d)
    opt = MtdaoOptimizer(cfg, d, x0=dev.x0_row())
    gdt = torch.bfloat16 if w.grad_dtype == "bf16" else torch.float32
    grads = torch.empty((K, P), dtype=gdt, device=d)
    dev.grads_into(1, grads)
    del dev
    torch.cuda.synchronize()
    st = torch.cuda.current_stream()
    reps = max(1, args.steps)
    xs = 2 if w.param_dtype == "bf16" else 4
    eb = step_bytes_per_element(w)
    step_bytes = K * P * eb
    # the plain call also runs the clip-norm pass when the workload clips
    plain_bytes = K * P * (eb + norm_bytes_per_element(w))
    mean_bytes = [2 * K * xs * P] + [2 * K * 4 * P] * (w.n_moments + (1 if w.has_v else 0))
    for _ in range(args.warmup):
        opt.step_sync(grads, w.lr, w.adopt_clip_value(2), 0)
    plain_s = _time_calls(lambda: opt.step_sync(grads, w.lr, w.adopt_clip_value(2), 0), reps, st)
    parts = []
    if args.row == "outer":
        # the outer step runs once per step s: every timed averaging of x
        # follows an untimed local step
        ms = []
        for _ in range(reps + 1):
            opt.step_sync(grads, w.lr, w.adopt_clip_value(2), 0)
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(st)
            opt.sync(1)
            e1.record(st)
            torch.cuda.synchronize()
            ms.append(e0.elapsed_time(e1))
        mean_s = sum(ms[1:]) / reps / 1e3
        fused_s = _time_calls(lambda: opt.step_sync(grads, w.lr, w.adopt_clip_value(2), 1), reps, st)
        ceil = achievable()
        parts.append(_part("mean of x + outer step", mean_s, mean_bytes[0] + 16 * P,
                           "k_replica_mean_waves (outer epilogue)", ceil["copy_GBps"]))
        parts.append(_part("fused step + mean of x + outer step", fused_s, step_bytes + 16 * P,
                           "k_local_step_sync_waves (outer epilogue)", ceil["copy_GBps"]))
    elif args.row == "stats":
        nst = len(mean_bytes)
        per_state = [_time_calls(lambda sid=sid: opt.sync_stats(1 << sid), reps, st) for sid in range(nst)]
        all_s = _time_calls(lambda: opt.sync_stats((1 << nst) - 1), reps, st)
        plain_mean = [_time_calls(lambda sid=sid: opt.sync(1 << sid), reps, st) for sid in range(nst)]
        ceil = achievable()
        for sid in range(nst):
            parts.append(_part(f"sync_stats state {sid}", per_state[sid], mean_bytes[sid],
                               "k_replica_mean_stats + k_stats_finalize + copy to host", ceil["copy_GBps"]))
            parts.append(_part(f"plain mean state {sid}", plain_mean[sid], mean_bytes[sid],
                               "k_replica_mean_waves", ceil["copy_GBps"]))
        parts.append(_part("sync_stats all states, one call", all_s, sum(mean_bytes),
                           "k_replica_mean_stats (fp32 states) + k_stats_finalize + copy to host", ceil["copy_GBps"]))
    else:
        mom = ((1 << w.n_moments) - 1) << 1
        prob_u_s = _time_calls(lambda: opt.step_sync(grads, w.lr, 0.0, mom), reps, st)
        prob_all_s = _time_calls(lambda: opt.step_sync(grads, w.lr, 0.0, mom | 1), reps, st)
        ceil = achievable()
        parts.append(_part("step with every momentum averaged in the step", prob_u_s, step_bytes,
                           "k_sgdm_averaged_momenta_waves (K <= 16)", ceil["copy_GBps"]))
        parts.append(_part("step with momenta and x averaged", prob_all_s, step_bytes,
                           "k_sgdm_averaged_momenta_waves (K <= 16)", ceil["copy_GBps"]))
    opt.close()
    out = {"row": args.row, "workload": w.name, "replicas": K, "params_per_replica": P, "form": w.form,
           "reps": reps, "plain_step": _part("plain local step, same buffers", plain_s, plain_bytes,
                                             "k_local_step" + (" + clip-norm pass" if plain_bytes > step_bytes else ""),
                                             ceil["copy_GBps"]),
           "device": device_info(),
           "parts": parts, "achievable": ceil, "peak_GBps": HBM_PEAK_GBS}
    print(json.dumps(out), flush=True)
    return 0


def window_start(w, steps: int, warmup: int) -> int:
    """Updates applied before the warm-up, so that the timed window of
    ``steps`` steps is centred on the first step at which every state is
    due together (the least common multiple of the periods): whatever
    --steps is, the window holds that all-states averaging event, and for
    a window of one such period the amortised share of every state's
    events.  Kept at >= 0; the updates themselves are not run."""
    periods = [h for h in (w.period_x, *w.period_u, w.period_v if w.has_v else 0) if h > 0]
    if not periods:
        return 0
    lcm = 1
    for h in periods:
        lcm = lcm * h // math.gcd(lcm, h)
    return max(0, lcm - (steps + 1) // 2 - warmup)


def measure_graph(args) -> int:
    """Per-step time of the 1M-parameter K=2 workload (launch-bound: its
    75 MB sit in the MALL) three ways, one JSON line: eager mtdao_step_sync
    calls, eager mtdao_step_sync_device calls, and replays of a HIP graph of
    one schedule period (16 steps) of mtdao_step_sync_device, whose eta_t
    and bias corrections are formed on the device at every replay."""
    import numpy as np
    import torch

    import synth
    from paper_2510_05361_amd import mtdao as abi
    from paper_2510_05361_amd.optimizer import MtdaoOptimizer
    from synth.device import DeviceInputs

    w = synth.WORKLOADS[args.workload if args.workload != DEFAULT_WORKLOAD else "adam_n2_k2_p1m"]
    d = torch.device("cuda:0")
    K, P = w.replicas, w.numel
    periods = [h for h in (w.period_x, *w.period_u, w.period_v if w.has_v else 0) if h > 0]
    window = 1
    for h in periods:
        window = window * h // math.gcd(window, h)
    reps = max(2, args.steps // window)
    print(f"bench --row graph: {w.name} K={K} P={P} window={window} reps={reps}", file=sys.stderr, flush=True)
    dev = DeviceInputs(w, d)
    n_total = 2 + window * (reps + args.warmup + 2)
    lr = torch.from_numpy(np.full(n_total, w.lr, dtype=np.float32)).to(d)
    clip = torch.from_numpy(np.array([w.adopt_clip_value(k + 1) for k in range(n_total)], dtype=np.float32)).to(d)
    opt = MtdaoOptimizer(abi.config_from_workload(w), d, x0=dev.x0_row(), grad_buffer=True)
    dev.grads_into(1, opt.grad)
    st = torch.cuda.current_stream()
    opt.step_sync(opt.grad, w.lr, w.adopt_clip_value(1))  # update 1 (ADOPT: v only) on the host path

    def eager():
        for _ in range(window):
            s = opt.step_count + 1
            opt.step_sync(opt.grad, w.lr, w.adopt_clip_value(s))

    opt.device_step(lr, clip if w.form == "adopt" else None)

    def eager_device():
        for _ in range(window):
            opt.step_sync_device(opt.grad)
        opt.device_step_advance()

    for _ in range(args.warmup):
        eager()
        eager_device()
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        eager_device()
    torch.cuda.synchronize()
    res = {}
    for name, fn in (("eager_step_sync", eager), ("eager_step_sync_device", eager_device), ("graph_replay", graph.replay)):
        if name != "eager_step_sync":
            opt.device_step(lr, clip if w.form == "adopt" else None)
        ms = _event_times(fn, reps, st)
        res[name] = {"us_per_step": 1e3 * sum(ms) / len(ms) / window, "windows": reps}
    eb = step_bytes_per_element(w) + norm_bytes_per_element(w)
    for v in res.values():
        v["GBps"] = K * P * eb / (v["us_per_step"] * 1e-6) / 1e9
    del graph
    opt.close()
    print(json.dumps({"row": "graph", "workload": w.name, "replicas": K, "params_per_replica": P, "window_steps": window,
                      "bytes_per_step": K * P * eb, "parts": res, "device": device_info(),
                      "note": "per-step time includes the window's averaging events; the working set is MALL-resident, "
                              "so this is a launch-overhead figure, not an HBM one"}), flush=True)
    return 0


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=256)
    ap.add_argument("--warmup", type=int, default=8)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--grad-in-arena", type=int, choices=[0, 1], default=1,
                    help="1: the gradient rows are carved from the optimizer's own allocation (default); "
                         "0: a separate torch allocation")
    ap.add_argument("--layout", choices=["tuned", "packed"], default="tuned",
                    help="order of x, the gradient rows, u^j and v in the optimizer's allocation: the "
                         "fastest of a set of candidates timed at start-up (default), or the fixed order "
                         "(--grad-in-arena 0 implies packed)")
    ap.add_argument("--row", choices=["step", "outer", "stats", "prob", "graph"], default="step",
                    help="step: the hot path (the default line); outer / stats / prob: the kernels of the "
                         "Nesterov OuterOpt, the averaging diagnostics, Algorithm 4's step (--steps = reps); "
                         "graph: eager and graph-replayed steps of the 1M-parameter workload")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="BYTES",
                    help="only run a plain copy of BYTES each way (counter calibration)")
    args = ap.parse_args()

    if args.gpus != 1:
        print(f"bench.py measures one GPU; --gpus {args.gpus} is not supported (the path is built "
              "and measured on a single MI355X; see the sharding notes of the design)", file=sys.stderr)
        return 2

    if args.calibrate_copy:
        calibrate_copy(args.calibrate_copy, max(1, args.steps))
        return 0
    if args.row == "graph":
        return measure_graph(args)
    if args.row != "step":
        return measure_row(args)

    import torch

    import synth
    from paper_2510_05361_amd import mtdao as abi
    from paper_2510_05361_amd.optimizer import MtdaoOptimizer
    from synth.device import DeviceInputs

    w = synth.WORKLOADS[args.workload]
    d = torch.device("cuda:0")
    K, P = w.replicas, w.numel
    start = window_start(w, args.steps, args.warmup)
    print(f"bench: {w.name} K={K} P={P} warmup={args.warmup} steps={args.steps} "
          f"window s={start + args.warmup + 1}..{start + args.warmup + args.steps}", file=sys.stderr, flush=True)
    dev = DeviceInputs(w, d)
    cfg = abi.config_from_workload(w, start_step=start)
    layout = args.layout if args.grad_in_arena else "packed"
    opt = MtdaoOptimizer(cfg, d, x0=dev.x0_row(), grad_buffer=bool(args.grad_in_arena), layout=layout)
    if opt.layout_report is not None:
        r = opt.layout_report
        print(f"bench: layout tuned over {r['candidates']} orders: packed {r['packed_ms']:.4f} ms, "
              f"best {r['best_ms']:.4f} ms, worst {r['worst_ms']:.4f} ms", file=sys.stderr, flush=True)
    if args.grad_in_arena:
        grads = opt.grad
    else:
        gdt = torch.bfloat16 if w.grad_dtype == "bf16" else torch.float32
        grads = torch.empty((K, P), dtype=gdt, device=d)
    dev.grads_into(1, grads)
    del dev
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()

    def one_step(s, ev=None, mask=abi.MTDAO_SYNC_AUTO):
        # local step of every replica + averaging of the states due at s, one call
        if ev is not None:
            ev[0].record(stream)
        applied = opt.step_sync(grads, w.lr, w.adopt_clip_value(s), mask)
        if ev is not None:
            ev[1].record(stream)
        return applied

    s = start
    for _ in range(args.warmup):
        s += 1
        one_step(s)
    torch.cuda.synchronize()

    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(args.steps)]
    syncs = {}
    masks = []
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(args.steps):
        s += 1
        applied = one_step(s, evs[k])
        masks.append(applied)
        if applied:
            syncs[s] = applied
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    call_ms = [a.elapsed_time(b) for a, b in evs]
    plain = [t for t, m in zip(call_ms, masks) if m == 0]
    fused = [t for t, m in zip(call_ms, masks) if m != 0]
    # the dominant kernel: the local step on steps with nothing due
    step_launch_s = (sum(plain) / len(plain) if plain else sum(call_ms) / len(call_ms)) / 1e3

    # outside the timed window: the fused step + averaging with x due, and
    # with every state due (10 launches each), then the same-mix bare stream
    nstates = 1 + w.n_moments + (1 if w.has_v else 0)
    fused_masks = {"x": 1, "all_states": (1 << nstates) - 1}
    fused_extra = {}
    for label, fm in fused_masks.items():
        def call(fm=fm):
            nonlocal s
            s += 1
            one_step(s, mask=fm)
        ms = _event_times(call, 10, stream)
        fused_extra[label] = ms
    mix_s = same_mix(opt, grads, w, stream)

    # per-state sync time (replica mean of one state), untimed region: the
    # median of 20 launches, each bracketed by its own events
    sync_s = []
    for sid in range(nstates):
        sync_s.append(_median(_event_times(lambda sid=sid: opt.sync(1 << sid), 20, stream)) / 1e3)
    layout_info = layout_json(opt, layout)
    opt.close()
    del opt, grads
    torch.cuda.empty_cache()
    ceil = achievable()

    eb_step = step_bytes_per_element(w)
    eb = eb_step + norm_bytes_per_element(w)
    # the timed call: the local step, preceded by the clip-norm pass when
    # clipping is on (its bytes are then part of the call's algorithmic bytes)
    launch_bytes = K * P * eb
    roof_kernel = "k_local_step" if norm_bytes_per_element(w) == 0 else \
        "k_sumsq_partial + k_clip_finalize + k_local_step"
    step_gbs = K * P * eb / step_launch_s / 1e9
    ceil["same_mix_GBps"] = K * P * eb / mix_s / 1e9
    ceil["same_mix_note"] = ("bare stream with the step's reads and writes (no arithmetic) on the same buffers, "
                             "same tile placement and windows" + (", after a plain read of g (the norm pass)"
                                                                   if norm_bytes_per_element(w) else "")
                             + "; median of 10 launches")
    sync_report = []
    names = ["x"] + [f"u{j + 1}" for j in range(w.n_moments)] + (["v"] if w.has_v else [])
    for sid, t in enumerate(sync_s):
        es = 2 if (sid == 0 and w.param_dtype == "bf16") else 4
        gbs = 2 * K * es * P / t / 1e9
        sync_report.append({"state": names[sid], "ms": t * 1e3, "GBps": gbs, "pct_hbm_peak": 100 * gbs / HBM_PEAK_GBS,
                            "pct_of_plain_copy": 100 * gbs / ceil["copy_GBps"]})

    def fused_entry(ms_list, what):
        mean = sum(ms_list) / len(ms_list)
        gbs = launch_bytes / (mean / 1e3) / 1e9
        return {"launches": len(ms_list), "mean_ms": mean, "median_ms": _median(ms_list), "GBps": gbs,
                "pct_hbm_peak": 100 * gbs / HBM_PEAK_GBS,
                "over_plain_step_pct": 100 * (mean / 1e3 / step_launch_s - 1), "note": what}

    step_sync_fused = {
        "in_window": fused_entry(fused, "the window's steps with due states") if fused else {"launches": 0},
        "x_due": fused_entry(fused_extra["x"], "outside the window: mtdao_step_sync with x due"),
        "all_states_due": fused_entry(fused_extra["all_states"],
                                      "outside the window: mtdao_step_sync with every state due"),
    }
    value = K * P * args.steps / wall
    traffic = load_traffic(w.name, launch_bytes)
    out = {
        "metric": METRIC,
        "value": value,
        "unit": "element-updates/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": wall / args.steps * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32" if w.param_dtype == "f32" else "bf16 params, f32 moments",
        "data": "synthetic (seeded gradients and parameters shaped like the paper's GPT tensor lists)",
        "config": {"workload": w.name, "replicas": K, "params_per_replica": P, "form": w.form,
                   "n_moments": w.n_moments, "param_dtype": w.param_dtype, "grad_dtype": w.grad_dtype,
                   "periods": {"x": w.period_x, "u": list(w.period_u), "v": w.period_v},
                   "window_steps": [start + args.warmup + 1, start + args.warmup + args.steps],
                   "syncs_in_window": {str(k): v for k, v in sorted(syncs.items())},
                   "grad_in_arena": bool(args.grad_in_arena),
                   "layout": layout_info},
        "device": device_info(),
        "step": {"mean_launch_ms": step_launch_s * 1e3,
                 "median_launch_ms": _median(plain if plain else call_ms),
                 "launches": len(plain),
                 "element_updates_per_s": K * P / step_launch_s,
                 "bytes_per_element_update": eb, "GBps": step_gbs,
                 "pct_hbm_peak": 100 * step_gbs / HBM_PEAK_GBS,
                 "pct_of_plain_copy": 100 * step_gbs / ceil["copy_GBps"],
                 "pct_of_same_mix": 100 * mix_s / step_launch_s},
        "achievable": ceil,
        "sync": sync_report,
        "step_sync_fused": step_sync_fused,
        "roofline": {"bound": "hbm", "achieved": launch_bytes / step_launch_s / 1e9, "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": launch_bytes / step_launch_s / 1e9 / HBM_PEAK_GBS,
                     "traffic": traffic, "kernel": roof_kernel,
                     "algorithmic_bytes_per_launch": launch_bytes},
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(w)
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
