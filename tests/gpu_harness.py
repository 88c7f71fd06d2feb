"""Shared pieces of the GPU parity tests: run a workload through the C ABI on
the GPU, run the CPU oracle on the same seeded inputs (all elements or a
deterministic sample), and compare.

Inputs for both sides come from ``synth``; no oracle input or expected
value is ever taken from the GPU path.
"""

from __future__ import annotations

import math
import os
import sys
import time
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass
from typing import Callable, Dict, List, Optional, Sequence, Tuple, Union

import numpy as np
import torch

import oracle
import synth
from paper_2510_05361_amd import mtdao as abi
from paper_2510_05361_amd.optimizer import MtdaoOptimizer
from synth.device import DeviceInputs

# Tolerances (derivations in the design notes):
#  fp32 states: max_i |a_i - b_i| / max(|b_i|, rms(b)) <= 1e-5, rms over an
#  unbiased subset of the row.
#  bf16 params: |a - b| in bf16 ulps at max(largest |x| of the element's
#  trajectory, rms(b)) times BF16_HEADROOM (XAbsMax).  The kernel rounds its
#  fp32 value and the oracle its fp64 value to bf16; when the exact value
#  lies within the fp32 error of a rounding boundary the two pick neighbours
#  one ulp apart (a flip), and that offset persists (x feeds every later
#  update).  An averaging of x carries a flip of one worker into the mean,
#  shifted by ulp/K, so it can move the rounded mean, and with it all K
#  workers, by one ulp.  Each such event adds at most one unit; three in
#  the same direction on one element are the most the 124M x 8 workload
#  shows over 128 steps (2.3e-4 of the elements >= 1 unit, 7.8e-6 > 1).
#  Bounds: at most BF16_MAX_ULPS units anywhere; at most
#  2 BF16_FLIP_RATE T n + BF16_SLACK elements (n compared, T steps; the 2
#  for the flips the averaging carries to other workers) one unit or more
#  apart, and at most a tenth of that (plus the slack) more than one unit.
REL_TOL = 1e-5
BF16_MAX_ULPS = 3
BF16_HEADROOM = 1.0 + 2.0 ** -5  # 4 ulps: how far the two trajectories may be apart
BF16_FLIP_RATE = 1e-5   # per element and step, against 2e-6 measured on 124M x 8 over 128 steps
BF16_SLACK = 32         # elements, for small comparisons
BF16_OUTER_MAX_ULPS = 16  # >= lr (1 + mu) / (1 - mu) = 13.3 for the tested (0.7, 0.9)
BF16_OUTER_FRAC = 1e-2  # 3.4e-3 measured over 96 steps


def bf16_bounds(n: float, steps: int):
    """(most elements >= 1 unit apart, most elements > 1 unit apart) for n
    compared bf16 values after ``steps`` steps."""
    r = 2 * BF16_FLIP_RATE * max(1, steps)
    return r * n + BF16_SLACK, 0.1 * r * n + BF16_SLACK


def log(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


def device() -> torch.device:
    return torch.device("cuda:0")


# ------------------------------------------------------------------ oracle


def oracle_cfg(w: synth.Workload, outer=None) -> oracle.OracleConfig:
    if outer is None:
        return oracle.OracleConfig.from_workload(w)
    return oracle.OracleConfig.from_workload(w, outer="nesterov", outer_lr=outer[0], outer_momentum=outer[1])


_SUMSQ_CACHE: Dict[tuple, float] = {}


def oracle_clip_scales(w: synth.Workload, s: int) -> Optional[np.ndarray]:
    """Per-worker clip factors from the oracle over the FULL gradient of
    step s.  Large rows use their periodic structure: a row is the scaled
    pool rotated by the worker's offset and repeated, so its sum of squares
    is q * sumsq(whole scaled pool) + sumsq(first r rotated values)."""
    if not w.clip_rho > 0 or w.form == "adopt":
        return None
    P = w.numel
    if P <= 1 << 22:
        return oracle.clip_scales(oracle_cfg(w), synth.host_grad_rows(w, s))
    sig = w.tensor_sigmas()
    assert np.all(sig == sig[0]) and w.grad_dtype == "f32"
    scaled = (sig[0] * synth.grad_pool(w)).astype(np.float32)
    key = (w.grad_dist, w.seed_g, float(sig[0]))
    if key not in _SUMSQ_CACHE:
        _SUMSQ_CACHE[key] = oracle.sumsq(scaled)
    q, r = divmod(P, synth.POOL_SIZE)
    out = np.empty(w.replicas)
    for m in range(w.replicas):
        off = synth.grad_offset(w.seed_g, m, s)
        head = scaled[off:off + r]
        tail = scaled[:max(0, r - head.size)]
        total = q * _SUMSQ_CACHE[key] + oracle.sumsq(head) + oracle.sumsq(tail)
        out[m] = oracle.clip_scale(math.sqrt(total), w.clip_rho)
    return out


Cols = Union[None, slice, np.ndarray]


class XAbsMax:
    """The largest |x| every element of every worker reached over the
    oracle's trajectory, from the initial state on (bf16 parameters only;
    None otherwise).  A bf16 rounding decision that the kernel (fp32) and
    the oracle (fp64) take differently puts the two x one bf16 ulp apart at
    the magnitude x had then, and that absolute offset persists, so the
    comparison counts in ulps at this magnitude."""

    def __init__(self, st: oracle.OracleState):
        self.a: Optional[np.ndarray] = None
        self.update(st)

    def update(self, st: oracle.OracleState) -> None:
        if st.x.dtype != np.uint16:
            return
        v = np.abs(synth.bf16_bits_to_f32(st.x))
        if self.a is None:
            self.a = v
        else:
            np.maximum(self.a, v, out=self.a)


@dataclass
class OracleResult:
    """Oracle states of the compared columns.  ``state`` holds columns
    ``idx`` (all when None); a parallel run keeps one state per disjoint
    column part in ``parts`` instead.  ``rms_cols`` marks which of the
    compared columns are an unbiased subset of the row (the evenly strided
    ones of a sample); the rms floor of the error metric is taken over
    them, None = over all compared columns.  ``x_absmax`` (one array per
    part) holds XAbsMax of bf16 parameters."""

    state: Optional[oracle.OracleState]
    masks: List[int]
    idx: Optional[np.ndarray]
    parts: Optional[List[Tuple[Cols, oracle.OracleState]]] = None
    rms_cols: Optional[np.ndarray] = None
    x_absmax: Optional[List[Optional[np.ndarray]]] = None
    steps: Optional[int] = None  # steps run, when ``masks`` does not list them

    def column_parts(self) -> List[Tuple[Cols, oracle.OracleState]]:
        return self.parts if self.parts is not None else [(self.idx, self.state)]


def run_oracle(w: synth.Workload, steps: Sequence[int], idx: Optional[np.ndarray] = None,
               init: Optional[oracle.OracleState] = None, outer=None) -> OracleResult:
    """Oracle over elements ``idx`` (all if None) for global steps ``steps``.
    Each element's trajectory depends only on its own inputs and, through
    the clip, on the per-worker norms, which are taken over full rows.
    ``outer`` = (outer_lr, outer_momentum) selects the Nesterov OuterOpt."""
    cfg = oracle_cfg(w, outer)
    if init is None:
        st = oracle.new_state(cfg, synth.host_x0_row(w, idx), w.replicas)
    else:
        st = init
    track = XAbsMax(st)
    masks = []
    for s in steps:
        masks += oracle.run(cfg, st, lambda s_: synth.host_grad_rows(w, s_, idx), [s], lambda s_: w.lr,
                            w.adopt_clip_value, scales=lambda s_, g: oracle_clip_scales(w, s_))
        track.update(st)
    return OracleResult(st, masks, idx, x_absmax=[track.a])


def oracle_threads() -> int:
    """Host threads for the oracle: the job's CPU share (at most 16)."""
    env = os.environ.get("OMP_NUM_THREADS", "")
    n = int(env) if env.isdigit() and int(env) > 0 else 16
    return max(1, min(16, n, os.cpu_count() or 1))


def run_oracle_parallel(w: synth.Workload, steps: Sequence[int], idx: Optional[np.ndarray] = None,
                        outer=None, init: Optional[Callable[[Cols], oracle.OracleState]] = None,
                        rms_cols: Optional[np.ndarray] = None, threads: Optional[int] = None) -> OracleResult:
    """The oracle, unchanged, over disjoint column parts on host threads:
    every element of the row (idx None: contiguous ranges, gradients built
    with synth.host_grad_range) or the columns idx.  An element's
    trajectory depends only on its own inputs and on the per-worker clip
    factors, which are computed over full rows before the parts start (the
    C oracle releases the GIL).  ``init(cols)`` supplies resumed states."""
    cfg = oracle_cfg(w, outer)
    steps = list(steps)
    n_threads = threads or oracle_threads()
    scales: Dict[int, Optional[np.ndarray]] = {}
    if w.clip_rho > 0 and w.form != "adopt":
        with ThreadPoolExecutor(n_threads) as ex:
            for s, sc in zip(steps, ex.map(lambda s_: oracle_clip_scales(w, s_), steps)):
                scales[s] = sc
    if idx is None:
        P = w.numel
        bounds = np.linspace(0, P, n_threads + 1).astype(np.int64)
        cols: List[Cols] = [slice(int(a), int(b)) for a, b in zip(bounds[:-1], bounds[1:]) if b > a]
    else:
        cols = [c for c in np.array_split(idx, n_threads) if c.size]
    t0 = time.perf_counter()

    def one(k: int):
        c = cols[k]
        if isinstance(c, slice):
            lo, hi = c.start, c.stop
            grads = lambda s: synth.host_grad_range(w, s, lo, hi)  # noqa: E731
            x0 = synth.host_x0_row(w, np.arange(lo, hi, dtype=np.int64))
        else:
            grads = lambda s: synth.host_grad_rows(w, s, c)  # noqa: E731
            x0 = synth.host_x0_row(w, c)
        st = init(c) if init is not None else oracle.new_state(cfg, x0, w.replicas)
        track = XAbsMax(st)
        masks = []
        for i, s in enumerate(steps):
            masks += oracle.run(cfg, st, grads, [s], lambda s_: w.lr, w.adopt_clip_value,
                                scales=lambda s_, g: scales.get(s_))
            track.update(st)
            if k == 0 and (i + 1) % max(1, len(steps) // 4) == 0:
                log(f"  oracle part 0/{len(cols)}: step {i + 1}/{len(steps)} ({time.perf_counter() - t0:.0f} s)")
        return c, st, masks, track.a

    synth.grad_pool(w), synth.x_pool(w)  # draw the pools once, before the threads
    with ThreadPoolExecutor(n_threads) as ex:
        done = list(ex.map(one, range(len(cols))))
    masks = done[0][2]
    assert all(d[2] == masks for d in done)
    log(f"  oracle: {len(cols)} parts, {sum(_ncols(c, w.numel) for c in cols)} columns x {w.replicas} workers x "
        f"{len(steps)} steps in {time.perf_counter() - t0:.1f} s on {n_threads} threads")
    return OracleResult(None, masks, idx, parts=[(c, st) for c, st, _, _ in done], rms_cols=rms_cols,
                        x_absmax=[a for _, _, _, a in done])


def _ncols(c: Cols, P: int) -> int:
    if c is None:
        return P
    if isinstance(c, slice):
        return c.stop - c.start
    return int(c.size)


# ------------------------------------------------------------------ GPU


@dataclass
class GpuResult:
    opt: MtdaoOptimizer
    masks: List[int]


def gpu_config(w: synth.Workload, start_step: int = 0, outer=None) -> abi.MtdaoConfig:
    if outer is None:
        return abi.config_from_workload(w, start_step=start_step)
    return abi.config_from_workload(w, start_step=start_step, outer_opt=abi.MTDAO_OUTER_NESTEROV,
                                    outer_lr=outer[0], outer_momentum=outer[1])


def run_gpu(w: synth.Workload, steps: Sequence[int], start_step: int = 0, dev: Optional[DeviceInputs] = None,
            opt: Optional[MtdaoOptimizer] = None, grads: Optional[torch.Tensor] = None, outer=None,
            fused: bool = False) -> GpuResult:
    """Run global steps ``steps`` through the C ABI: mtdao_local_step +
    mtdao_sync (schedule), or mtdao_step_sync when ``fused``."""
    d = device()
    dev = dev or DeviceInputs(w, d)
    if opt is None:
        opt = MtdaoOptimizer(gpu_config(w, start_step, outer), d, x0=dev.x0_row())
    gdt = torch.bfloat16 if w.grad_dtype == "bf16" else torch.float32
    if grads is None:
        grads = torch.empty((w.replicas, w.numel), dtype=gdt, device=d)
    masks = []
    for s in steps:
        dev.grads_into(s, grads)
        if fused:
            masks.append(opt.step_sync(grads, w.lr, w.adopt_clip_value(s)))
        else:
            opt.step(grads, w.lr, w.adopt_clip_value(s))
            masks.append(opt.sync())
    torch.cuda.synchronize()
    return GpuResult(opt, masks)


def gather_state(t: torch.Tensor, idx: Cols) -> np.ndarray:
    """Host copy of a [K][P] device state (all columns, a column range or
    the columns idx); bf16 states come back as uint16 bit patterns."""
    if isinstance(idx, slice):
        t = t[:, idx]
    elif idx is not None:
        t = t[:, torch.from_numpy(idx).to(t.device)]
    if t.dtype == torch.bfloat16:
        return t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
    return t.contiguous().cpu().numpy()


# ------------------------------------------------------------------ compare


def rel_err(a: np.ndarray, b: np.ndarray, rms: Optional[float] = None) -> float:
    """max_i |a_i - b_i| / max(|b_i|, rms), rms = rms(b) unless given."""
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    if rms is None:
        rms = math.sqrt(float(np.mean(b * b))) if b.size else 0.0
    den = np.maximum(np.abs(b), rms)
    err = np.abs(a - b)
    if not np.all(np.isfinite(a)):
        return float("inf")
    with np.errstate(invalid="ignore", divide="ignore"):
        r = np.where(den > 0, err / np.where(den > 0, den, 1.0), err)
    return float(r.max()) if r.size else 0.0


def ulp_unit(scale: np.ndarray) -> np.ndarray:
    """One bf16 ulp at each |scale| (8 significant bits)."""
    scale = np.where(scale > 0, scale, 2.0 ** -126)
    return np.exp2(np.floor(np.log2(scale)) - 7)


def bf16_floored_ulps(a_bits: np.ndarray, b_bits: np.ndarray, rms: Optional[float] = None) -> np.ndarray:
    """|a - b| in units of one bf16 ulp at max(|b_i|, rms), rms = rms(b)
    unless given."""
    a = synth.bf16_bits_to_f32(a_bits).astype(np.float64)
    b = synth.bf16_bits_to_f32(b_bits).astype(np.float64)
    if rms is None:
        rms = math.sqrt(float(np.mean(b * b))) if b.size else 0.0
    return np.abs(a - b) / ulp_unit(np.maximum(np.abs(b), rms))


def _as_f64(a: np.ndarray, bf16: bool) -> np.ndarray:
    return (synth.bf16_bits_to_f32(a) if bf16 else a).astype(np.float64)


# Findings of every compare() in this process, for the session summary.
REPORT: List[Tuple[str, Dict[str, float]]] = []

_CHUNK = 1 << 23  # columns x rows per metric chunk


def _metrics(kind: str, a: np.ndarray, b: np.ndarray, rms: float, ref: Optional[np.ndarray], ref_rms: float,
             bf16: bool) -> Dict[str, float]:
    """Partial metrics of one chunk (merged with _merge).  ``ref``: the
    outer parameters (kind "outer") or the trajectory's largest |x| (kind
    "bf16")."""
    af, bf = _as_f64(a, bf16), _as_f64(b, bf16)
    d = np.abs(af - bf)
    out = {"n": float(d.size), "finite": float(np.all(np.isfinite(af))),
           "max_abs_diff": float(d.max(initial=0.0)), "max_abs_want": float(np.abs(bf).max(initial=0.0))}
    if kind == "f32":
        out["rel_err"] = float((d / np.maximum(np.maximum(np.abs(bf), rms), 1e-300)).max(initial=0.0))
        nz = bf != 0
        out["rel_err_unfloored"] = float((d[nz] / np.abs(bf[nz])).max(initial=0.0))
    elif kind == "bf16":
        # the kernel's trajectory stays within a few ulps of the oracle's, so
        # it may cross into the next binade where the oracle's largest
        # magnitude lies just below one: units at BF16_HEADROOM times it
        scale = np.maximum(np.maximum(np.abs(bf), ref.astype(np.float64)), rms) * BF16_HEADROOM
        ul = d / ulp_unit(scale)
        out.update(max_ulps=float(ul.max(initial=0.0)), n_ge1=float((ul >= 1).sum()), n_gt1=float((ul > 1).sum()),
                   rel_err=float((d / np.maximum(np.maximum(np.abs(bf), rms), 1e-300)).max(initial=0.0)))
    else:  # measured at the scale of the outer parameters (ref)
        den = np.maximum(np.abs(ref.astype(np.float64)), ref_rms)
        out["err_of_x_outer"] = float((d / np.maximum(den, 1e-300)).max(initial=0.0))
        out["n_off"] = float((d > REL_TOL * den).sum())
        out["max_ulps_of_x"] = float((d / ulp_unit(den)).max(initial=0.0))
    return out


def _merge(ms: List[Dict[str, float]]) -> Dict[str, float]:
    out: Dict[str, float] = {}
    for m in ms:
        for k, v in m.items():
            if k in ("n", "n_ge1", "n_gt1", "n_off"):
                out[k] = out.get(k, 0.0) + v
            elif k == "finite":
                out[k] = min(out.get(k, 1.0), v)
            else:
                out[k] = max(out.get(k, 0.0), v)
    return out


def _rms(parts: List[Tuple[np.ndarray, Optional[np.ndarray]]], bf16: bool) -> float:
    """rms over the given (values, mask) parts; mask selects the unbiased
    columns of a sample (None: all)."""
    ss, n = 0.0, 0
    for vals, mask in parts:
        v = vals if mask is None else vals[..., mask]
        for lo in range(0, v.shape[-1], max(1, _CHUNK // max(1, v.shape[0]))):
            c = _as_f64(v[..., lo:lo + max(1, _CHUNK // max(1, v.shape[0]))], bf16)
            ss += float(np.sum(c * c))
            n += c.size
    return math.sqrt(ss / n) if n else 0.0


def compare(w: synth.Workload, gpu: MtdaoOptimizer, orc: OracleResult, label: str) -> Dict[str, Dict[str, float]]:
    """Every state of every replica against the oracle on the compared
    columns; raises on failure.  Per state (R19): max_i |a_i - b_i| /
    max(|b_i|, rms(b)) with rms over an unbiased subset of the row; bf16 x
    in bf16 ulps of the same floor; the Nesterov outer momentum at the
    scale of the outer parameters."""
    parts = orc.column_parts()
    names = ["x"] + [f"u{j + 1}" for j in range(w.n_moments)] + (["v"] if w.has_v else [])
    gs = gpu.states()
    nest = gpu.x_outer is not None
    if nest:
        names += ["x_outer", "outer_mom"]
        gs = gs + [gpu.x_outer.view(1, -1), gpu.x_outer_mom.view(1, -1)]
    masks: List[Optional[np.ndarray]] = []
    off = 0
    for c, _ in parts:
        n = _ncols(c, w.numel)
        masks.append(None if orc.rms_cols is None else orc.rms_cols[off:off + n])
        off += n
    bf16x = w.param_dtype == "bf16"

    def ostate(st: oracle.OracleState, k: int) -> np.ndarray:
        arrs = st.arrays()
        if k < len(arrs):
            return arrs[k]
        return (st.x_outer if names[k] == "x_outer" else st.outer_mom).reshape(1, -1)

    xo_rms = _rms([(ostate(st, names.index("x_outer")), m) for (_, st), m in zip(parts, masks)], False) if nest else 0.0
    report: Dict[str, Dict[str, float]] = {}
    with ThreadPoolExecutor(oracle_threads()) as ex:
        for k, name in enumerate(names):
            is_bf16 = name == "x" and bf16x
            rms = _rms([(ostate(st, k), m) for (_, st), m in zip(parts, masks)], is_bf16)
            if name in ("x_outer", "outer_mom") and (bf16x or name == "outer_mom"):
                kind = "outer"
            else:
                kind = "bf16" if is_bf16 else "f32"

            def one(i: int, k=k, kind=kind, rms=rms, is_bf16=is_bf16) -> Dict[str, float]:
                c, st = parts[i]
                a = gather_state(gs[k], c)
                b = ostate(st, k)
                ref = None
                if kind == "outer":
                    ref = ostate(st, names.index("x_outer"))
                elif kind == "bf16":
                    assert orc.x_absmax is not None and orc.x_absmax[i] is not None, \
                        "bf16 parameters are compared at their trajectory's largest magnitude (XAbsMax)"
                    ref = orc.x_absmax[i]
                step = max(1, _CHUNK // a.shape[0])
                return _merge([_metrics(kind, a[:, lo:lo + step], b[:, lo:lo + step], rms,
                                        None if ref is None else ref[:, lo:lo + step], xo_rms, is_bf16)
                               for lo in range(0, a.shape[1], step)])

            m = _merge(list(ex.map(one, range(len(parts)))))
            m["rms_floor"] = rms
            report[name] = m
    worst = {}
    for name, m in report.items():
        assert m["finite"] == 1.0, (label, name, "non-finite values")
        if "rel_err" in m and "max_ulps" not in m:
            log(f"  {label} {name}: rel_err={m['rel_err']:.3e} (unfloored {m['rel_err_unfloored']:.3e}, "
                f"max|a-b|/max|b|={m['max_abs_diff'] / max(m['max_abs_want'], 1e-300):.3e})")
            assert m["rel_err"] <= REL_TOL, (label, name, m)
            worst[name] = m["rel_err"]
        elif "max_ulps" in m:
            fge, fgt = m["n_ge1"] / m["n"], m["n_gt1"] / m["n"]
            steps = orc.steps if orc.steps is not None else len(orc.masks)
            log(f"  {label} {name}: max_ulps={m['max_ulps']:.3g} frac>=1ulp={fge:.3e} frac>1ulp={fgt:.3e} "
                f"steps={steps} rel_err={m['rel_err']:.3e}")
            if nest:
                # every worker restarts from the outer parameters, which carry
                # flips amplified by lr (1 + mu) / (1 - mu)
                assert m["max_ulps"] <= BF16_OUTER_MAX_ULPS and fge <= BF16_OUTER_FRAC, (label, name, m)
            else:
                ge_max, gt_max = bf16_bounds(m["n"], steps)
                assert m["max_ulps"] <= BF16_MAX_ULPS, (label, name, m)
                assert m["n_ge1"] <= ge_max and m["n_gt1"] <= gt_max, (label, name, m, ge_max, gt_max)
            worst[name + "_ulps"] = m["max_ulps"]
            worst[name + "_frac_ge1"] = fge
        else:
            frac_off = m["n_off"] / m["n"]
            log(f"  {label} {name}: err/scale(x_outer)={m['err_of_x_outer']:.3e} ulps(x_outer)="
                f"{m['max_ulps_of_x']:.3g} frac_off={frac_off:.3e}")
            if bf16x:
                # A bf16 rounding flip of one worker's x moves the worker mean
                # by ulp(x)/K; the Nesterov step carries it into the outer
                # parameters with gain lr (1 + mu) and into the momentum, which
                # keeps it for 1/(1 - mu) events: bounded in bf16 ulps of the
                # outer parameters, the affected fraction by the flip rate.
                assert m["max_ulps_of_x"] <= BF16_OUTER_MAX_ULPS and frac_off <= BF16_OUTER_FRAC, (label, name, m)
            else:
                # b sums outer gradients d = x_outer - E_m[x^m] with |d| << |x|,
                # so its fp32 rounding errors are those of x-scale operands: it
                # is held to the 1e-5 bound at the scale of the outer parameters
                assert m["err_of_x_outer"] <= REL_TOL, (label, name, m)
            worst[name + "_of_x_outer"] = m["err_of_x_outer"]
    REPORT.append((label, worst))
    return report


def free(*objs) -> None:
    for o in objs:
        if isinstance(o, GpuResult):
            o.opt.close()
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
