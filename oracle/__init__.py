"""Python driver of the CPU oracle (test infrastructure only).

Only ``tests/``, the smoke check and the benchmark's CPU-baseline leg may
import this package.  The GPU library never calls it and never falls back
to it.

The arithmetic lives in ``mtdao_oracle.c`` (plain C, fp64).  This module
marshals numpy arrays into it and strings the calls together in the order of
the paper's algorithms: for every global step s = 1..T, every worker's local
update (Algorithm 1, 2 or 3 body), then the replica mean of each state whose
period divides s.
"""

from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass
from typing import Callable, List, Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "mtdao_oracle.c")
# MTDAO_ORACLE_SANITIZE=1 selects a build with AddressSanitizer and
# UndefinedBehaviorSanitizer (load it with gcc's libasan preloaded).
SANITIZE = os.environ.get("MTDAO_ORACLE_SANITIZE") == "1"
SAN_FLAGS = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-g"]
_LIB = os.path.join(_HERE, "_liboracle_san.so" if SANITIZE else "_liboracle.so")

MAX_N = 4
F32, BF16, F64 = 0, 1, 2
ADAM, ADOPT, SGDM = 0, 1, 2
ADOPT_PREV, ADOPT_CUR = 0, 1

_FORMS = {"adam": ADAM, "adopt": ADOPT, "sgdm": SGDM}
_DTYPES = {"f32": F32, "bf16": BF16, "f64": F64}
_NP_DTYPE = {F32: np.float32, BF16: np.uint16, F64: np.float64}


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (no fast-math, no FMA contraction; with
    the sanitizers when MTDAO_ORACLE_SANITIZE=1)."""
    if force or not os.path.exists(_LIB):
        cmd = ["gcc", "-O2", "-std=c11", "-ffp-contract=off", "-fno-fast-math", "-fPIC", "-shared",
               "-Wall", "-Wextra", *(SAN_FLAGS if SANITIZE else []), "-o", _LIB + ".tmp", _SRC, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(_LIB + ".tmp", _LIB)
    return _LIB


class _Cfg(ctypes.Structure):
    _fields_ = [
        ("form", ctypes.c_int32), ("n", ctypes.c_int32), ("x_dtype", ctypes.c_int32),
        ("g_dtype", ctypes.c_int32), ("m_dtype", ctypes.c_int32),
        ("bias_correction", ctypes.c_int32), ("adopt_order", ctypes.c_int32),
        ("beta1", ctypes.c_float * MAX_N), ("omega", ctypes.c_float * MAX_N),
        ("beta2", ctypes.c_float), ("eps", ctypes.c_float),
    ]


_lib = None
_lib_path = _LIB


def use_library(path: str) -> None:
    """Point this driver at another build of the oracle source (the mutation
    tests load deliberately broken copies)."""
    global _lib, _lib_path
    _lib, _lib_path = None, path


def lib():
    global _lib
    if _lib is None:
        if _lib_path == _LIB and not os.path.exists(_LIB):
            build()
        L = ctypes.CDLL(_lib_path)
        L.oracle_schedule.restype = ctypes.c_uint32
        L.oracle_schedule.argtypes = [ctypes.c_int64, ctypes.c_int32, ctypes.c_int32,
                                      ctypes.POINTER(ctypes.c_int32), ctypes.c_int32, ctypes.c_int32]
        L.oracle_sumsq.restype = ctypes.c_double
        L.oracle_sumsq.argtypes = [ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64]
        L.oracle_clip_scale.restype = ctypes.c_double
        L.oracle_clip_scale.argtypes = [ctypes.c_double, ctypes.c_double]
        L.oracle_local_step.restype = None
        L.oracle_local_step.argtypes = [ctypes.POINTER(_Cfg), ctypes.c_int64, ctypes.c_float,
                                        ctypes.c_float, ctypes.c_void_p, ctypes.c_void_p,
                                        ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                        ctypes.c_int64, ctypes.c_int64]
        L.oracle_replica_mean.restype = None
        L.oracle_outer_nesterov.restype = None
        L.oracle_outer_nesterov.argtypes = [ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p,
                                            ctypes.c_float, ctypes.c_float, ctypes.c_int64, ctypes.c_int64]
        L.oracle_state_stats.restype = None
        L.oracle_state_stats.argtypes = [ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p, ctypes.c_int64,
                                         ctypes.c_int64, ctypes.c_void_p]
        L.oracle_sgdm_prob_step.restype = None
        L.oracle_sgdm_prob_step.argtypes = [ctypes.POINTER(_Cfg), ctypes.c_float, ctypes.c_uint32,
                                            ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                            ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64]
        L.oracle_replica_mean.argtypes = [ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64,
                                          ctypes.c_int64]
        _lib = L
    return _lib


@dataclass
class OracleConfig:
    """Hyper-parameters of one optimizer (the Require blocks of Algorithms
    1-3).  ``beta1``/``omega`` hold beta_{1,j} and omega_j; periods are the
    paper's K_x, K_j, K_v (0 = never)."""

    form: str
    beta1: Sequence[float]
    omega: Sequence[float]
    beta2: float = 0.999
    eps: float = 1e-8
    clip_rho: float = 0.0
    bias_correction: bool = True
    adopt_order: str = "prev"
    x_dtype: str = "f32"
    g_dtype: str = "f32"
    m_dtype: str = "f32"
    period_x: int = 1
    period_u: Sequence[int] = (1,)
    period_v: int = 1
    outer: str = "average"          # OuterOpt at x events: "average" | "nesterov"
    outer_lr: float = 1.0
    outer_momentum: float = 0.0

    @property
    def n(self) -> int:
        return len(self.beta1)

    @property
    def has_v(self) -> bool:
        return self.form in ("adam", "adopt")

    def c_struct(self) -> _Cfg:
        c = _Cfg()
        c.form = _FORMS[self.form]
        c.n = self.n
        c.x_dtype = _DTYPES[self.x_dtype]
        c.g_dtype = _DTYPES[self.g_dtype]
        c.m_dtype = _DTYPES[self.m_dtype]
        c.bias_correction = int(bool(self.bias_correction))
        c.adopt_order = ADOPT_PREV if self.adopt_order == "prev" else ADOPT_CUR
        for j in range(self.n):
            c.beta1[j] = self.beta1[j]
            c.omega[j] = self.omega[j]
        c.beta2 = self.beta2
        c.eps = self.eps
        return c

    @classmethod
    def from_workload(cls, w, m_dtype: str = "f32", outer: str = "average", outer_lr: float = 1.0,
                      outer_momentum: float = 0.0) -> "OracleConfig":
        return cls(form=w.form, beta1=tuple(w.beta1), omega=tuple(w.omega), beta2=w.beta2,
                   eps=w.eps, clip_rho=w.clip_rho, bias_correction=w.bias_correction, adopt_order=w.adopt_order,
                   x_dtype=w.param_dtype, g_dtype=w.grad_dtype, m_dtype=m_dtype,
                   period_x=w.period_x, period_u=tuple(w.period_u), period_v=w.period_v,
                   outer=outer, outer_lr=outer_lr, outer_momentum=outer_momentum)


def _ptr(a: np.ndarray) -> int:
    assert a.flags.c_contiguous
    return a.ctypes.data


def schedule(cfg: OracleConfig, s: int) -> int:
    pu = (ctypes.c_int32 * MAX_N)(*([int(p) for p in cfg.period_u] + [0] * (MAX_N - cfg.n)))
    return int(lib().oracle_schedule(int(s), cfg.n, int(cfg.period_x), pu, int(cfg.period_v),
                                     int(cfg.has_v)))


def sumsq(g: np.ndarray, g_dtype: str = "f32") -> float:
    dt = _DTYPES[g_dtype]
    a = np.ascontiguousarray(g, dtype=_NP_DTYPE[dt])
    return float(lib().oracle_sumsq(_ptr(a), dt, a.size))


def clip_scale(norm: float, rho: float) -> float:
    return float(lib().oracle_clip_scale(float(norm), float(rho)))


def clip_scales(cfg: OracleConfig, g: np.ndarray) -> Optional[np.ndarray]:
    """Per-worker clip factors for a [K][P] gradient (None when clip is off)."""
    if not cfg.clip_rho > 0:
        return None
    return np.array([clip_scale(np.sqrt(sumsq(g[m], cfg.g_dtype)), cfg.clip_rho)
                     for m in range(g.shape[0])], dtype=np.float64)


@dataclass
class OracleState:
    """All per-worker states, [K][P] arrays in their storage types; with a
    Nesterov OuterOpt also the outer parameters and momentum (fp32 [P])."""

    x: np.ndarray
    u: List[np.ndarray]
    v: Optional[np.ndarray]
    x_outer: Optional[np.ndarray] = None
    outer_mom: Optional[np.ndarray] = None

    def copy(self) -> "OracleState":
        return OracleState(self.x.copy(), [a.copy() for a in self.u],
                           None if self.v is None else self.v.copy(),
                           None if self.x_outer is None else self.x_outer.copy(),
                           None if self.outer_mom is None else self.outer_mom.copy())

    def arrays(self) -> List[np.ndarray]:
        return [self.x] + list(self.u) + ([self.v] if self.v is not None else [])


def new_state(cfg: OracleConfig, x0_row: np.ndarray, K: int) -> OracleState:
    """Every worker starts from the same x_0; first and second moments start
    at zero (the initial u_{-1} = 0 of the analysis)."""
    xd = _NP_DTYPE[_DTYPES[cfg.x_dtype]]
    md = _NP_DTYPE[_DTYPES[cfg.m_dtype]]
    P = x0_row.size
    x = np.repeat(np.asarray(x0_row, dtype=xd).reshape(1, P), K, axis=0)  # always a fresh copy
    u = [np.zeros((K, P), dtype=md) for _ in range(cfg.n)]
    v = np.zeros((K, P), dtype=md) if cfg.has_v else None
    st = OracleState(x, u, v)
    if cfg.outer == "nesterov":
        xf = np.asarray(x0_row)
        if cfg.x_dtype == "bf16":
            xf = (xf.astype(np.uint32) << np.uint32(16)).view(np.float32)
        st.x_outer = np.array(xf, dtype=np.float32).reshape(P)
        st.outer_mom = np.zeros(P, dtype=np.float32)
    return st


def local_step(cfg: OracleConfig, st: OracleState, g: np.ndarray, s: int, lr: float,
               clip_c: float = 0.0, scale: Optional[np.ndarray] = None) -> None:
    K, P = st.x.shape
    gd = _NP_DTYPE[_DTYPES[cfg.g_dtype]]
    g = np.ascontiguousarray(g, dtype=gd)
    assert g.shape == (K, P)
    uarr = (ctypes.c_void_p * MAX_N)(*([_ptr(a) for a in st.u] + [None] * (MAX_N - cfg.n)))
    sc = None
    if scale is not None:
        scale = np.ascontiguousarray(scale, dtype=np.float64)
        sc = _ptr(scale)
    c = cfg.c_struct()
    lib().oracle_local_step(ctypes.byref(c), int(s), float(lr), float(clip_c), sc, _ptr(st.x),
                            ctypes.cast(uarr, ctypes.c_void_p),
                            None if st.v is None else _ptr(st.v), _ptr(g), K, P)


def sgdm_prob_step(cfg: OracleConfig, st: OracleState, g: np.ndarray, lr: float, mask: int,
                   scale: Optional[np.ndarray] = None) -> None:
    """One step of the probabilistic SGDM variant (Algorithm 4) with this
    step's averaging events ``mask``; averaged moments feed this step's
    update."""
    assert cfg.form == "sgdm"
    K, P = st.x.shape
    g = np.ascontiguousarray(g, dtype=_NP_DTYPE[_DTYPES[cfg.g_dtype]])
    uarr = (ctypes.c_void_p * MAX_N)(*([_ptr(a) for a in st.u] + [None] * (MAX_N - cfg.n)))
    sc = None
    if scale is not None:
        scale = np.ascontiguousarray(scale, dtype=np.float64)
        sc = _ptr(scale)
    c = cfg.c_struct()
    lib().oracle_sgdm_prob_step(ctypes.byref(c), float(lr), int(mask) & 0xFFFFFFFF, sc, _ptr(st.x),
                                ctypes.cast(uarr, ctypes.c_void_p), _ptr(g), K, P)


def run_probabilistic(cfg: OracleConfig, st: OracleState, grads: Callable[[int], np.ndarray],
                      steps: Sequence[int], lr: Callable[[int], float], masks: Callable[[int], int],
                      scales: Optional[Callable[[int, np.ndarray], Optional[np.ndarray]]] = None) -> List[int]:
    """Algorithm 4 over global steps ``steps`` with caller-drawn events."""
    applied = []
    for s in steps:
        g = grads(s)
        sc = scales(s, g) if scales is not None else clip_scales(cfg, g)
        m = masks(s)
        sgdm_prob_step(cfg, st, g, lr(s), m, sc)
        applied.append(m)
    return applied


def replica_mean(a: np.ndarray, dtype: str) -> None:
    K, P = a.shape
    lib().oracle_replica_mean(_ptr(a), _DTYPES[dtype], K, P)


def outer_nesterov(cfg: OracleConfig, st: OracleState) -> None:
    """Nesterov OuterOpt at an averaging event of x (in place)."""
    K, P = st.x.shape
    assert st.x_outer is not None and st.outer_mom is not None
    lib().oracle_outer_nesterov(_ptr(st.x), _DTYPES[cfg.x_dtype], _ptr(st.x_outer), _ptr(st.outer_mom),
                                float(cfg.outer_lr), float(cfg.outer_momentum), K, P)


def state_stats(a: np.ndarray, dtype: str, x_outer: Optional[np.ndarray] = None) -> np.ndarray:
    """Diagnostics of a [K][P] state before it is averaged (see
    oracle_state_stats): [||cbar||^2, cross-worker variance, ||x_outer||^2, 0,
    ||c^m||^2 (K), <c^m, cbar> (K)], c^m = S^m or x_outer - x^m."""
    K, P = a.shape
    out = np.zeros(4 + 2 * K, dtype=np.float64)
    xo = None
    if x_outer is not None:
        x_outer = np.ascontiguousarray(x_outer, dtype=np.float32)
        xo = _ptr(x_outer)
    lib().oracle_state_stats(_ptr(a), _DTYPES[dtype], xo, K, P, _ptr(out))
    return out


def sync_stats(cfg: OracleConfig, st: OracleState, mask: int) -> dict:
    """Diagnostics of every state in mask from its pre-average values, then
    the averaging itself.  Returns {state id: stats array}."""
    out = {}
    if mask & 1:
        out[0] = state_stats(st.x, cfg.x_dtype, st.x_outer if cfg.outer == "nesterov" else None)
    for j in range(cfg.n):
        if mask & (1 << (j + 1)):
            out[j + 1] = state_stats(st.u[j], cfg.m_dtype)
    if st.v is not None and mask & (1 << (cfg.n + 1)):
        out[cfg.n + 1] = state_stats(st.v, cfg.m_dtype)
    sync(cfg, st, mask)
    return out


def sync(cfg: OracleConfig, st: OracleState, mask: int) -> None:
    """Average every state whose bit is set in ``mask`` (bit 0 = x, bit j =
    u^j, bit N+1 = v)."""
    if mask & 1:
        if cfg.outer == "nesterov":
            outer_nesterov(cfg, st)
        else:
            replica_mean(st.x, cfg.x_dtype)
    for j in range(cfg.n):
        if mask & (1 << (j + 1)):
            replica_mean(st.u[j], cfg.m_dtype)
    if st.v is not None and mask & (1 << (cfg.n + 1)):
        replica_mean(st.v, cfg.m_dtype)


def run(cfg: OracleConfig, st: OracleState, grads: Callable[[int], np.ndarray], steps: Sequence[int],
        lr: Callable[[int], float], clip_c: Callable[[int], float] = lambda s: 0.0,
        scales: Optional[Callable[[int, np.ndarray], Optional[np.ndarray]]] = None,
        masks: Optional[Callable[[int], int]] = None) -> List[int]:
    """Run local steps ``steps`` (global 1-based numbers) in place: local
    update of every worker, then the averaging of the states due at s.
    ``scales(s, g)`` may supply the per-worker clip factors (default: from
    the full gradient ``g``); ``masks(s)`` may override the schedule.
    Returns the applied mask of every step."""
    applied = []
    for s in steps:
        g = grads(s)
        sc = scales(s, g) if scales is not None else clip_scales(cfg, g)
        local_step(cfg, st, g, s, lr(s), clip_c(s), sc)
        mask = masks(s) if masks is not None else schedule(cfg, s)
        sync(cfg, st, mask)
        applied.append(mask)
    return applied
