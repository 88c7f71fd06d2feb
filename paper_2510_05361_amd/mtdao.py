"""ctypes binding of the C ABI in include/mtdao.h (argument marshalling only).

Function names match the C entry points.  Device buffers are passed as raw
pointers (ints, e.g. ``tensor.data_ptr()``) and streams as raw HIP stream
handles (``torch.cuda.current_stream().cuda_stream``); every step of the
optimizer runs in the HIP kernels of ``libmtdao.so``.  There is no CPU
fallback: if the library is missing, loading fails with an error.
"""

from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libmtdao.so")

MTDAO_MAX_N = 4
MTDAO_MAX_REPLICAS = 1024
MTDAO_SYNC_AUTO = 0xFFFFFFFF
MTDAO_ADAM, MTDAO_ADOPT, MTDAO_SGDM = 0, 1, 2
MTDAO_F32, MTDAO_BF16 = 0, 1
MTDAO_ADOPT_PREV, MTDAO_ADOPT_CUR = 0, 1
MTDAO_SYNC_AFTER_STEP, MTDAO_SYNC_MOMENTA_IN_STEP = 0, 1
MTDAO_OUTER_AVERAGE, MTDAO_OUTER_NESTEROV = 0, 1
MTDAO_STATE_X_OUTER, MTDAO_STATE_OUTER_MOM = 6, 7
MTDAO_STATS_MAX_REPLICAS, MTDAO_STATS_STRIDE = 16, 36
MTDAO_STAT_MEAN_SQ, MTDAO_STAT_VARIANCE, MTDAO_STAT_OUTER_SQ = 0, 1, 2
MTDAO_STAT_WORKER_SQ, MTDAO_STAT_WORKER_DOT = 4, 20
MTDAO_OK = 0
MTDAO_ERR_INVALID_ARG = -1
MTDAO_ERR_ALIGN = -2
MTDAO_ERR_HIP = -3
MTDAO_ERR_RANGE = -4
MTDAO_ERR_WORKSPACE = -5
MTDAO_STATIC_SCRATCH_BYTES = 64 << 20

FORMS = {"adam": MTDAO_ADAM, "adopt": MTDAO_ADOPT, "sgdm": MTDAO_SGDM}
DTYPES = {"f32": MTDAO_F32, "bf16": MTDAO_BF16}
ORDERS = {"prev": MTDAO_ADOPT_PREV, "cur": MTDAO_ADOPT_CUR}


class MtdaoError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"mtdao error {code}: {msg}")
        self.code = code


class MtdaoConfig(ctypes.Structure):
    _fields_ = [
        ("form", ctypes.c_int32), ("replicas", ctypes.c_int32), ("n_moments", ctypes.c_int32),
        ("param_dtype", ctypes.c_int32), ("grad_dtype", ctypes.c_int32),
        ("adopt_order", ctypes.c_int32), ("bias_correction", ctypes.c_int32),
        ("beta1", ctypes.c_float * MTDAO_MAX_N), ("omega", ctypes.c_float * MTDAO_MAX_N),
        ("beta2", ctypes.c_float), ("eps", ctypes.c_float), ("clip_rho", ctypes.c_float),
        ("period_x", ctypes.c_int32), ("period_u", ctypes.c_int32 * MTDAO_MAX_N),
        ("period_v", ctypes.c_int32), ("start_step", ctypes.c_int64), ("numel", ctypes.c_int64),
        ("n_tensors", ctypes.c_int32), ("tensor_numel", ctypes.POINTER(ctypes.c_int64)),
        ("sync_order", ctypes.c_int32), ("outer_opt", ctypes.c_int32), ("outer_lr", ctypes.c_float),
        ("outer_momentum", ctypes.c_float),
    ]


class MtdaoBuffers(ctypes.Structure):
    _fields_ = [
        ("x", ctypes.c_void_p), ("u", ctypes.c_void_p * MTDAO_MAX_N), ("v", ctypes.c_void_p),
        ("init_states", ctypes.c_int32), ("x_outer", ctypes.c_void_p), ("x_outer_mom", ctypes.c_void_p),
    ]


_lib = None


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"HIP library {LIB_PATH} is not built "
                               "(python -m paper_2510_05361_amd.build)")
        L = ctypes.CDLL(LIB_PATH)
        P, VP, I32, I64, U32 = ctypes.POINTER, ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_uint32
        L.mtdao_workspace_bytes.argtypes = [P(MtdaoConfig), P(ctypes.c_size_t)]
        L.mtdao_workspace_bytes.restype = I32
        L.mtdao_init.argtypes = [P(MtdaoConfig), P(MtdaoBuffers), VP, ctypes.c_size_t, VP, P(VP)]
        L.mtdao_init.restype = I32
        L.mtdao_local_step.argtypes = [VP, VP, ctypes.c_float, ctypes.c_float, VP]
        L.mtdao_local_step.restype = I32
        L.mtdao_sync.argtypes = [VP, U32, P(U32), VP]
        L.mtdao_sync.restype = I32
        L.mtdao_step_sync.argtypes = [VP, VP, ctypes.c_float, ctypes.c_float, U32, P(U32), VP]
        L.mtdao_step_sync.restype = I32
        L.mtdao_stats_scratch_bytes.argtypes = [P(MtdaoConfig), P(ctypes.c_size_t)]
        L.mtdao_stats_scratch_bytes.restype = I32
        L.mtdao_sync_stats.argtypes = [VP, U32, P(U32), VP, ctypes.c_size_t, VP, VP]
        L.mtdao_sync_stats.restype = I32
        L.mtdao_sync_stats_static.argtypes = [VP, U32, P(U32), VP, VP]
        L.mtdao_sync_stats_static.restype = I32
        L.mtdao_device_step_set.argtypes = [VP, VP, I64, VP]
        L.mtdao_device_step_set.restype = I32
        L.mtdao_step_sync_device.argtypes = [VP, VP, VP, VP, VP, I64, U32, P(U32), VP]
        L.mtdao_step_sync_device.restype = I32
        L.mtdao_device_step_advance.argtypes = [VP, VP, VP]
        L.mtdao_device_step_advance.restype = I32
        L.mtdao_schedule.argtypes = [P(MtdaoConfig), I64, P(U32)]
        L.mtdao_schedule.restype = I32
        L.mtdao_read_state.argtypes = [VP, I32, I32, I64, I64, VP, VP]
        L.mtdao_read_state.restype = I32
        L.mtdao_step_count.argtypes = [VP]
        L.mtdao_step_count.restype = I64
        L.mtdao_last_error.argtypes = [VP]
        L.mtdao_last_error.restype = ctypes.c_char_p
        L.mtdao_destroy.argtypes = [VP]
        L.mtdao_destroy.restype = None
        _lib = L
    return _lib


def _check(code: int, handle=None) -> None:
    if code != MTDAO_OK:
        raise MtdaoError(code, lib().mtdao_last_error(handle).decode())


def make_config(form: str, replicas: int, beta1: Sequence[float], omega: Sequence[float],
                numel: int, beta2: float = 0.999, eps: float = 1e-8, clip_rho: float = 0.0,
                param_dtype: str = "f32", grad_dtype: str = "f32", adopt_order: str = "prev",
                bias_correction: bool = True, period_x: int = 0,
                period_u: Sequence[int] = (0,), period_v: int = 0, start_step: int = 0,
                tensor_numel: Optional[Sequence[int]] = None, sync_order: int = 0,
                outer_opt: int = 0, outer_lr: float = 1.0, outer_momentum: float = 0.0) -> MtdaoConfig:
    """Fill an ``mtdao_config``.  The returned structure keeps a reference to
    its tensor-size array (``_tensor_arr``) for as long as it lives."""
    n = len(beta1)
    c = MtdaoConfig()
    c.form = FORMS[form] if isinstance(form, str) else int(form)
    c.replicas = int(replicas)
    c.n_moments = n
    c.param_dtype = DTYPES[param_dtype] if isinstance(param_dtype, str) else int(param_dtype)
    c.grad_dtype = DTYPES[grad_dtype] if isinstance(grad_dtype, str) else int(grad_dtype)
    c.adopt_order = ORDERS[adopt_order] if isinstance(adopt_order, str) else int(adopt_order)
    c.bias_correction = int(bool(bias_correction))
    for j in range(min(n, MTDAO_MAX_N)):
        c.beta1[j] = beta1[j]
        c.omega[j] = omega[j]
        c.period_u[j] = int(period_u[j] if j < len(period_u) else period_u[-1])
    c.beta2 = beta2
    c.eps = eps
    c.clip_rho = clip_rho
    c.period_x = int(period_x)
    c.period_v = int(period_v)
    c.start_step = int(start_step)
    c.numel = int(numel)
    c.sync_order = int(sync_order)
    c.outer_opt = int(outer_opt)
    c.outer_lr = outer_lr
    c.outer_momentum = outer_momentum
    if tensor_numel is not None and len(tensor_numel) > 0:
        arr = (ctypes.c_int64 * len(tensor_numel))(*[int(t) for t in tensor_numel])
        c.n_tensors = len(tensor_numel)
        c.tensor_numel = ctypes.cast(arr, ctypes.POINTER(ctypes.c_int64))
        c._tensor_arr = arr
    else:
        c.n_tensors = 0
        c.tensor_numel = None
    return c


def config_from_workload(w, start_step: int = 0, numel: Optional[int] = None,
                         tensor_numel: Optional[Sequence[int]] = None, sync_order: int = 0,
                outer_opt: int = 0, outer_lr: float = 1.0, outer_momentum: float = 0.0) -> MtdaoConfig:
    """``mtdao_config`` of a ``synth.Workload``."""
    tn = [t.numel for t in w.tensors] if tensor_numel is None and numel is None else tensor_numel
    return make_config(w.form, w.replicas, w.beta1, w.omega, w.numel if numel is None else numel,
                       beta2=w.beta2, eps=w.eps, clip_rho=w.clip_rho, param_dtype=w.param_dtype,
                       grad_dtype=w.grad_dtype, adopt_order=w.adopt_order, bias_correction=w.bias_correction,
                       period_x=w.period_x, period_u=w.period_u, period_v=w.period_v,
                       start_step=start_step, tensor_numel=tn, sync_order=sync_order, outer_opt=outer_opt,
                       outer_lr=outer_lr, outer_momentum=outer_momentum)


def mtdao_workspace_bytes(cfg: MtdaoConfig) -> int:
    out = ctypes.c_size_t(0)
    _check(lib().mtdao_workspace_bytes(ctypes.byref(cfg), ctypes.byref(out)))
    return int(out.value)


def mtdao_schedule(cfg: MtdaoConfig, s: int) -> int:
    out = ctypes.c_uint32(0)
    _check(lib().mtdao_schedule(ctypes.byref(cfg), int(s), ctypes.byref(out)))
    return int(out.value)


def make_buffers(x: int, u: Sequence[int], v: Optional[int], init_states: bool,
                 x_outer: Optional[int] = None, x_outer_mom: Optional[int] = None) -> MtdaoBuffers:
    b = MtdaoBuffers()
    b.x = x
    b.x_outer = x_outer
    b.x_outer_mom = x_outer_mom
    for j, p in enumerate(u):
        b.u[j] = p
    b.v = v
    b.init_states = int(bool(init_states))
    return b


def mtdao_init(cfg: MtdaoConfig, bufs: MtdaoBuffers, workspace: Optional[int], workspace_bytes: int,
               stream: Optional[int]) -> int:
    h = ctypes.c_void_p()
    _check(lib().mtdao_init(ctypes.byref(cfg), ctypes.byref(bufs), workspace, int(workspace_bytes),
                            stream, ctypes.byref(h)))
    return int(h.value)


def mtdao_local_step(h: int, grads: int, lr: float, adopt_clip: float, stream: Optional[int]) -> None:
    _check(lib().mtdao_local_step(h, grads, float(lr), float(adopt_clip), stream), h)


def mtdao_sync(h: int, mask: int, stream: Optional[int]) -> int:
    applied = ctypes.c_uint32(0)
    _check(lib().mtdao_sync(h, int(mask) & 0xFFFFFFFF, ctypes.byref(applied), stream), h)
    return int(applied.value)


def mtdao_step_sync(h: int, grads: int, lr: float, adopt_clip: float, mask: int,
                    stream: Optional[int]) -> int:
    applied = ctypes.c_uint32(0)
    _check(lib().mtdao_step_sync(h, grads, float(lr), float(adopt_clip), int(mask) & 0xFFFFFFFF,
                                 ctypes.byref(applied), stream), h)
    return int(applied.value)


def mtdao_stats_scratch_bytes(cfg: MtdaoConfig) -> int:
    out = ctypes.c_size_t(0)
    _check(lib().mtdao_stats_scratch_bytes(ctypes.byref(cfg), ctypes.byref(out)))
    return int(out.value)


def mtdao_sync_stats(h: int, mask: int, scratch: Optional[int], scratch_bytes: int,
                     stream: Optional[int]):
    """Returns (applied mask, stats array [MTDAO_MAX_N + 2][MTDAO_STATS_STRIDE])."""
    applied = ctypes.c_uint32(0)
    out = np.empty((MTDAO_MAX_N + 2, MTDAO_STATS_STRIDE), dtype=np.float64)
    _check(lib().mtdao_sync_stats(h, int(mask) & 0xFFFFFFFF, ctypes.byref(applied), scratch, int(scratch_bytes),
                                  out.ctypes.data, stream), h)
    return int(applied.value), out


def mtdao_sync_stats_static(h: int, mask: int, stream: Optional[int]):
    """mtdao_sync_stats on the library's static device scratch (no caller
    buffer).  Returns (applied mask, stats array)."""
    applied = ctypes.c_uint32(0)
    out = np.empty((MTDAO_MAX_N + 2, MTDAO_STATS_STRIDE), dtype=np.float64)
    _check(lib().mtdao_sync_stats_static(h, int(mask) & 0xFFFFFFFF, ctypes.byref(applied), out.ctypes.data,
                                         stream), h)
    return int(applied.value), out


class MtdaoDeviceStep(ctypes.Structure):
    """Layout of mtdao_device_step (the block lives in device memory)."""
    _fields_ = [("s", ctypes.c_int64), ("reserved", ctypes.c_int64)]


MTDAO_DEVICE_STEP_BYTES = ctypes.sizeof(MtdaoDeviceStep)


def mtdao_device_step_set(h: int, d: int, s: int, stream: Optional[int]) -> None:
    _check(lib().mtdao_device_step_set(h, d, int(s), stream), h)


def mtdao_step_sync_device(h: int, grads: int, d: int, lr_table: int, clip_table: Optional[int], table_len: int,
                           mask: int, stream: Optional[int]) -> int:
    """mtdao_step_sync with the update number taken on the device (d:
    mtdao_device_step, tables: device fp32 arrays); returns the applied
    mask."""
    applied = ctypes.c_uint32(0)
    _check(lib().mtdao_step_sync_device(h, grads, d, lr_table, clip_table, int(table_len), int(mask) & 0xFFFFFFFF,
                                        ctypes.byref(applied), stream), h)
    return int(applied.value)


def mtdao_device_step_advance(h: int, d: int, stream: Optional[int]) -> None:
    _check(lib().mtdao_device_step_advance(h, d, stream), h)


def mtdao_read_state(h: int, state: int, replica: int, offset: int, count: int,
                     host_dst: np.ndarray, stream: Optional[int]) -> None:
    assert host_dst.flags.c_contiguous
    _check(lib().mtdao_read_state(h, int(state), int(replica), int(offset), int(count),
                                  host_dst.ctypes.data, stream), h)


def mtdao_step_count(h: int) -> int:
    return int(lib().mtdao_step_count(h))


def mtdao_last_error(h: Optional[int]) -> str:
    return lib().mtdao_last_error(h).decode()


def mtdao_destroy(h: Optional[int]) -> None:
    lib().mtdao_destroy(h)
