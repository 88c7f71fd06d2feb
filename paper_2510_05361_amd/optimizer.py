"""Torch-side holder of one MT-DAO optimizer instance.

Torch only allocates the device buffers ([K][P] state rows, the gradient
rows, the workspace) and supplies the current HIP stream; every step runs in
the library's kernels through the C ABI (``mtdao.py``).
"""

from __future__ import annotations

import itertools
import random
from typing import List, Optional

import torch

from . import mtdao as abi

_TORCH_DTYPE = {abi.MTDAO_F32: torch.float32, abi.MTDAO_BF16: torch.bfloat16}


def _stream() -> int:
    return torch.cuda.current_stream().cuda_stream


class MtdaoOptimizer:
    """States of K worker replicas for one flat multi-tensor parameter
    buffer of P elements, plus the handle that updates them.

    ``x0``: [P] initial parameters (broadcast to every replica), or, with
    ``resume=True``, full [K][P] states ``x``, ``u`` (list of N) and ``v``
    that are taken as they are (e.g. read back from a checkpoint).
    ``grad_buffer``: also carve a [K][P] gradient buffer (``grad``) from the
    states' allocation, for callers that fill gradients in place.
    ``layout``: where the [K][P] buffers (x, the gradient rows, u^1..u^N, v)
    sit in that allocation.  "packed": back to back in that order.
    "tuned" (needs ``grad_buffer``): back to back in the order, among a set
    of candidates, under which the local step ran fastest when timed here
    (``layout_report`` holds the timings).  The HBM rate of a step that
    streams several large buffers at once depends on where they lie
    relative to one another in physical memory, which the process cannot
    see: measured on MI355X, the same step over the same bytes ran at
    74-80% of the peak (K=16, 354M parameters) and 71-79% (K=4, 16.8M)
    depending only on the order of its buffers in the allocation."""

    def __init__(self, cfg: abi.MtdaoConfig, device: torch.device, x0: Optional[torch.Tensor] = None,
                 resume: bool = False, x: Optional[torch.Tensor] = None,
                 u: Optional[List[torch.Tensor]] = None, v: Optional[torch.Tensor] = None,
                 x_outer: Optional[torch.Tensor] = None, x_outer_mom: Optional[torch.Tensor] = None,
                 grad_buffer: bool = False, layout: str = "packed"):
        self.cfg = cfg
        K, P, N = cfg.replicas, cfg.numel, cfg.n_moments
        self.K, self.P, self.N = K, P, N
        self.has_v = cfg.form != abi.MTDAO_SGDM
        xdt = _TORCH_DTYPE[cfg.param_dtype]
        nesterov = cfg.outer_opt == abi.MTDAO_OUTER_NESTEROV
        self.x_outer = self.x_outer_mom = None
        self._arena = None
        self.grad: Optional[torch.Tensor] = None
        self.layout_order: Optional[List[int]] = None
        self.layout_report: Optional[dict] = None
        if resume:
            assert x is not None and u is not None and len(u) == N
            assert (v is not None) == self.has_v
            self.x, self.u, self.v = x, list(u), v
            if nesterov:
                assert x_outer is not None and x_outer_mom is not None
                self.x_outer, self.x_outer_mom = x_outer, x_outer_mom
        else:
            # the [K][P] buffers: x, the gradient rows (when carved here), u^1..u^N, v
            rows = [((K, P), xdt)]
            if grad_buffer:
                rows.append(((K, P), _TORCH_DTYPE[cfg.grad_dtype]))
            rows += [((K, P), torch.float32)] * (N + (1 if self.has_v else 0))
            tail = [((P,), torch.float32)] * 2 if nesterov else []
            order = list(range(len(rows)))
            if layout == "tuned":
                if not grad_buffer:
                    raise ValueError("layout='tuned' times the step over the carved gradient rows: "
                                     "it needs grad_buffer=True")
                order = self._tune_layout(rows, tail, device)
            elif layout != "packed":
                raise ValueError(f"unknown layout {layout!r}")
            self.layout_order = order
            views = self._carve(rows, tail, order, device)
            if grad_buffer:
                self.grad = views.pop(1)
            self.x, self.u = views[0], views[1:1 + N]
            self.v = views[1 + N] if self.has_v else None
            if nesterov:
                self.x_outer, self.x_outer_mom = views[-2], views[-1]
            if x0 is not None:
                self.x[0].copy_(x0.to(device=device, dtype=xdt))
        ws = abi.mtdao_workspace_bytes(cfg)
        self.workspace = torch.empty(max(ws, 1), dtype=torch.uint8, device=device)
        bufs = abi.make_buffers(self.x.data_ptr(), [a.data_ptr() for a in self.u],
                                self.v.data_ptr() if self.v is not None else None, resume,
                                self.x_outer.data_ptr() if self.x_outer is not None else None,
                                self.x_outer_mom.data_ptr() if self.x_outer_mom is not None else None)
        self.handle = abi.mtdao_init(cfg, bufs, self.workspace.data_ptr(), self.workspace.numel(), _stream())

    @staticmethod
    def _nbytes(shape, dt) -> int:
        n = 1
        for d in shape:
            n *= d
        return n * torch.empty((), dtype=dt).element_size()

    def _carve(self, rows, tail, order, device) -> List[torch.Tensor]:
        """Every buffer in one device allocation, each view 256-byte
        aligned: rows[order[0]], rows[order[1]], ..., then the tail buffers.
        Returns the views of rows in their own order, then the tail's.

        Measured on MI355X at 1.31B parameters x 4 replicas: the local step
        over five state buffers allocated one by one ran at 73% of the HBM
        peak in a fresh process (the same in every run), and at 78% over
        the same buffers carved from one allocation."""
        placed = [rows[i] for i in order] + list(tail)
        offs, total = [], 0
        for shape, dt in placed:
            offs.append(total)
            total += (self._nbytes(shape, dt) + 255) // 256 * 256
        if self._arena is None or self._arena.numel() < total:
            self._arena = torch.empty(max(total, 256), dtype=torch.uint8, device=device)
        views = [self._arena[off:off + self._nbytes(shape, dt)].view(dt).view(shape)
                 for (shape, dt), off in zip(placed, offs)]
        out = [None] * len(rows)
        for k, i in enumerate(order):
            out[i] = views[k]
        return out + views[len(rows):]

    def _tune_layout(self, rows, tail, device, max_candidates: int = 24) -> List[int]:
        """The order of rows (x, gradient rows, u^1..u^N, v) under which the
        local step runs fastest over this process's allocation: every order
        when there are at most max_candidates, else the packed order and a
        fixed-seed sample of the others.  Each candidate runs the library's
        local step over zeroed buffers through a handle that keeps the
        states as they are (no initialisation pass): two untimed calls, then
        enough timed calls for about 0.1 s of work."""
        n = len(rows)
        orders = list(itertools.permutations(range(n)))
        if len(orders) > max_candidates:
            rest = orders[1:]
            random.Random(20251006).shuffle(rest)
            orders = orders[:1] + rest[:max_candidates - 1]
        N, cfg = self.N, self.cfg
        ws = torch.empty(max(abi.mtdao_workspace_bytes(cfg), 1), dtype=torch.uint8, device=device)
        stream = torch.cuda.current_stream()
        results = []
        for order in orders:
            views = self._carve(rows, tail, list(order), device)
            if not results:
                self._arena.zero_()
            x, g, u = views[0], views[1], views[2:2 + N]
            v = views[2 + N] if self.has_v else None
            outer = views[n:]
            bufs = abi.make_buffers(x.data_ptr(), [a.data_ptr() for a in u], v.data_ptr() if v is not None else None,
                                    True, outer[0].data_ptr() if outer else None,
                                    outer[1].data_ptr() if outer else None)
            h = abi.mtdao_init(cfg, bufs, ws.data_ptr(), ws.numel(), stream.cuda_stream)
            try:
                for _ in range(2):
                    abi.mtdao_local_step(h, g.data_ptr(), 1e-3, 0.0, stream.cuda_stream)
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record(stream)
                abi.mtdao_local_step(h, g.data_ptr(), 1e-3, 0.0, stream.cuda_stream)
                e1.record(stream)
                e1.synchronize()
                reps = min(50, max(3, int(100.0 / max(e0.elapsed_time(e1), 1e-3))))
                e0.record(stream)
                for _ in range(reps):
                    abi.mtdao_local_step(h, g.data_ptr(), 1e-3, 0.0, stream.cuda_stream)
                e1.record(stream)
                e1.synchronize()
                results.append((e0.elapsed_time(e1) / reps, list(order)))
            finally:
                abi.mtdao_destroy(h)
        best = min(results)
        self.layout_report = {"candidates": len(results), "packed_ms": results[0][0], "best_ms": best[0],
                              "worst_ms": max(results)[0], "order": best[1]}
        return best[1]

    # state id 0 = x, 1..N = u^j, N+1 = v
    def states(self) -> List[torch.Tensor]:
        return [self.x] + self.u + ([self.v] if self.v is not None else [])

    def step(self, grads: torch.Tensor, lr: float, adopt_clip: float = 0.0) -> None:
        assert grads.is_contiguous() and grads.shape == (self.K, self.P)
        abi.mtdao_local_step(self.handle, grads.data_ptr(), lr, adopt_clip, _stream())

    def step_sync(self, grads: torch.Tensor, lr: float, adopt_clip: float = 0.0,
                  mask: int = abi.MTDAO_SYNC_AUTO) -> int:
        """Local step and the averaging of ``mask`` (default: the schedule)
        in one fused pass; returns the applied mask."""
        assert grads.is_contiguous() and grads.shape == (self.K, self.P)
        return abi.mtdao_step_sync(self.handle, grads.data_ptr(), lr, adopt_clip, mask, _stream())

    def device_step(self, lr_table: torch.Tensor, clip_table: Optional[torch.Tensor] = None) -> None:
        """Keep the update number on the device from now on (for HIP graph
        capture): allocates the mtdao_device_step block on first use, sets
        it to the current step count, and keeps the fp32 device tables of
        eta_t (and c_t) indexed by s - 1 that step_sync_device reads (a
        captured graph holds their addresses: keep them alive)."""
        assert lr_table.dtype == torch.float32 and lr_table.is_contiguous() and lr_table.numel() >= 1
        assert clip_table is None or (clip_table.dtype == torch.float32 and clip_table.numel() == lr_table.numel())
        # one block for the optimizer's life: captured graphs keep its address
        if getattr(self, "_dstep", None) is None:
            self._dstep = torch.zeros(abi.MTDAO_DEVICE_STEP_BYTES // 8, dtype=torch.int64, device=self.x.device)
        self._lr_table, self._clip_table = lr_table, clip_table
        abi.mtdao_device_step_set(self.handle, self._dstep.data_ptr(), self.step_count, _stream())

    def step_sync_device(self, grads: torch.Tensor, mask: int = abi.MTDAO_SYNC_AUTO) -> int:
        """step_sync whose eta_t, c_t and bias corrections come from the
        device-side update number (see device_step); the k-th call since the
        last device_step / device_step_advance performs update s + k."""
        assert grads.is_contiguous() and grads.shape == (self.K, self.P)
        clip = self._clip_table.data_ptr() if self._clip_table is not None else None
        return abi.mtdao_step_sync_device(self.handle, grads.data_ptr(), self._dstep.data_ptr(),
                                          self._lr_table.data_ptr(), clip, self._lr_table.numel(), mask, _stream())

    def device_step_advance(self) -> None:
        """Move the device-side update count on by the step_sync_device
        calls since the last device_step or advance (capture it with the
        window it closes)."""
        abi.mtdao_device_step_advance(self.handle, self._dstep.data_ptr(), _stream())

    def sync(self, mask: int = abi.MTDAO_SYNC_AUTO) -> int:
        return abi.mtdao_sync(self.handle, mask, _stream())

    def sync_stats(self, mask: int = abi.MTDAO_SYNC_AUTO):
        """mtdao_sync with the averaging diagnostics of every averaged state;
        returns (applied mask, [state id][stat] array, NaN rows for states not
        averaged).  The scratch buffer is allocated on first use."""
        if getattr(self, "_stats_scratch", None) is None:
            n = abi.mtdao_stats_scratch_bytes(self.cfg)
            self._stats_scratch = torch.empty(n, dtype=torch.uint8, device=self.x.device)
        return abi.mtdao_sync_stats(self.handle, mask, self._stats_scratch.data_ptr(),
                                    self._stats_scratch.numel(), _stream())

    @property
    def step_count(self) -> int:
        return abi.mtdao_step_count(self.handle)

    def close(self) -> None:
        if self.handle:
            abi.mtdao_destroy(self.handle)
            self.handle = 0

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
