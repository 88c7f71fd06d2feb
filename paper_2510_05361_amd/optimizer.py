"""Torch-side holder of one MT-DAO optimizer instance.

Torch only allocates the device buffers ([K][P] state rows, the gradient
rows, the workspace) and supplies the current HIP stream; every step runs in
the library's kernels through the C ABI (``mtdao.py``).
"""

from __future__ import annotations

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
    that are taken as they are (e.g. read back from a checkpoint)."""

    def __init__(self, cfg: abi.MtdaoConfig, device: torch.device, x0: Optional[torch.Tensor] = None,
                 resume: bool = False, x: Optional[torch.Tensor] = None,
                 u: Optional[List[torch.Tensor]] = None, v: Optional[torch.Tensor] = None,
                 x_outer: Optional[torch.Tensor] = None, x_outer_mom: Optional[torch.Tensor] = None):
        self.cfg = cfg
        K, P, N = cfg.replicas, cfg.numel, cfg.n_moments
        self.K, self.P, self.N = K, P, N
        self.has_v = cfg.form != abi.MTDAO_SGDM
        xdt = _TORCH_DTYPE[cfg.param_dtype]
        if resume:
            assert x is not None and u is not None and len(u) == N
            assert (v is not None) == self.has_v
            self.x, self.u, self.v = x, list(u), v
        else:
            self.x = torch.empty((K, P), dtype=xdt, device=device)
            if x0 is not None:
                self.x[0].copy_(x0.to(device=device, dtype=xdt))
            self.u = [torch.empty((K, P), dtype=torch.float32, device=device) for _ in range(N)]
            self.v = torch.empty((K, P), dtype=torch.float32, device=device) if self.has_v else None
        self.x_outer = self.x_outer_mom = None
        if cfg.outer_opt == abi.MTDAO_OUTER_NESTEROV:
            if resume:
                assert x_outer is not None and x_outer_mom is not None
                self.x_outer, self.x_outer_mom = x_outer, x_outer_mom
            else:
                self.x_outer = torch.empty(P, dtype=torch.float32, device=device)
                self.x_outer_mom = torch.empty(P, dtype=torch.float32, device=device)
        ws = abi.mtdao_workspace_bytes(cfg)
        self.workspace = torch.empty(max(ws, 1), dtype=torch.uint8, device=device)
        bufs = abi.make_buffers(self.x.data_ptr(), [a.data_ptr() for a in self.u],
                                self.v.data_ptr() if self.v is not None else None, resume,
                                self.x_outer.data_ptr() if self.x_outer is not None else None,
                                self.x_outer_mom.data_ptr() if self.x_outer_mom is not None else None)
        self.handle = abi.mtdao_init(cfg, bufs, self.workspace.data_ptr(), self.workspace.numel(), _stream())

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
