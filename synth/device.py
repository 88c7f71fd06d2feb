"""Device-side (torch) versions of the seeded input generators.

They produce, on the GPU, exactly the values ``synth.workloads`` produces on
the host for the same workload, step and worker: every gradient element is
one fp32 multiply sigma * pool[(i + off) mod POOL_SIZE] (then RNE to bf16
when the gradients are bf16), which torch and numpy both round exactly.
Input generation only: nothing here belongs to the optimizer.
"""

from __future__ import annotations

from typing import Dict, Optional

import numpy as np
import torch

from .workloads import POOL_SIZE, Workload, grad_offset, grad_pool, x_pool

_TORCH_DTYPE = {"f32": torch.float32, "bf16": torch.bfloat16}


class DeviceInputs:
    """Pools and per-element constants of one workload resident on a device."""

    def __init__(self, w: Workload, device: torch.device):
        self.w = w
        self.device = device
        self.pool = torch.from_numpy(grad_pool(w)).to(device)
        self.xpool = torch.from_numpy(x_pool(w)).to(device)
        sig = w.tensor_sigmas()
        self.uniform_sigma = bool(np.all(sig == sig[0]))
        self.sigma = torch.tensor(float(sig[0]), dtype=torch.float32, device=device)
        self.sig_elem: Optional[torch.Tensor] = None
        if not self.uniform_sigma:
            counts = torch.from_numpy(w.tensor_numels()).to(device)
            self.sig_elem = torch.repeat_interleave(torch.from_numpy(sig).to(device), counts)
        self._row: Optional[torch.Tensor] = None

    def _tile(self, src: torch.Tensor, out: torch.Tensor) -> None:
        """out[i] = src[i mod POOL_SIZE] for a 1-D out."""
        P = out.numel()
        for start in range(0, P, POOL_SIZE):
            n = min(POOL_SIZE, P - start)
            out[start:start + n].copy_(src[:n])

    def rotated(self, off: int, stream: int = 0) -> torch.Tensor:
        """rolled[j] = pool[(j + off) mod POOL_SIZE]."""
        return torch.roll(self.pool, -off)

    def grads_into(self, step: int, out: torch.Tensor) -> None:
        """Gradients of every worker at local step ``step`` into out [K][P]."""
        w = self.w
        K, P = out.shape
        f32_direct = out.dtype == torch.float32
        if not f32_direct and (self._row is None or self._row.numel() != P):
            self._row = torch.empty(P, dtype=torch.float32, device=self.device)
        for m in range(K):
            rolled = self.rotated(grad_offset(w.seed_g, m, step))
            row = out[m] if f32_direct else self._row
            if self.uniform_sigma:
                self._tile(rolled * self.sigma, row)
            else:
                self._tile(rolled, row)
                row.mul_(self.sig_elem)
            if not f32_direct:
                out[m].copy_(row)

    def pool_rows_into(self, stream: int, scale: float, out: torch.Tensor, absolute: bool = False) -> None:
        """Seeded per-worker fields (resume tests): scale * pool value."""
        w = self.w
        K, P = out.shape
        row = torch.empty(P, dtype=torch.float32, device=self.device)
        s = torch.tensor(scale, dtype=torch.float32, device=self.device)
        for m in range(K):
            rolled = self.rotated(grad_offset(w.seed_g, m, 0, stream=stream))
            if absolute:
                rolled = rolled.abs()
            self._tile(rolled * s, row)
            out[m].copy_(row)

    def x0_row(self) -> torch.Tensor:
        """x_0 of the workload as an fp32 (or bf16) device row."""
        w = self.w
        row = torch.empty(w.numel, dtype=torch.float32, device=self.device)
        self._tile(self.xpool * torch.tensor(w.x_std, dtype=torch.float32, device=self.device), row)
        offs = w.tensor_offsets()
        for t, spec in enumerate(w.tensors):
            if spec.kind == "norm":
                row[int(offs[t]):int(offs[t + 1])] = 1.0
        return row.to(_TORCH_DTYPE[w.param_dtype])
