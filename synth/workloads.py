"""Workload definitions and seeded input generators (host side, numpy).

Shapes follow the paper's GPT models (Appendix, Table 4 and the architecture
paragraph): Peri-LN blocks with four norm vectors each plus a final norm,
tied embedding, no biases, feed-forward width 4*d.  Parameters are
initialised N(0, sigma=0.02) for matrices and 1.0 for norm vectors
(Table 4 caption gives sigma=0.02).  The paper's data (SmolLM2) and trained
weights are not used; gradients are synthetic and seeded.

Reproducible gradients without storing terabytes: for every distribution a
pool of POOL_SIZE fp32 values is drawn once from a seeded numpy PCG64
generator, and the gradient of worker m at local step s, element i is

    g[m][s][i] = fp32( sigma(i) * pool[(i + off(m, s)) mod POOL_SIZE] )

with off(m, s) a fixed integer hash and sigma(i) one fp32 constant per tensor.
One exactly rounded fp32 multiply per element, so the host (numpy) and the
device (torch, see synth.device) produce bit-identical values.  bf16
gradients are the round-to-nearest-even bf16 of that fp32 value.

Nothing here updates moments, averages replicas or clips gradients.
"""

from __future__ import annotations

import dataclasses
import math
from dataclasses import dataclass
from typing import Dict, Optional, Sequence, Tuple

import numpy as np

# Largest prime below 2**24.  A non power of two keeps the pool's period from
# lining up with tensor, replica-row or tile boundaries.
POOL_SIZE = 16_777_213

_MASK64 = (1 << 64) - 1


@dataclass(frozen=True)
class TensorSpec:
    name: str
    numel: int
    kind: str  # "matrix" (N(0, x_std) init) or "norm" (init 1.0)


@dataclass(frozen=True)
class Workload:
    """One synthetic optimizer workload: hyper-parameters in the paper's
    notation (Algorithms 1-3 Require blocks) plus the tensor list and the
    gradient distribution.  ``replicas`` is the paper's number of workers M;
    ``period_*`` are the paper's K_x, K_j, K_v."""

    name: str
    replicas: int
    form: str                      # "adam" | "adopt" | "sgdm"
    beta1: Tuple[float, ...]
    omega: Tuple[float, ...]
    beta2: float
    eps: float
    lr: float
    clip_rho: float                # 0 disables the global-norm clip
    adopt_order: str               # "prev" | "cur"  (ADOPT only)
    adopt_clip: str                # "quarter_power" (c_t = t**0.25) | "off"
    period_x: int
    period_u: Tuple[int, ...]
    period_v: int
    steps: int
    param_dtype: str               # "f32" | "bf16"
    grad_dtype: str                # "f32" | "bf16"
    tensors: Tuple[TensorSpec, ...]
    grad_dist: str                 # "normal" | "student_t3"
    grad_std: float                # scalar sigma when no per-tensor scale
    grad_tensor_scale: Optional[Tuple[float, float]] = None  # U[lo, hi] per tensor
    x_std: float = 0.02
    seed_x: int = 0
    seed_g: int = 1000
    bias_correction: bool = True   # Adam: u_j/(1 - beta_j^s), v/(1 - beta_2^s)

    @property
    def n_moments(self) -> int:
        return len(self.beta1)

    @property
    def numel(self) -> int:
        return int(sum(t.numel for t in self.tensors))

    @property
    def has_v(self) -> bool:
        return self.form in ("adam", "adopt")

    def tensor_numels(self) -> np.ndarray:
        return np.array([t.numel for t in self.tensors], dtype=np.int64)

    def tensor_offsets(self) -> np.ndarray:
        n = self.tensor_numels()
        return np.concatenate([[0], np.cumsum(n)]).astype(np.int64)

    def tensor_sigmas(self) -> np.ndarray:
        """fp32 gradient scale per tensor (a constant, or U[lo, hi] per tensor)."""
        nt = len(self.tensors)
        if self.grad_tensor_scale is None:
            return np.full(nt, self.grad_std, dtype=np.float32)
        lo, hi = self.grad_tensor_scale
        rng = np.random.Generator(np.random.PCG64(self.seed_g + 7))
        return rng.uniform(lo, hi, size=nt).astype(np.float32)

    def adopt_clip_value(self, s: int) -> float:
        """Per-call clip c_t for ADOPT, t = number of moment updates applied
        including this one (s-1 with the previous-v order, s with the
        current-v order).  0 means off."""
        if self.form != "adopt" or self.adopt_clip == "off":
            return 0.0
        t = s - 1 if self.adopt_order == "prev" else s
        return float(np.float32(max(t, 0) ** 0.25)) if t > 0 else 0.0

    def replace(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


def _gpt_tensors(d: int, blocks: int, vocab: int, ffn_mult: int = 4) -> Tuple[TensorSpec, ...]:
    """Peri-LN GPT tensor list: tied embedding, per block QKV, out-proj,
    up, down, four norm vectors; final norm."""
    out = [TensorSpec("embed", vocab * d, "matrix")]
    f = ffn_mult * d
    for b in range(blocks):
        out += [
            TensorSpec(f"b{b}.qkv", d * 3 * d, "matrix"),
            TensorSpec(f"b{b}.out", d * d, "matrix"),
            TensorSpec(f"b{b}.up", d * f, "matrix"),
            TensorSpec(f"b{b}.down", f * d, "matrix"),
        ]
        out += [TensorSpec(f"b{b}.norm{k}", d, "norm") for k in range(4)]
    out.append(TensorSpec("final_norm", d, "norm"))
    return tuple(out)


WORKLOADS: Dict[str, Workload] = {}


def _register(w: Workload) -> Workload:
    WORKLOADS[w.name] = w
    return w


# K=2, one flat 1,048,576 tensor, Adam N=2.
ADAM_N2_K2_P1M = _register(Workload(
    name="adam_n2_k2_p1m", replicas=2, form="adam", beta1=(0.9, 0.99), omega=(0.5, 0.5),
    beta2=0.999, eps=1e-8, lr=1e-3, clip_rho=0.0, adopt_order="prev", adopt_clip="off",
    period_x=4, period_u=(8, 8), period_v=16, steps=32, param_dtype="f32", grad_dtype="f32",
    tensors=(TensorSpec("flat", 1_048_576, "matrix"),), grad_dist="normal", grad_std=1e-2,
    seed_g=1001))

# K=4, 16.8M small transformer (vocab 8192, d 512, 4 blocks), Adam N=3.
ADAM_N3_K4_P16M = _register(Workload(
    name="adam_n3_k4_p16m", replicas=4, form="adam", beta1=(0.9, 0.99, 0.999),
    omega=(0.3, 0.3, 0.3), beta2=0.999, eps=1e-8, lr=1e-3, clip_rho=0.0, adopt_order="prev",
    adopt_clip="off", period_x=32, period_u=(64, 64, 64), period_v=128, steps=256,
    param_dtype="f32", grad_dtype="f32", tensors=_gpt_tensors(512, 4, 8192),
    grad_dist="normal", grad_std=1e-2, seed_g=1002))

# K=8, 124M GPT (d 768, 12 blocks, vocab 50304), bf16 params and grads, ADOPT N=2.
ADOPT_N2_K8_P124M = _register(Workload(
    name="adopt_n2_k8_p124m_bf16", replicas=8, form="adopt", beta1=(0.9, 0.995),
    omega=(0.3, 0.6), beta2=0.9999, eps=1e-8, lr=2.0 ** -8, clip_rho=0.0, adopt_order="prev",
    adopt_clip="quarter_power", period_x=64, period_u=(64, 64), period_v=64, steps=128,
    param_dtype="bf16", grad_dtype="bf16", tensors=_gpt_tensors(768, 12, 50304),
    grad_dist="normal", grad_std=1.0, grad_tensor_scale=(1e-4, 1e-2), seed_g=1003))

# K=4, 1.31B GPT (d 2048, 24 blocks, ffn 8192, vocab 50304), fp32, Adam N=3.
ADAM_N3_K4_P1311M = _register(Workload(
    name="adam_n3_k4_p1311m", replicas=4, form="adam", beta1=(0.9, 0.99, 0.999),
    omega=(0.3, 0.3, 0.3), beta2=0.999, eps=1e-8, lr=1e-3, clip_rho=0.0, adopt_order="prev",
    adopt_clip="off", period_x=64, period_u=(128, 128, 128), period_v=256, steps=256,
    param_dtype="f32", grad_dtype="f32", tensors=_gpt_tensors(2048, 24, 50304),
    grad_dist="normal", grad_std=1e-3, seed_g=1004))

# K=16, 354M GPT (d 1024, 24 blocks, vocab 50304), fp32, SGDM N=2, global-norm clip 1.0.
SGDM_N2_K16_P354M = _register(Workload(
    name="sgdm_n2_k16_p354m_clip", replicas=16, form="sgdm", beta1=(0.9, 0.99),
    omega=(0.3, 0.6), beta2=0.0, eps=0.0, lr=1e-3, clip_rho=1.0, adopt_order="prev",
    adopt_clip="off", period_x=16, period_u=(32, 32), period_v=0, steps=64,
    param_dtype="f32", grad_dtype="f32", tensors=_gpt_tensors(1024, 24, 50304),
    grad_dist="student_t3", grad_std=1e-3, seed_g=1005))


def workload(name: str) -> Workload:
    return WORKLOADS[name]


def small_variant(w: Workload, target_numel: int, tail: int = 0, name: Optional[str] = None) -> Workload:
    """Same hyper-parameters and tensor structure, every tensor shrunk by one
    common factor so the total is about ``target_numel``; ``tail`` appends one
    more norm-kind tensor of that many elements (a ragged end)."""
    factor = max(1, math.ceil(w.numel / max(1, target_numel)))
    ts = [TensorSpec(t.name, max(1, t.numel // factor), t.kind) for t in w.tensors]
    if tail:
        ts.append(TensorSpec("tail", tail, "norm"))
    return w.replace(name=name or f"{w.name}_small{target_numel}", tensors=tuple(ts))


# ---------------------------------------------------------------------------
# pools and offsets


def _splitmix64(z: int) -> int:
    z = (z + 0x9E3779B97F4A7C15) & _MASK64
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & _MASK64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & _MASK64
    return z ^ (z >> 31)


def grad_offset(seed: int, replica: int, step: int, stream: int = 0) -> int:
    """Pool offset for (worker, local step); ``stream`` separates other
    seeded fields drawn from the same pool (initial moments)."""
    key = ((seed & 0xFFFFFFFF) << 32) ^ ((stream & 0xFF) << 56) ^ ((replica & 0xFFFF) << 20) ^ (step & 0xFFFFF)
    return _splitmix64(key) % POOL_SIZE


_POOL_CACHE: Dict[Tuple[str, int], np.ndarray] = {}


def _draw_pool(dist: str, seed: int) -> np.ndarray:
    key = (dist, seed)
    if key not in _POOL_CACHE:
        rng = np.random.Generator(np.random.PCG64(seed))
        if dist == "normal":
            p = rng.standard_normal(POOL_SIZE)
        elif dist == "student_t3":
            p = rng.standard_t(3.0, POOL_SIZE)
        else:
            raise ValueError(dist)
        _POOL_CACHE[key] = p.astype(np.float32)
    return _POOL_CACHE[key]


def grad_pool(w: Workload) -> np.ndarray:
    return _draw_pool(w.grad_dist, w.seed_g)


def x_pool(w: Workload) -> np.ndarray:
    return _draw_pool("normal", w.seed_x)


# ---------------------------------------------------------------------------
# bf16 bit conversions (storage format of inputs only)


def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round-to-nearest-even fp32 -> bf16, returned as uint16 bit patterns."""
    b = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    nan = (b & 0x7FFFFFFF) > 0x7F800000
    r = (b + np.uint32(0x7FFF) + ((b >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    r = np.where(nan, (b >> np.uint32(16)) | np.uint32(0x40), r)
    return r.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


# ---------------------------------------------------------------------------
# host-side rows for a set of element indices


def element_sigmas(w: Workload, idx: np.ndarray) -> np.ndarray:
    """fp32 gradient sigma for each element index."""
    sig = w.tensor_sigmas()
    t = np.searchsorted(w.tensor_offsets(), idx, side="right") - 1
    return sig[t]


def element_is_norm(w: Workload, idx: np.ndarray) -> np.ndarray:
    kinds = np.array([t.kind == "norm" for t in w.tensors])
    t = np.searchsorted(w.tensor_offsets(), idx, side="right") - 1
    return kinds[t]


def host_grad_rows(w: Workload, step: int, idx: Optional[np.ndarray] = None) -> np.ndarray:
    """Gradients of every worker at local step ``step`` (1-based) for element
    indices ``idx`` (all elements if None): float32 [K][n], or uint16 bf16
    bit patterns when the workload's gradients are bf16."""
    if idx is None:
        idx = np.arange(w.numel, dtype=np.int64)
    pool = grad_pool(w)
    sig = element_sigmas(w, idx)
    rows = np.empty((w.replicas, idx.size), dtype=np.float32)
    for m in range(w.replicas):
        off = grad_offset(w.seed_g, m, step)
        rows[m] = sig * pool[(idx + off) % POOL_SIZE]
    if w.grad_dtype == "bf16":
        return f32_to_bf16_bits(rows)
    return rows


def _rotated_into(pool: np.ndarray, start: int, out: np.ndarray) -> None:
    """out[k] = pool[(start + k) mod POOL_SIZE], copied as contiguous runs."""
    n, pos, j = out.size, 0, start % POOL_SIZE
    while pos < n:
        take = min(n - pos, POOL_SIZE - j)
        out[pos:pos + take] = pool[j:j + take]
        pos += take
        j = 0


def host_grad_range(w: Workload, step: int, lo: int, hi: int) -> np.ndarray:
    """host_grad_rows(w, step, arange(lo, hi)), built from contiguous runs of
    the pool and one fp32 multiply per tensor segment (the same exactly
    rounded products), for long contiguous element ranges."""
    n = hi - lo
    pool = grad_pool(w)
    sig = w.tensor_sigmas()
    offs = w.tensor_offsets()
    first = int(np.searchsorted(offs, lo, side="right")) - 1
    segs = []
    t = max(first, 0)
    while t < len(w.tensors) and offs[t] < hi:
        a, b = max(int(offs[t]), lo), min(int(offs[t + 1]), hi)
        if b > a:
            segs.append((a - lo, b - lo, sig[t]))
        t += 1
    rows = np.empty((w.replicas, n), dtype=np.float32)
    for m in range(w.replicas):
        _rotated_into(pool, lo + grad_offset(w.seed_g, m, step), rows[m])
        for a, b, sg in segs:
            np.multiply(rows[m, a:b], sg, out=rows[m, a:b])
    if w.grad_dtype == "bf16":
        return f32_to_bf16_bits(rows)
    return rows


def host_pool_rows(w: Workload, stream: int, scale: float, idx: np.ndarray, absolute: bool = False,
                   dtype: str = "f32") -> np.ndarray:
    """Seeded per-worker fields for resume tests (initial moments or
    per-worker parameters): scale * pool value, fp32 [K][n]."""
    pool = grad_pool(w)
    rows = np.empty((w.replicas, idx.size), dtype=np.float32)
    for m in range(w.replicas):
        off = grad_offset(w.seed_g, m, 0, stream=stream)
        vals = pool[(idx + off) % POOL_SIZE]
        if absolute:
            vals = np.abs(vals)
        rows[m] = np.float32(scale) * vals
    if dtype == "bf16":
        return f32_to_bf16_bits(rows)
    return rows


def host_x0_row(w: Workload, idx: Optional[np.ndarray] = None) -> np.ndarray:
    """Initial parameters x_0 (one row, shared by all workers): 1.0 for norm
    vectors, fp32(x_std * z) for matrices.  float32, or uint16 bf16 bits."""
    if idx is None:
        idx = np.arange(w.numel, dtype=np.int64)
    z = x_pool(w)[idx % POOL_SIZE]
    row = np.float32(w.x_std) * z
    row = np.where(element_is_norm(w, idx), np.float32(1.0), row).astype(np.float32)
    if w.param_dtype == "bf16":
        return f32_to_bf16_bits(row)
    return row


def sample_indices(w: Workload, n_stride: int = 1 << 20, edge: int = 64) -> np.ndarray:
    """Deterministic element subsample: the first and last ``edge`` elements
    of every tensor, ``n_stride`` evenly strided elements (strided_mask marks
    them: an unbiased subset), the last element overall, and ``edge``
    columns on either side of every column where a flat element index
    m P + i or a flat byte offset of an fp32 or bf16 buffer reaches 2^31,
    2^32 or 2^33 (where 32-bit index arithmetic would wrap).  Sorted and
    unique (int64)."""
    offs = w.tensor_offsets()
    parts = []
    for a, b in zip(offs[:-1], offs[1:]):
        parts.append(np.arange(a, min(b, a + edge)))
        parts.append(np.arange(max(a, b - edge), b))
    P = w.numel
    stride = max(1, P // max(1, n_stride))
    parts.append(np.arange(0, P, stride, dtype=np.int64)[:n_stride])
    parts.append(np.array([P - 1]))
    for flat in sorted({1 << k for k in (29, 30, 31, 32, 33)}):
        for m in range(w.replicas):
            c = flat - m * P
            if 0 <= c < P:
                parts.append(np.arange(max(0, c - edge), min(P, c + edge)))
    return np.unique(np.concatenate(parts).astype(np.int64))


def strided_mask(w: Workload, idx: np.ndarray, n_stride: int = 1 << 20) -> np.ndarray:
    """Which entries of a sample_indices(w, n_stride) sample are its evenly
    strided elements: a subset whose statistics (an rms) are those of the
    whole row, unlike the tensor edges, where the short norm vectors are
    over-represented."""
    stride = max(1, w.numel // max(1, n_stride))
    return (idx % stride == 0) & (idx // stride < n_stride)


def bernoulli_masks(seed: int, steps: int, n_moments: int, p_x: float, p_u: Sequence[float],
                    p_v: float = 0.0, has_v: bool = False) -> list:
    """Seeded averaging events of the probabilistic variant (Algorithm 4):
    after every step each state is averaged with its own probability,
    independently, the same event for all workers.  Returns one mask per
    step (bit 0 = x, bit j = u^j, bit N+1 = v)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    probs = [p_x] + list(p_u) + ([p_v] if has_v else [])
    out = []
    for _ in range(steps):
        draws = rng.random(len(probs))
        out.append(int(sum(1 << b for b, (d, p) in enumerate(zip(draws, probs)) if d < p)))
    return out
