"""Seeded synthetic workloads for the MT-DAO optimizer hot path.

This package only generates inputs: tensor lists shaped like the paper's
GPT models, hyper-parameter sets, initial parameters and per-worker
gradients.  It holds none of the method's arithmetic (no moment updates, no
averaging, no clipping), so both the CPU oracle's tests and the GPU path's
tests and benchmark can draw identical inputs from it.
"""

from .workloads import (  # noqa: F401
    POOL_SIZE,
    Workload,
    TensorSpec,
    WORKLOADS,
    workload,
    small_variant,
    grad_offset,
    grad_pool,
    x_pool,
    host_grad_rows,
    host_grad_range,
    host_pool_rows,
    host_x0_row,
    f32_to_bf16_bits,
    bf16_bits_to_f32,
    sample_indices,
    strided_mask,
    bernoulli_masks,
)
