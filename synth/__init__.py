"""Seeded synthetic workloads for bucket-level gradient-conflict resolution.

This package only *draws inputs*: model-shaped parameter lists, fixed-size
bucket cuts, per-bucket target correlations between the K per-language
gradients, the per-(bucket, task) PCGrad visiting orders, and the gradient
vectors themselves.  It holds none of the method's arithmetic (no inner
products, no solver, no weighted sum), so both the HIP path's tests and the
float64 oracle can consume its output without sharing any code with each
other.
"""

from .workloads import (  # noqa: F401
    WORKLOADS,
    Workload,
    bucket_correlations,
    fill_grads,
    fixed_bucket_offsets,
    gpt2_small_tensors,
    host_rows,
    llama_tensors,
    pcgrad_orders,
    per_task_scales,
    small_workload,
)
