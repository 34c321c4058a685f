"""Seeded synthetic inputs shared by the oracle tests, the GPU parity tests and
the benchmark.  Nothing in this package computes any part of the spectral-norm
method: it only draws random weights, start vectors and tokens with the shapes
of the models the paper evaluates (Table "Model architectures", App. G)."""

from .synth import (  # noqa: F401
    WORKLOADS,
    Workload,
    bf16_round,
    layer_master,
    layer_weights,
    all_weights,
    start_vectors,
    layer_start_vectors,
    perturb_master,
    tokens,
    device_tokens,
    planted_singular_values,
    seed_of,
)
