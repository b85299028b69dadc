"""Seeded synthetic inputs shaped like the prefill workloads of the residual workload predictor.

This package generates inputs only: random draws, their rounding to bfloat16 storage, and placement
tables. It holds none of the predictor's or the planner's arithmetic. The GPU path and the CPU
checker both consume the exact bytes produced here.
"""
from .synth import (  # noqa: F401
    CONFIGS,
    SEED_ROOT,
    LayerInputs,
    Workload,
    bf16_bits_from_f32,
    contiguous_placement,
    make_layer,
    random_replicated_placement,
    replicated_placement,
    rng,
    sweep_workload,
    truncated_zipf_probs,
)
