"""Seeded synthetic workloads for the fused RL log-prob path.

This package draws random inputs and packs them; it holds none of the
method's arithmetic (no log-softmax, log-sum-exp, ratio, sequence
statistic, advantage or loss).  Both the oracle-side tests and the GPU
path consume what it produces.
"""
from .gen import (  # noqa: F401
    CONFIGS,
    Structure,
    bf16_bits_to_f32,
    f32_to_bf16_bits,
    make_structure,
    make_tensors_numpy,
    make_tensors_torch,
    sample_targets_numpy,
    sample_targets_torch,
    scaled_config,
    zipf_targets,
)
