"""Seeded synthetic inputs shared by the oracle, the tests and the benchmark.

This package describes workloads (model shapes, tree sizes, prompt lengths)
and draws their inputs: random-init weights and uniform-random prompt tokens.
It holds none of the method's arithmetic, so both the CPU oracle and the GPU
path can take their inputs from it without sharing any computation.
"""
from .configs import CloverConfig, CONFIGS, SWEEP_CONTEXTS, SWEEP_TREES, get_config, tiny_test_config  # noqa: F401
from .weights import weight_specs, make_weights, is_matrix  # noqa: F401
from .prompts import make_prompt, make_prompt_lengths  # noqa: F401
