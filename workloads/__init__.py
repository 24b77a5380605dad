"""Seeded synthetic inputs shared by the oracle, the tests and the benchmark.

This package holds no arithmetic of the rollout method itself: it only draws
model shapes, random weights, prompt token ids and forced response lengths.
Both the CPU oracle and the HIP path consume what it returns; neither of them
is imported here.
"""
from .gen import (  # noqa: F401
    ModelShape,
    RLBatch,
    SHAPES,
    Workload,
    WORKLOADS,
    make_rl_batch,
    make_weights,
    make_workload,
    tensor_names,
    truncated,
    weights_to_numpy,
)
