"""Seeded synthetic workloads shared by the oracle tests, the GPU tests and the benchmark.

This package draws random inputs and nothing else: it holds none of the attention
method's arithmetic (no tree, no softmax, no pooling, no top-k).
"""
from .gen import CONFIGS, Config, HeadInputs, make_inputs, make_block_inputs, make_points, round_bf16  # noqa: F401
