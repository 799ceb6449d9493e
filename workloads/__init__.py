"""Workload definitions and seeded synthetic input generators.

This package holds no arithmetic of the Complementary Sparsity method: it only
describes the five layer configurations (shapes, complement factors, k-WTA
sizes, requantisation shifts, seeds) and draws their random inputs.  Both the
GPU path and the CPU oracle consume what it produces.
"""
from .configs import CONFIGS, Config, LayerSpec, get_config  # noqa: F401
from .generate import (  # noqa: F401
    block_complementary_weights,
    channel_complementary_weights,
    complementary_weights,
    generate,
    sparse_rows,
    tensor_digest,
)
