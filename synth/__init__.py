"""Seeded synthetic workloads (shapes, prompts, weights) shared by the oracle and the HIP path.

Holds none of the forward pass's arithmetic.
"""
from .configs import CONFIGS, TEST_CONFIGS, ModelConfig, get_config  # noqa: F401
from . import gen  # noqa: F401
