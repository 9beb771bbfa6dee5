"""Seeded synthetic inputs for the PreLRShared hot path.

This package only draws random numbers and fixes shapes, positions and
lengths.  It holds none of the method's arithmetic, so the oracle side and the
GPU side can both take their inputs from it without sharing any computation.
"""
from .configs import CONFIGS, Config  # noqa: F401
from .gen import (  # noqa: F401
    normal_bf16,
    lora_case,
    attention_case,
    precompute_case,
    seed_for,
)
