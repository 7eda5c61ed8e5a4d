"""Seeded synthetic Q/K/V generators shared by the tests, the bench and the smoke check.

This package holds no arithmetic of the attention method itself: it only draws
inputs. Both the CPU oracle and the GPU path are fed from here; neither side
imports the other.
"""
from .gen import (  # noqa: F401
    CONFIGS,
    bf16_round,
    keep_to_k,
    make_config,
    mixture_inputs,
    field_inputs,
)
