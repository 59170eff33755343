"""Seeded synthetic inputs for the routed threshold-sparsified gated MLP.

This package only draws random numbers and lays them out in the storage
formats the library consumes (bf16 bit patterns or float32).  It contains none
of the method's arithmetic: no projection, activation, mask or routing rule.
Both the CPU oracle and the GPU path take their inputs from here.
"""
from .configs import CONFIGS, Config, get_config  # noqa: F401
from . import synth  # noqa: F401
