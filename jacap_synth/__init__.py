"""Seeded synthetic KV caches for the Jacap scoring path.

This module only draws random numbers and lays them out. It holds none of the
method's arithmetic, so both the GPU path and the CPU oracle can consume its
output without sharing any of the scoring code.

The distributions stand in for the Llama-3-8B / Llama3.1-8B-shaped caches the
paper evaluates on (Sec. 4, LongBench/NIAH); no dataset or model weights are
used. See ``WORKLOADS`` for the five shapes and the recipe.
"""

from .cases import (  # noqa: F401
    WORKLOADS,
    Case,
    make_case,
    unit_seed,
)
