"""Seeded synthetic inputs for the tree-verify path.

This package only draws random numbers and lays them out in the cache format
that both the CPU oracle and the GPU library consume.  It holds none of the
method's arithmetic (no masks, compression, scoring or attention).
"""
from .inputs import (  # noqa: F401
    CONFIGS,
    VOCAB,
    Selection,
    make_selection,
    Workload,
    make_workload,
    config_dims,
)
