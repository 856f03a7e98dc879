"""Seeded synthetic workloads for tree-packed linear attention.

This package only draws random forests and random tensors; it holds none of
the method's arithmetic, so both the oracle (``oracle/``) and the HIP path
(``paper_2608_28158_amd``) can be fed from it without sharing any code.
"""
from .trees import (  # noqa: F401
    Forest,
    figure1_forest,
    spine_forest,
    agentic_forest,
    forest_for_config,
    CONFIGS,
    trajectory_tokens,
)
from .tensors import config_inputs, draw_inputs, to_bf16_roundtrip  # noqa: F401
