"""Seeded synthetic attention-layer inputs (Q, K, V in bf16) for the CRISP path.

This package only draws random numbers and plants structure; it holds none of
CRISP's arithmetic (no softmax, no scores, no selection).  Both the HIP path and
the CPU oracle consume the tensors it returns.
"""
from .synth import (  # noqa: F401
    GEN_VERSION,
    LayerConfig,
    HeadSpec,
    CONFIGS,
    stress_config,
    make_layer,
    head_specs,
    kv_group_columns,
    custom_config,
    STRESS_ALPHAS,
    STRESS_BLOCKS,
    PE_SWEEP_LENGTHS,
    structured_pe_config,
)
