"""Seeded synthetic FluxBin layers (shared by the tests, the oracle's callers and the benchmark).

This package only draws random inputs of the right shapes and distributions. It holds none of the method's
arithmetic: no reconstruction, no lookup tables, no scale application.
"""
from .layers import (  # noqa: F401
    LayerSpec,
    SyntheticLayer,
    CONFIGS,
    config_layers,
    make_layer,
    make_activations,
    salient_count,
    kernel_variant_layers,
    fused_decoder_layers,
    shard_layers,
    make_weight_matrix,
    vcm_off_equivalent,
    paper_config,
    kernel_latency_layers,
)
