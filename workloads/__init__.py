"""Seeded synthetic workloads shared by the GPU path and the CPU oracle.

This package only describes shapes and draws random inputs.  It holds none
of the method's arithmetic: no normalisation, projection, attention,
scoring, selection or slot mapping lives here.
"""

from .configs import CONFIGS, ModelDims, SeqLayout, Workload, get_config
from .gen import (
    LayerWeightsBits,
    bf16_bits_from_f32,
    draw_donor_rows,
    draw_embedding,
    draw_hidden_rows,
    draw_layer_qkv,
    draw_layer_weights,
    layer_norm_gains,
    draw_lm_head,
    draw_noise,
    draw_scores,
    draw_ints,
    draw_permutation,
    draw_tensor,
    draw_token_ids,
    rng_for,
)

__all__ = [
    "CONFIGS",
    "ModelDims",
    "SeqLayout",
    "Workload",
    "get_config",
    "draw_lm_head",
    "LayerWeightsBits",
    "bf16_bits_from_f32",
    "draw_donor_rows",
    "draw_embedding",
    "draw_hidden_rows",
    "draw_layer_qkv",
    "draw_layer_weights",
    "layer_norm_gains",
    "draw_noise",
    "draw_scores",
    "draw_ints",
    "draw_permutation",
    "draw_tensor",
    "draw_token_ids",
    "rng_for",
]
