"""Seeded synthetic SpMM workloads (inputs only).

This package draws W, its keep-mask and X for the layer shapes of Section 5
(decode-phase SpMM, M/K/N notation of Section 5.1). It holds none of the
method's arithmetic: no encoding, no product. Both the oracle tests and the
GPU tests take their inputs from here.
"""
from .gen import (  # noqa: F401
    BLOCKS,
    CONFIGS,
    SHARDS,
    Instance,
    draw_weights,
    instance_list,
    keep_count,
    layer_config,
    make_block,
    make_instance,
    make_mask,
    make_random,
    make_small_int,
    make_x,
    prune_global,
    prune_per_row,
    seed_for,
)
