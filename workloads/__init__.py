"""Seeded synthetic inputs shaped like VGGT global-attention layers.

This package draws Q/K/V and per-head pattern tables. It holds none of the
method's arithmetic (no pooling, scoring, selection or attention), so both the
oracle and the GPU path can consume its outputs without sharing code.
"""
from .gen import (  # noqa: F401
    DENSE,
    FRAME_LOCAL,
    TOPK,
    WORKLOADS,
    Workload,
    bf16_bits_from_f32,
    bf16_bits_to_f32,
    dense_table,
    layer_tau,
    make_layer,
    make_qkv,
    make_table,
    num_blocks,
)
