"""Seeded synthetic workloads: sprite frame sequences, occlusion boxes and weights.

This package holds input generation only. It computes none of the method's
arithmetic (no diff, dilation, convolution or head), so the CPU oracle and the
GPU path can both consume its bytes without sharing any of the method's code.
"""
from .frames import (  # noqa: F401
    WORKLOADS,
    Workload,
    sprite_sequence,
    sprite_batch,
    full_change_sequence,
    occlusion_base,
    occlusion_variant_frame,
    occlusion_boxes,
    stacked_view,
    net_weights,
    to_f32,
)
