"""Seeded synthetic KV caches and queries shaped like the paper's workloads.

This module holds no codec arithmetic. It only draws inputs; both the CPU
oracle (in tests) and the HIP path consume them. See ``caches`` for the recipe.
"""
from .caches import (  # noqa: F401
    WORKLOADS, Workload, StreamSpec, stream_spec, numpy_stream, numpy_query,
    bf16_bits_to_f32, f32_to_bf16_bits, device_streams, device_queries, numpy_layer_stream, device_layer_stream,
)
from .calib import calibration_layers  # noqa: F401,E402
