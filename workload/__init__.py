"""Seeded synthetic workloads for the chunk-local update.

This package is shared by the oracle tests, the GPU parity tests and the
benchmark.  It holds shapes, seeded random draws and the next-token label
shift only -- none of the method's arithmetic (no norm, attention, head,
loss or optimizer code lives here).
"""
from .configs import CONFIGS, LORA_TARGETS, ChunkShape, base_specs, get_config, param_specs  # noqa: F401
from .gen import (  # noqa: F401
    bf16_round_trip_input,
    embed_tokens,
    init_params,
    labels_from_tokens,
    make_batch,
    uniform_tokens,
    zipf_tokens,
)
