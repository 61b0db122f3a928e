"""Seeded synthetic workloads shared by the oracle tests, the GPU tests and the bench.

This package only draws inputs (keys, values, window queries, decode queries and the
offline calibration basis). It holds none of the codec's arithmetic: salience,
allocation, projection and decode live in ``oracle/`` (CPU reference) and in the HIP
library, and neither of those imports the other.
"""
from .synth import (  # noqa: F401
    CONFIGS,
    LayerInputs,
    bf16_round,
    make_layer,
    make_head_model,
    rope_theta,
    joint_calibration_basis,
    calibration_basis,
    decode_queries,
    seed_for,
    splitmix64,
)
