"""Seeded synthetic inputs for the verify path (shared by the oracle tests,
the HIP parity tests, smoke() and bench.py).

This package only draws and lays out inputs in the library's documented
formats; it computes none of the method's arithmetic (no attention, no
argmax).  Expected acceptance results it returns are known by construction
(the planted scheme), not computed.
"""
from .gen import (  # noqa: F401
    BF16_NAN,
    BLOCK_WIDTH,
    PAGE_SIZE,
    SEED_BASE,
    AcceptInputs,
    AttnInputs,
    bf16_bits,
    bf16_to_f32,
    config_accept_inputs,
    config_attn_inputs,
    config_rng,
    cu_from_lengths,
    k_tile_offset,
    make_accept_inputs,
    make_attn_inputs,
    repack,
    v_tile_offset,
    verify_lengths,
    CONFIGS,
    StressPlan,
    StressStep,
    DvlInputs,
    make_dvl_inputs,
    plant_boosts,
    PREDICTOR_DIMS,
    PredictorInputs,
    make_predictor_inputs,
)
