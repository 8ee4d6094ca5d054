"""Seeded synthetic inputs shared by the oracle's tests, the GPU tests and the benchmark."""

from .gen import (
    BF16,
    CONFIGS,
    F32,
    FP8,
    LayerInputs,
    LayerSpec,
    TraceStep,
    agentic_trace,
    bf16_bits_to_f32,
    f32_to_bf16_bits,
    logits_of,
    make_config,
    make_layer,
    seed_of,
    tie_logits,
)

__all__ = [
    "BF16",
    "CONFIGS",
    "F32",
    "FP8",
    "LayerInputs",
    "LayerSpec",
    "TraceStep",
    "agentic_trace",
    "bf16_bits_to_f32",
    "f32_to_bf16_bits",
    "logits_of",
    "make_config",
    "make_layer",
    "seed_of",
    "tie_logits",
]
