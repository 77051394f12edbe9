"""Seeded synthetic inputs for the suffix-prefill path.

This package only draws inputs: random numbers, their rounding to bfloat16
storage, artifact lengths and request compositions.  It holds none of the
method's arithmetic (no projection, normalisation, rotation or attention), so
both the fp64 oracle and the HIP path can take their inputs from it.
"""

from .bf16 import f32_to_bf16_bits, bf16_bits_to_f32
from .workloads import (
    ModelShape,
    Request,
    Workload,
    WORKLOADS,
    make_workload,
    custom_workload,
    layer_weights,
    artifact_kv,
    suffix_hidden,
    prefill_hidden,
    decoder_weights,
    lm_weights,
    suffix_tokens,
)

__all__ = [
    "f32_to_bf16_bits",
    "bf16_bits_to_f32",
    "ModelShape",
    "Request",
    "Workload",
    "WORKLOADS",
    "make_workload",
    "custom_workload",
    "layer_weights",
    "artifact_kv",
    "suffix_hidden",
    "prefill_hidden",
    "decoder_weights",
    "lm_weights",
    "suffix_tokens",
]
