"""Seeded synthetic inputs shared by the oracle tests, the GPU tests and the benchmark.

This package only draws random numbers and stores them in the formats the
library consumes (fp32 activations, bf16 weights as raw 16-bit patterns,
int32 token ids). It contains none of the method's arithmetic: no gate,
activation, threshold, softmax or selection is computed here.
"""

from .inputs import (  # noqa: F401
    bf16_bits,
    ffn_weights,
    decode_inputs,
    calibration_inputs,
    griffin_prompt,
    verify_inputs,
    tree_build_inputs,
    tree_verify_inputs,
    attn_inputs,
    model_weights,
    prompt_tokens,
    ModelShape,
    TINY_MODEL,
    TINY,
    LLAMA3_8B,
    LLAMA3_70B,
    VERIFY_TINY,
    VERIFY_8B,
)
