"""Seeded synthetic inputs for the FP8 speculative-verify path.

This package is shared by the CPU oracle's tests, the GPU parity tests and the
bench.  It only draws random numbers and lays them out (bf16 bit patterns,
int32 token ids, fp32 uniforms); it holds none of the method's arithmetic
(no E4M3 coding, no GEMM, no softmax, no acceptance rule).
"""

from .gen import (  # noqa: F401
    bf16_bits_from_f32,
    f32_from_bf16_bits,
    linear_activations,
    linear_weights,
    fp8_code_bytes,
    uniform_scales,
    student_t_activations,
    gated_ffn_input,
    accept_logits,
    draft_tokens_greedy,
    draft_tokens_sampled,
    philox_uniforms,
    tree_shape,
    tree_tokens_topk,
    paged_slot_mapping,
    calibration_sets,
)
from .configs import CONFIGS, C4_CORRELATION, TREE25  # noqa: F401
