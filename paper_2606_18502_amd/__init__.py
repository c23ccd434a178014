"""FP8 speculative-decoding verify path for AMD Instinct MI355X (gfx950).

The hot path of the inference-optimization stage of arxiv 2606.18502: the
target model's verification step of speculative decoding run in FP8 E4M3
W8A8 -- dynamic per-token activation quantization, per-output-channel weight
scales, an fp32-accumulated FP8-MFMA GEMM with a scale epilogue -- followed by
greedy or speculative-sampling acceptance of the drafted tokens.

Beside the chain verify step it offers the LM-head GEMM with the acceptance
statistics in its epilogue (gemm_logit_stats, then verify_accept with
target_stats), the gate|up GEMM with the SiLU gate in its epilogue
(gemm_silu_mul), token-tree verification (verify_accept_tree) with its
attention masks (tree_attention_mask), and the
FP8 KV-cache write of the new tokens' keys and values (kv_cache_write).

The computation lives in libspecfp8.so (HIP kernels behind the C ABI of
include/spec_fp8.h); this package only marshals torch tensors into that ABI.

A verify step, in outline (tensors on the GPU; shapes as in the docstrings):

    import paper_2606_18502_amd as p
    w_q, w_s = p.quantize(w_bf16)                 # once per weight: per-channel E4M3
    a_q, a_s = p.quantize(x_bf16)                 # per token, at run time
    y = p.gemm(a_q, a_s, w_q, w_s)                # bf16 [M, N], fp32 accumulation
    h_q, h_s = p.quantize(y_gate_up, silu_mul=True)   # SiLU-gated input of the down projection
    out, num = p.verify_accept(target_logits, draft_logits, draft_tokens, uniforms, 0.7)

`out[b, :num[b] + 1]` are the tokens sequence b emits (accepted drafts, then
the resampled or bonus token).  Static per-tensor scales: p.calibrate over
calibration batches, then p.quantize(x, per_tensor_scale=s).
"""

from ._lib import SpecError, load as load_library, LIB_PATH  # noqa: F401
from .ops import (  # noqa: F401
    quantize,
    calibrate,
    clip_count,
    silu_mul,
    kv_cache_write,
    gemm,
    gemm_workspace_bytes,
    gemm_logit_stats,
    gemm_silu_mul,
    logit_stats_count,
    verify_accept,
    verify_accept_noalloc,
    accept_workspace_bytes,
    verify_accept_tree,
    tree_attention_mask,
    accept_tree_workspace_bytes,
)

__version__ = "0.1.0"
