"""Torch-facing wrappers of the C ABI.

Argument marshalling only: every step of the verify path runs in the HIP
kernels of libspecfp8.so; torch provides device memory and the current stream.
There is no CPU or torch fallback: without the built library every call raises.
"""

from __future__ import annotations

from typing import Optional, Tuple

import torch

from . import _lib
from ._lib import check


def _stream() -> int:
    return torch.cuda.current_stream().cuda_stream


def _dev(t: torch.Tensor, dtype: torch.dtype, name: str) -> None:
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise ValueError(f"{name} must be a CUDA (HIP) tensor")
    if t.dtype != dtype:
        raise ValueError(f"{name} must have dtype {dtype}, got {t.dtype}")


def _rowmajor(t: torch.Tensor, name: str) -> int:
    """Leading dimension of a 2-D row-major view (unit stride in the last dim)."""
    if t.dim() != 2 or (t.shape[1] > 1 and t.stride(1) != 1):
        raise ValueError(f"{name} must be a 2-D row-major view")
    return t.stride(0) if t.shape[0] > 1 else max(t.shape[1], t.stride(0))


def quantize(x: torch.Tensor, per_tensor_scale: Optional[torch.Tensor] = None, silu_mul: bool = False,
             out: Optional[torch.Tensor] = None, scales: Optional[torch.Tensor] = None
             ) -> Tuple[torch.Tensor, torch.Tensor]:
    """E4M3 row quantization of bf16 rows (spec_fp8_quantize).

    x: bf16 [rows, cols] (or [rows, 2*cols] with silu_mul).  Dynamic per-row
    scales unless `per_tensor_scale` (fp32 [1]) is given.
    Returns (codes uint8 [rows, cols], scales fp32 [rows] or the given [1]).
    """
    lib = _lib.load()
    _dev(x, torch.bfloat16, "x")
    rows = x.shape[0]
    cols = x.shape[1] // 2 if silu_mul else x.shape[1]
    ld_x = _rowmajor(x, "x")
    if out is None:
        out = torch.empty((rows, cols), dtype=torch.uint8, device=x.device)
    _dev(out, torch.uint8, "out")
    ld_q = _rowmajor(out, "out")
    if per_tensor_scale is not None:
        _dev(per_tensor_scale, torch.float32, "per_tensor_scale")
        scales = per_tensor_scale
        mode = _lib.SCALE_PER_TENSOR
    else:
        if scales is None:
            scales = torch.empty((rows,), dtype=torch.float32, device=x.device)
        _dev(scales, torch.float32, "scales")
        mode = _lib.SCALE_PER_ROW
    kind = _lib.QIN_SILU_MUL_BF16 if silu_mul else _lib.QIN_BF16
    check("spec_fp8_quantize", lib.spec_fp8_quantize(x.data_ptr(), rows, cols, ld_x, kind, mode,
                                                     scales.data_ptr(), out.data_ptr(), ld_q, _stream()))
    return out, scales


def calibrate(x: torch.Tensor, running_scale: torch.Tensor, silu_mul: bool = False) -> torch.Tensor:
    """Static min-max calibration step (spec_fp8_quantize, SPEC_SCALE_CALIBRATE).

    running_scale: fp32 [1], updated in place to max(running_scale, scale of
    the largest |x|); start it at 0 and pass every calibration batch.
    """
    lib = _lib.load()
    _dev(x, torch.bfloat16, "x")
    _dev(running_scale, torch.float32, "running_scale")
    if running_scale.numel() != 1:
        raise ValueError("running_scale must hold one fp32 value")
    rows = x.shape[0]
    cols = x.shape[1] // 2 if silu_mul else x.shape[1]
    kind = _lib.QIN_SILU_MUL_BF16 if silu_mul else _lib.QIN_BF16
    check("spec_fp8_quantize", lib.spec_fp8_quantize(x.data_ptr(), rows, cols, _rowmajor(x, "x"), kind,
                                                     _lib.SCALE_CALIBRATE, running_scale.data_ptr(), None, 0,
                                                     _stream()))
    return running_scale


def silu_mul(x: torch.Tensor, out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """h = bf16(silu(gate) * up) for x = [gate | up] bf16 [rows, 2*cols] (spec_silu_mul_bf16)."""
    lib = _lib.load()
    _dev(x, torch.bfloat16, "x")
    rows, cols = x.shape[0], x.shape[1] // 2
    if out is None:
        out = torch.empty((rows, cols), dtype=torch.bfloat16, device=x.device)
    _dev(out, torch.bfloat16, "out")
    check("spec_silu_mul_bf16", lib.spec_silu_mul_bf16(x.data_ptr(), rows, cols, _rowmajor(x, "x"),
                                                       out.data_ptr(), _rowmajor(out, "out"), _stream()))
    return out


def clip_count(x: torch.Tensor, scale: torch.Tensor, count: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Values of bf16 rows x that the static per-tensor scale clips (spec_fp8_clip_count):
    |fl32(x * fl32(1/scale))| > 448.  Accumulates into `count` (int64 [1]
    holding the uint64 count; a new zeroed counter if None) and returns it."""
    lib = _lib.load()
    _dev(x, torch.bfloat16, "x")
    _dev(scale, torch.float32, "scale")
    if scale.numel() != 1:
        raise ValueError("scale must hold one fp32 value")
    if count is None:
        count = torch.zeros(1, dtype=torch.int64, device=x.device)
    _dev(count, torch.int64, "count")
    rows, cols = x.shape
    check("spec_fp8_clip_count", lib.spec_fp8_clip_count(x.data_ptr(), rows, cols, _rowmajor(x, "x"),
                                                         scale.data_ptr(), count.data_ptr(), _stream()))
    return count


def kv_cache_write(k: torch.Tensor, v: torch.Tensor, slot_mapping: torch.Tensor, k_cache: torch.Tensor,
                   v_cache: torch.Tensor, k_scale: torch.Tensor, v_scale: torch.Tensor,
                   per_tensor: bool = False) -> None:
    """Quantize new keys and values to E4M3 into the FP8 KV cache (spec_fp8_kv_cache_write).

    k, v: bf16 [T, H, D] views (unit stride over D and heads packed side by
    side, e.g. column blocks of the QKV output viewed as [T, H, D]);
    slot_mapping: int64 [T] (negative = skip); k_cache, v_cache: uint8
    [num_slots, H, D] contiguous (a paged [blocks, block_size, H, D] cache
    viewed flat).  Per-row scales: k_scale, v_scale fp32 [num_slots, H],
    written at the stored slots; per_tensor=True: fp32 [1], read.
    """
    lib = _lib.load()
    _dev(k, torch.bfloat16, "k")
    _dev(v, torch.bfloat16, "v")
    _dev(slot_mapping, torch.int64, "slot_mapping")
    _dev(k_cache, torch.uint8, "k_cache")
    _dev(v_cache, torch.uint8, "v_cache")
    _dev(k_scale, torch.float32, "k_scale")
    _dev(v_scale, torch.float32, "v_scale")
    if k.dim() != 3 or v.shape != k.shape:
        raise ValueError("k and v must be [T, H, D] of the same shape")
    T, H, D = k.shape
    for name, t in (("k", k), ("v", v)):
        if (D > 1 and t.stride(2) != 1) or (H > 1 and t.stride(1) != D):
            raise ValueError(f"{name} must have unit stride over D and heads packed side by side")
    if k_cache.dim() != 3 or k_cache.shape[1:] != (H, D) or v_cache.shape != k_cache.shape \
            or not k_cache.is_contiguous() or not v_cache.is_contiguous():
        raise ValueError("k_cache and v_cache must be contiguous [num_slots, H, D]")
    if slot_mapping.shape != (T,) or not slot_mapping.is_contiguous():
        raise ValueError("slot_mapping must be a contiguous int64 [T]")
    num_slots = k_cache.shape[0]
    if per_tensor:
        if k_scale.numel() != 1 or v_scale.numel() != 1:
            raise ValueError("per-tensor scales hold one fp32 value each")
        mode = _lib.SCALE_PER_TENSOR
    else:
        if k_scale.shape != (num_slots, H) or v_scale.shape != (num_slots, H) \
                or not k_scale.is_contiguous() or not v_scale.is_contiguous():
            raise ValueError("per-row scales must be contiguous fp32 [num_slots, H]")
        mode = _lib.SCALE_PER_ROW
    ld_k = k.stride(0) if T > 1 else H * D
    ld_v = v.stride(0) if T > 1 else H * D
    check("spec_fp8_kv_cache_write",
          lib.spec_fp8_kv_cache_write(k.data_ptr(), ld_k, v.data_ptr(), ld_v, slot_mapping.data_ptr(), T, H, D,
                                      num_slots, mode, k_scale.data_ptr(), v_scale.data_ptr(),
                                      k_cache.data_ptr(), v_cache.data_ptr(), _stream()))


def gemm_workspace_bytes(M: int, N: int, K: int) -> int:
    return int(_lib.load().spec_fp8_gemm_workspace_bytes(M, N, K))


def gemm(a: torch.Tensor, sa: torch.Tensor, w: torch.Tensor, sw: torch.Tensor,
         out_dtype: torch.dtype = torch.bfloat16, out: Optional[torch.Tensor] = None,
         workspace: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Y = dec(A) dec(W)^T * sa * sw (spec_fp8_gemm).

    a: uint8 E4M3 [M,K]; sa: fp32 [M] (per token) or [1] (per tensor);
    w: uint8 E4M3 [N,K]; sw: fp32 [N] (per channel) or [1].
    """
    lib = _lib.load()
    _dev(a, torch.uint8, "a")
    _dev(w, torch.uint8, "w")
    _dev(sa, torch.float32, "sa")
    _dev(sw, torch.float32, "sw")
    M, K = a.shape
    N = w.shape[0]
    if w.shape[1] != K:
        raise ValueError("a and w disagree on K")
    a_mode = _lib.SCALE_PER_TENSOR if sa.numel() == 1 and M != 1 else _lib.SCALE_PER_ROW
    w_mode = _lib.SCALE_PER_TENSOR if sw.numel() == 1 and N != 1 else _lib.SCALE_PER_ROW
    if a_mode == _lib.SCALE_PER_ROW and sa.numel() < M:
        raise ValueError("sa must hold M per-row scales or one per-tensor scale")
    if w_mode == _lib.SCALE_PER_ROW and sw.numel() < N:
        raise ValueError("sw must hold N per-channel scales or one per-tensor scale")
    if out is None:
        # the ABI wants a row stride that is a multiple of 8 elements
        ld = (N + 7) // 8 * 8
        out = torch.empty((M, ld), dtype=out_dtype, device=a.device)[:, :N]
    if out.dtype not in (torch.bfloat16, torch.float32):
        raise ValueError("out must be bf16 or fp32")
    _dev(out, out.dtype, "out")
    odt = _lib.OUT_F32 if out.dtype == torch.float32 else _lib.OUT_BF16
    need = gemm_workspace_bytes(M, N, K)
    ws_ptr, ws_bytes = None, 0
    if need:
        if workspace is None or workspace.numel() * workspace.element_size() < need:
            workspace = torch.zeros((need,), dtype=torch.uint8, device=a.device)   # tickets start at zero
        ws_ptr, ws_bytes = workspace.data_ptr(), workspace.numel() * workspace.element_size()
    check("spec_fp8_gemm", lib.spec_fp8_gemm(a.data_ptr(), _rowmajor(a, "a"), sa.data_ptr(), a_mode,
                                             w.data_ptr(), _rowmajor(w, "w"), sw.data_ptr(), w_mode, M, N, K,
                                             out.data_ptr(), _rowmajor(out, "out"), odt, ws_ptr, ws_bytes,
                                             _stream()))
    return out


def _scale_modes(a, sa, w, sw):
    M, N = a.shape[0], w.shape[0]
    a_mode = _lib.SCALE_PER_TENSOR if sa.numel() == 1 and M != 1 else _lib.SCALE_PER_ROW
    w_mode = _lib.SCALE_PER_TENSOR if sw.numel() == 1 and N != 1 else _lib.SCALE_PER_ROW
    if a_mode == _lib.SCALE_PER_ROW and sa.numel() < M:
        raise ValueError("sa must hold M per-row scales or one per-tensor scale")
    if w_mode == _lib.SCALE_PER_ROW and sw.numel() < N:
        raise ValueError("sw must hold N per-channel scales or one per-tensor scale")
    return a_mode, w_mode


def gemm_silu_mul(a: torch.Tensor, sa: torch.Tensor, w: torch.Tensor, sw: torch.Tensor,
                  out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """h = bf16(silu(gate) * up) of the fused gate|up projection (spec_fp8_gemm_silu_mul).

    a: uint8 E4M3 [M,K]; w: uint8 E4M3 [2I,K] (gate rows, then up rows);
    sa, sw as for gemm.  Returns h bf16 [M,I].
    """
    lib = _lib.load()
    _dev(a, torch.uint8, "a")
    _dev(w, torch.uint8, "w")
    _dev(sa, torch.float32, "sa")
    _dev(sw, torch.float32, "sw")
    M, K = a.shape
    if w.shape[1] != K or w.shape[0] % 2:
        raise ValueError("w must be [2I, K] with the activations' K")
    I = w.shape[0] // 2
    a_mode, w_mode = _scale_modes(a, sa, w, sw)
    if out is None:
        ld = (I + 7) // 8 * 8
        out = torch.empty((M, ld), dtype=torch.bfloat16, device=a.device)[:, :I]
    _dev(out, torch.bfloat16, "out")
    check("spec_fp8_gemm_silu_mul", lib.spec_fp8_gemm_silu_mul(
        a.data_ptr(), _rowmajor(a, "a"), sa.data_ptr(), a_mode, w.data_ptr(), _rowmajor(w, "w"), sw.data_ptr(),
        w_mode, M, I, K, out.data_ptr(), _rowmajor(out, "out"), _stream()))
    return out


def logit_stats_count(M: int, V: int, K: int) -> int:
    return int(_lib.load().spec_logit_stats_count(M, V, K))


def gemm_logit_stats(a: torch.Tensor, sa: torch.Tensor, w: torch.Tensor, sw: torch.Tensor, temperature: float,
                     out: Optional[torch.Tensor] = None, stats: Optional[torch.Tensor] = None
                     ) -> Tuple[torch.Tensor, torch.Tensor]:
    """LM-head GEMM with the acceptance statistics in its epilogue (spec_fp8_gemm_logit_stats).

    a: uint8 E4M3 [M,K] (final hidden states of the verify rows); w: uint8 E4M3 [V,K];
    sa, sw as for gemm.  Returns (logits bf16 [M,V], stats fp32 [M,G,2]) with
    G = logit_stats_count(M, V, K) column groups per row.
    """
    lib = _lib.load()
    _dev(a, torch.uint8, "a")
    _dev(w, torch.uint8, "w")
    _dev(sa, torch.float32, "sa")
    _dev(sw, torch.float32, "sw")
    M, K = a.shape
    V = w.shape[0]
    if w.shape[1] != K:
        raise ValueError("a and w disagree on K")
    a_mode, w_mode = _scale_modes(a, sa, w, sw)
    G = logit_stats_count(M, V, K)
    if out is None:
        ld = (V + 7) // 8 * 8
        out = torch.empty((M, ld), dtype=torch.bfloat16, device=a.device)[:, :V]
    _dev(out, torch.bfloat16, "out")
    if stats is None:
        stats = torch.empty((M, G, 2), dtype=torch.float32, device=a.device)
    _dev(stats, torch.float32, "stats")
    if stats.dim() != 3 or stats.shape[0] != M or stats.shape[2] != 2 or stats.stride(2) != 1 or \
            stats.stride(1) != 2:
        raise ValueError("stats must be [M, >=G, 2] with contiguous pairs")
    check("spec_fp8_gemm_logit_stats", lib.spec_fp8_gemm_logit_stats(
        a.data_ptr(), _rowmajor(a, "a"), sa.data_ptr(), a_mode, w.data_ptr(), _rowmajor(w, "w"), sw.data_ptr(),
        w_mode, M, V, K, float(temperature), out.data_ptr(), _rowmajor(out, "out"), stats.data_ptr(),
        stats.stride(0) // 2, _stream()))
    return out, stats


def accept_workspace_bytes(B: int, k: int, V: int) -> int:
    return int(_lib.load().spec_verify_accept_workspace_bytes(B, k, V))


def verify_accept(target_logits: torch.Tensor, draft_logits: Optional[torch.Tensor], draft_tokens: torch.Tensor,
                  uniforms: Optional[torch.Tensor], temperature: float,
                  workspace: Optional[torch.Tensor] = None,
                  out_tokens: Optional[torch.Tensor] = None, num_accepted: Optional[torch.Tensor] = None,
                  target_stats: Optional[torch.Tensor] = None) -> Tuple[torch.Tensor, torch.Tensor]:
    """Greedy (T=0) or speculative-sampling (T>0) acceptance (spec_verify_accept, or
    spec_verify_accept_stats when target_stats from gemm_logit_stats are given).

    target_logits bf16 [B,k+1,V]; draft_logits bf16 [B,k,V] or None;
    draft_tokens int32 [B,k]; uniforms fp32 [B,k+1] (T>0);
    target_stats fp32 [B*(k+1), G, 2] (pairs) or None.
    Returns (out_tokens int32 [B,k+1] (-1 padded), num_accepted int32 [B]).
    """
    lib = _lib.load()
    _dev(target_logits, torch.bfloat16, "target_logits")
    B, k1, V = target_logits.shape
    k = k1 - 1
    if not target_logits.is_contiguous():
        raise ValueError("target_logits must be contiguous")
    if draft_logits is not None:
        _dev(draft_logits, torch.bfloat16, "draft_logits")
        if tuple(draft_logits.shape) != (B, k, V) or not draft_logits.is_contiguous():
            raise ValueError("draft_logits must be contiguous [B,k,V]")
    _dev(draft_tokens, torch.int32, "draft_tokens")
    if tuple(draft_tokens.shape) != (B, k) or not draft_tokens.is_contiguous():
        raise ValueError("draft_tokens must be contiguous [B,k]")
    if uniforms is not None:
        _dev(uniforms, torch.float32, "uniforms")
        if tuple(uniforms.shape) != (B, k1) or not uniforms.is_contiguous():
            raise ValueError("uniforms must be contiguous [B,k+1]")
    if out_tokens is None:
        out_tokens = torch.empty((B, k1), dtype=torch.int32, device=target_logits.device)
    if num_accepted is None:
        num_accepted = torch.empty((B,), dtype=torch.int32, device=target_logits.device)
    need = accept_workspace_bytes(B, k, V)
    if workspace is None or workspace.numel() * workspace.element_size() < need:
        workspace = torch.empty((max(need, 1),), dtype=torch.uint8, device=target_logits.device)
    if target_stats is None:
        check("spec_verify_accept", lib.spec_verify_accept(
            target_logits.data_ptr(), None if draft_logits is None else draft_logits.data_ptr(),
            draft_tokens.data_ptr(), None if uniforms is None else uniforms.data_ptr(), B, k, V,
            float(temperature), out_tokens.data_ptr(), num_accepted.data_ptr(), workspace.data_ptr(),
            workspace.numel() * workspace.element_size(), _stream()))
    else:
        _dev(target_stats, torch.float32, "target_stats")
        if target_stats.dim() != 3 or target_stats.shape[0] != B * k1 or target_stats.shape[2] != 2 or \
                target_stats.stride(2) != 1 or target_stats.stride(1) != 2:
            raise ValueError("target_stats must be [B*(k+1), G, 2] with contiguous pairs")
        check("spec_verify_accept_stats", lib.spec_verify_accept_stats(
            target_logits.data_ptr(), target_stats.data_ptr(), target_stats.shape[1], target_stats.stride(0) // 2,
            None if draft_logits is None else draft_logits.data_ptr(), draft_tokens.data_ptr(),
            None if uniforms is None else uniforms.data_ptr(), B, k, V, float(temperature), out_tokens.data_ptr(),
            num_accepted.data_ptr(), workspace.data_ptr(), workspace.numel() * workspace.element_size(),
            _stream()))
    return out_tokens, num_accepted


def verify_accept_noalloc(target_logits: torch.Tensor, draft_logits: Optional[torch.Tensor],
                          draft_tokens: torch.Tensor, uniforms: Optional[torch.Tensor], temperature: float,
                          out_tokens: torch.Tensor, num_accepted: torch.Tensor) -> Tuple[torch.Tensor, torch.Tensor]:
    """verify_accept through spec_verify_accept_noalloc: no workspace, the
    library's fixed device scratch instead, and no allocation here either (the
    outputs are the caller's).  Same arguments and results as verify_accept."""
    lib = _lib.load()
    _dev(target_logits, torch.bfloat16, "target_logits")
    B, k1, V = target_logits.shape
    k = k1 - 1
    if not target_logits.is_contiguous():
        raise ValueError("target_logits must be contiguous")
    if draft_logits is not None:
        _dev(draft_logits, torch.bfloat16, "draft_logits")
        if tuple(draft_logits.shape) != (B, k, V) or not draft_logits.is_contiguous():
            raise ValueError("draft_logits must be contiguous [B,k,V]")
    _dev(draft_tokens, torch.int32, "draft_tokens")
    if tuple(draft_tokens.shape) != (B, k) or not draft_tokens.is_contiguous():
        raise ValueError("draft_tokens must be contiguous [B,k]")
    if uniforms is not None:
        _dev(uniforms, torch.float32, "uniforms")
        if tuple(uniforms.shape) != (B, k1) or not uniforms.is_contiguous():
            raise ValueError("uniforms must be contiguous [B,k+1]")
    _dev(out_tokens, torch.int32, "out_tokens")
    _dev(num_accepted, torch.int32, "num_accepted")
    if tuple(out_tokens.shape) != (B, k1) or not out_tokens.is_contiguous():
        raise ValueError("out_tokens must be contiguous [B,k+1]")
    if tuple(num_accepted.shape) != (B,) or not num_accepted.is_contiguous():
        raise ValueError("num_accepted must be contiguous [B]")
    check("spec_verify_accept_noalloc", lib.spec_verify_accept_noalloc(
        target_logits.data_ptr(), None if draft_logits is None else draft_logits.data_ptr(),
        draft_tokens.data_ptr(), None if uniforms is None else uniforms.data_ptr(), B, k, V,
        float(temperature), out_tokens.data_ptr(), num_accepted.data_ptr(), _stream()))
    return out_tokens, num_accepted


def accept_tree_workspace_bytes(B: int, N: int, V: int) -> int:
    return int(_lib.load().spec_verify_accept_tree_workspace_bytes(B, N, V))


def verify_accept_tree(target_logits: torch.Tensor, parents: torch.Tensor, tokens: torch.Tensor,
                       uniforms: Optional[torch.Tensor], temperature: float,
                       workspace: Optional[torch.Tensor] = None, out_tokens: Optional[torch.Tensor] = None,
                       accepted_nodes: Optional[torch.Tensor] = None, num_accepted: Optional[torch.Tensor] = None
                       ) -> Tuple[torch.Tensor, torch.Tensor, torch.Tensor]:
    """Token-tree acceptance (spec_verify_accept_tree).

    target_logits bf16 [B,N+1,V]; parents, tokens int32 [B,N]; uniforms fp32 [B,N+1] (T>0).
    Returns (out_tokens int32 [B,N+1], accepted_nodes int32 [B,N], num_accepted int32 [B]).
    """
    lib = _lib.load()
    _dev(target_logits, torch.bfloat16, "target_logits")
    B, N1, V = target_logits.shape
    N = N1 - 1
    if not target_logits.is_contiguous():
        raise ValueError("target_logits must be contiguous")
    for name, t in (("parents", parents), ("tokens", tokens)):
        _dev(t, torch.int32, name)
        if tuple(t.shape) != (B, N) or not t.is_contiguous():
            raise ValueError(f"{name} must be contiguous [B,N]")
    if uniforms is not None:
        _dev(uniforms, torch.float32, "uniforms")
        if tuple(uniforms.shape) != (B, N1) or not uniforms.is_contiguous():
            raise ValueError("uniforms must be contiguous [B,N+1]")
    dev = target_logits.device
    if out_tokens is None:
        out_tokens = torch.empty((B, N1), dtype=torch.int32, device=dev)
    if accepted_nodes is None:
        accepted_nodes = torch.empty((B, N), dtype=torch.int32, device=dev)
    if num_accepted is None:
        num_accepted = torch.empty((B,), dtype=torch.int32, device=dev)
    need = accept_tree_workspace_bytes(B, N, V)
    if workspace is None or workspace.numel() * workspace.element_size() < need:
        workspace = torch.empty((max(need, 1),), dtype=torch.uint8, device=dev)
    check("spec_verify_accept_tree", lib.spec_verify_accept_tree(
        target_logits.data_ptr(), parents.data_ptr(), tokens.data_ptr(),
        None if uniforms is None else uniforms.data_ptr(), B, N, V, float(temperature), out_tokens.data_ptr(),
        accepted_nodes.data_ptr(), num_accepted.data_ptr(), workspace.data_ptr(),
        workspace.numel() * workspace.element_size(), _stream()))
    return out_tokens, accepted_nodes, num_accepted


def tree_attention_mask(parents: torch.Tensor, mask: Optional[torch.Tensor] = None,
                        depth: Optional[torch.Tensor] = None) -> Tuple[torch.Tensor, torch.Tensor]:
    """Ancestor-or-self masks and depths of B drafted trees (spec_tree_attention_mask).

    parents: int32 [B, N] (N <= 64).  Returns (mask int64 [B, N] holding the
    uint64 bit patterns, bit j = node j; depth int32 [B, N]).
    """
    lib = _lib.load()
    _dev(parents, torch.int32, "parents")
    if parents.dim() != 2 or not parents.is_contiguous():
        raise ValueError("parents must be a contiguous int32 [B, N]")
    B, N = parents.shape
    if mask is None:
        mask = torch.empty((B, N), dtype=torch.int64, device=parents.device)
    if depth is None:
        depth = torch.empty((B, N), dtype=torch.int32, device=parents.device)
    _dev(mask, torch.int64, "mask")
    _dev(depth, torch.int32, "depth")
    if mask.shape != (B, N) or depth.shape != (B, N) or not mask.is_contiguous() or not depth.is_contiguous():
        raise ValueError("mask and depth must be contiguous [B, N]")
    check("spec_tree_attention_mask", lib.spec_tree_attention_mask(parents.data_ptr(), B, N, mask.data_ptr(),
                                                                   depth.data_ptr(), _stream()))
    return mask, depth
