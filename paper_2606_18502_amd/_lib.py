"""ctypes declarations of libspecfp8.so (the C ABI in include/spec_fp8.h)."""

from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libspecfp8.so")

# enums and limits (include/spec_fp8.h)
ACCEPT_SCRATCH_BYTES = 16 << 20
SPEC_OK = 0
STATUS_NAMES = {0: "SPEC_OK", 1: "SPEC_ERR_NULL", 2: "SPEC_ERR_SHAPE", 3: "SPEC_ERR_UNSUPPORTED",
                4: "SPEC_ERR_ENUM", 5: "SPEC_ERR_ALIGN", 6: "SPEC_ERR_WORKSPACE", 7: "SPEC_ERR_HIP",
                8: "SPEC_ERR_VALUE", 9: "SPEC_ERR_SCRATCH"}
SCALE_PER_ROW, SCALE_PER_TENSOR, SCALE_CALIBRATE = 0, 1, 2
QIN_BF16, QIN_SILU_MUL_BF16 = 0, 1
OUT_BF16, OUT_F32 = 0, 1

EXPORTS = ("spec_fp8_quantize", "spec_silu_mul_bf16", "spec_fp8_kv_cache_write", "spec_fp8_clip_count", "spec_fp8_gemm_workspace_bytes", "spec_fp8_gemm",
           "spec_fp8_gemm_silu_mul", "spec_logit_stats_count", "spec_fp8_gemm_logit_stats",
           "spec_verify_accept_workspace_bytes", "spec_verify_accept", "spec_verify_accept_noalloc",
           "spec_verify_accept_stats",
           "spec_verify_accept_tree_workspace_bytes", "spec_verify_accept_tree", "spec_tree_attention_mask",
           "spec_status_string", "spec_last_hip_error", "spec_version")

_lib = None


class SpecError(RuntimeError):
    def __init__(self, fn: str, status: int):
        self.status = status
        msg = f"{fn} failed: {STATUS_NAMES.get(status, status)}"
        if status == 7 and _lib is not None:
            msg += f" (hipError {_lib.spec_last_hip_error()})"
        super().__init__(msg)


def load() -> ctypes.CDLL:
    """Load libspecfp8.so; raises if it has not been built (there is no fallback)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with `python -m paper_2606_18502_amd.build`")
    _lib = declare(ctypes.CDLL(LIB_PATH))
    return _lib


def declare(lib: ctypes.CDLL) -> ctypes.CDLL:
    """Set the argument and result types of every entry point on a loaded
    library that exports the C ABI."""
    i64, vp, f32, sz, i32 = ctypes.c_int64, ctypes.c_void_p, ctypes.c_float, ctypes.c_size_t, ctypes.c_int
    lib.spec_fp8_quantize.argtypes = [vp, i64, i64, i64, i32, i32, vp, vp, i64, vp]
    lib.spec_fp8_quantize.restype = i32
    lib.spec_silu_mul_bf16.argtypes = [vp, i64, i64, i64, vp, i64, vp]
    lib.spec_silu_mul_bf16.restype = i32
    lib.spec_fp8_clip_count.argtypes = [vp, i64, i64, i64, vp, vp, vp]
    lib.spec_fp8_clip_count.restype = i32
    lib.spec_fp8_kv_cache_write.argtypes = [vp, i64, vp, i64, vp, i64, i64, i64, i64, i32, vp, vp, vp, vp, vp]
    lib.spec_fp8_kv_cache_write.restype = i32
    lib.spec_fp8_gemm_workspace_bytes.argtypes = [i64, i64, i64]
    lib.spec_fp8_gemm_workspace_bytes.restype = sz
    lib.spec_fp8_gemm.argtypes = [vp, i64, vp, i32, vp, i64, vp, i32, i64, i64, i64, vp, i64, i32, vp, sz, vp]
    lib.spec_fp8_gemm.restype = i32
    lib.spec_fp8_gemm_silu_mul.argtypes = [vp, i64, vp, i32, vp, i64, vp, i32, i64, i64, i64, vp, i64, vp]
    lib.spec_fp8_gemm_silu_mul.restype = i32
    lib.spec_logit_stats_count.argtypes = [i64, i64, i64]
    lib.spec_logit_stats_count.restype = sz
    lib.spec_fp8_gemm_logit_stats.argtypes = [vp, i64, vp, i32, vp, i64, vp, i32, i64, i64, i64, f32, vp, i64, vp,
                                              i64, vp]
    lib.spec_fp8_gemm_logit_stats.restype = i32
    lib.spec_verify_accept_stats.argtypes = [vp, vp, i64, i64, vp, vp, vp, i64, i64, i64, f32, vp, vp, vp, sz, vp]
    lib.spec_verify_accept_stats.restype = i32
    lib.spec_verify_accept_tree_workspace_bytes.argtypes = [i64, i64, i64]
    lib.spec_verify_accept_tree_workspace_bytes.restype = sz
    lib.spec_verify_accept_tree.argtypes = [vp, vp, vp, vp, i64, i64, i64, f32, vp, vp, vp, vp, sz, vp]
    lib.spec_verify_accept_tree.restype = i32
    lib.spec_tree_attention_mask.argtypes = [vp, i64, i64, vp, vp, vp]
    lib.spec_tree_attention_mask.restype = i32
    lib.spec_verify_accept_workspace_bytes.argtypes = [i64, i64, i64]
    lib.spec_verify_accept_workspace_bytes.restype = sz
    lib.spec_verify_accept.argtypes = [vp, vp, vp, vp, i64, i64, i64, f32, vp, vp, vp, sz, vp]
    lib.spec_verify_accept.restype = i32
    lib.spec_verify_accept_noalloc.argtypes = [vp, vp, vp, vp, i64, i64, i64, f32, vp, vp, vp]
    lib.spec_verify_accept_noalloc.restype = i32
    lib.spec_status_string.argtypes = [i32]
    lib.spec_status_string.restype = ctypes.c_char_p
    lib.spec_last_hip_error.argtypes = []
    lib.spec_last_hip_error.restype = i32
    lib.spec_version.argtypes = []
    lib.spec_version.restype = i32
    return lib


def check(fn: str, status: int) -> None:
    if status != SPEC_OK:
        raise SpecError(fn, status)
