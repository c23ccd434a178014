#include "validate.hpp"

#include <math.h>
#include <stdint.h>

namespace specfp8 {

namespace {

inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

constexpr int64_t kMaxGrid = 2147483647;   // grid.x limit
constexpr int64_t kMaxGridY = 65535;       // grid.y limit

}  // namespace

spec_status check_quantize(const void* x, int64_t rows, int64_t cols, int64_t ld_x, int in_kind, int mode,
                           const float* scales, const void* q, int64_t ld_q) {
    if (in_kind != SPEC_QIN_BF16 && in_kind != SPEC_QIN_SILU_MUL_BF16) return SPEC_ERR_ENUM;
    if (mode != SPEC_SCALE_PER_ROW && mode != SPEC_SCALE_PER_TENSOR && mode != SPEC_SCALE_CALIBRATE)
        return SPEC_ERR_ENUM;
    const bool codes = mode != SPEC_SCALE_CALIBRATE;   // calibration writes no codes
    if (rows < 0 || cols <= 0) return SPEC_ERR_SHAPE;
    const int64_t in_cols = in_kind == SPEC_QIN_SILU_MUL_BF16 ? 2 * cols : cols;
    if (ld_x < in_cols || (codes && ld_q < cols)) return SPEC_ERR_SHAPE;
    if (rows > kMaxGrid) return SPEC_ERR_UNSUPPORTED;
    if (cols % 8 != 0) return SPEC_ERR_UNSUPPORTED;
    if (rows == 0) return SPEC_OK;
    if (!x || (codes && !q) || !scales) return SPEC_ERR_NULL;
    if (ld_x % 8 != 0 || !aligned16(x)) return SPEC_ERR_ALIGN;
    if (codes && (ld_q % 8 != 0 || !aligned16(q))) return SPEC_ERR_ALIGN;
    if ((reinterpret_cast<uintptr_t>(scales) & 3u) != 0) return SPEC_ERR_ALIGN;
    return SPEC_OK;
}

spec_status check_silu_mul(const void* x, int64_t rows, int64_t cols, int64_t ld_x, const void* h,
                           int64_t ld_h) {
    if (rows < 0 || cols <= 0) return SPEC_ERR_SHAPE;
    if (ld_x < 2 * cols || ld_h < cols) return SPEC_ERR_SHAPE;
    if (cols % 8 != 0) return SPEC_ERR_UNSUPPORTED;
    if ((cols / 8 + 255) / 256 > kMaxGrid) return SPEC_ERR_UNSUPPORTED;
    if (rows == 0) return SPEC_OK;
    if (!x || !h) return SPEC_ERR_NULL;
    if (ld_x % 8 != 0 || ld_h % 8 != 0 || !aligned16(x) || !aligned16(h)) return SPEC_ERR_ALIGN;
    return SPEC_OK;
}

spec_status check_kv_cache_write(const void* k, int64_t ld_k, const void* v, int64_t ld_v,
                                 const int64_t* slot_mapping, int64_t T, int64_t H, int64_t D, int64_t num_slots,
                                 int mode, const float* k_scale, const float* v_scale, const void* k_cache,
                                 const void* v_cache) {
    if (mode != SPEC_SCALE_PER_ROW && mode != SPEC_SCALE_PER_TENSOR) return SPEC_ERR_ENUM;
    if (T < 0 || H <= 0 || D <= 0 || num_slots < 0) return SPEC_ERR_SHAPE;
    if (H > kMaxGrid || D > 512 || D % 8 != 0) return SPEC_ERR_UNSUPPORTED;
    if (ld_k < H * D || ld_v < H * D) return SPEC_ERR_SHAPE;
    if (T > kMaxGrid || num_slots > INT64_MAX / (H * D)) return SPEC_ERR_UNSUPPORTED;
    int64_t g = 1;                               // lanes per (token, head) row
    while (g * 8 < D) g *= 2;
    if ((T * H + 256 / g - 1) / (256 / g) > kMaxGrid) return SPEC_ERR_UNSUPPORTED;
    if (T == 0) return SPEC_OK;
    if (!k || !v || !slot_mapping || !k_scale || !v_scale || !k_cache || !v_cache) return SPEC_ERR_NULL;
    if (ld_k % 8 != 0 || ld_v % 8 != 0 || !aligned16(k) || !aligned16(v)) return SPEC_ERR_ALIGN;
    if (!aligned16(k_cache) || !aligned16(v_cache)) return SPEC_ERR_ALIGN;
    if ((reinterpret_cast<uintptr_t>(slot_mapping) & 7u) != 0) return SPEC_ERR_ALIGN;
    if ((reinterpret_cast<uintptr_t>(k_scale) & 3u) != 0 || (reinterpret_cast<uintptr_t>(v_scale) & 3u) != 0)
        return SPEC_ERR_ALIGN;
    return SPEC_OK;
}

spec_status check_tree_mask(const int32_t* parents, int64_t B, int64_t N, const uint64_t* mask,
                            const int32_t* depth) {
    if (B < 0 || N < 1) return SPEC_ERR_SHAPE;
    if (N > 64) return SPEC_ERR_UNSUPPORTED;
    if ((B + 3) / 4 > kMaxGrid) return SPEC_ERR_UNSUPPORTED;
    if (B == 0) return SPEC_OK;
    if (!parents || !mask || !depth) return SPEC_ERR_NULL;
    if ((reinterpret_cast<uintptr_t>(parents) & 3u) != 0 || (reinterpret_cast<uintptr_t>(depth) & 3u) != 0 ||
        (reinterpret_cast<uintptr_t>(mask) & 7u) != 0)
        return SPEC_ERR_ALIGN;
    return SPEC_OK;
}

spec_status check_clip_count(const void* x, int64_t rows, int64_t cols, int64_t ld_x, const float* scale,
                             const void* count) {
    if (rows < 0 || cols <= 0 || ld_x < cols) return SPEC_ERR_SHAPE;
    if (cols % 8 != 0) return SPEC_ERR_UNSUPPORTED;
    if (rows > INT64_MAX / cols) return SPEC_ERR_UNSUPPORTED;
    if (rows == 0) return SPEC_OK;
    if (!x || !scale || !count) return SPEC_ERR_NULL;
    if (ld_x % 8 != 0 || !aligned16(x)) return SPEC_ERR_ALIGN;
    if ((reinterpret_cast<uintptr_t>(scale) & 3u) != 0 || (reinterpret_cast<uintptr_t>(count) & 7u) != 0)
        return SPEC_ERR_ALIGN;
    return SPEC_OK;
}

spec_status check_gemm(const void* a, int64_t lda, const float* a_scale, int a_mode, const void* w,
                       int64_t ldw, const float* w_scale, int w_mode, int64_t M, int64_t N, int64_t K,
                       const void* y, int64_t ldy, int out_dtype) {
    if (a_mode != SPEC_SCALE_PER_ROW && a_mode != SPEC_SCALE_PER_TENSOR) return SPEC_ERR_ENUM;
    if (w_mode != SPEC_SCALE_PER_ROW && w_mode != SPEC_SCALE_PER_TENSOR) return SPEC_ERR_ENUM;
    if (out_dtype != SPEC_OUT_BF16 && out_dtype != SPEC_OUT_F32) return SPEC_ERR_ENUM;
    if (M < 0 || N <= 0 || K <= 0) return SPEC_ERR_SHAPE;
    if (lda < K || ldw < K || ldy < N) return SPEC_ERR_SHAPE;
    if (K % 128 != 0) return SPEC_ERR_UNSUPPORTED;
    if (M > 2147483647LL || N > 2147483647LL || K > 2147483647LL) return SPEC_ERR_UNSUPPORTED;
    if (M == 0) return SPEC_OK;
    if (!a || !w || !a_scale || !w_scale || !y) return SPEC_ERR_NULL;
    if (lda % 16 != 0 || ldw % 16 != 0 || !aligned16(a) || !aligned16(w)) return SPEC_ERR_ALIGN;
    if (ldy % 8 != 0 || !aligned16(y)) return SPEC_ERR_ALIGN;
    if ((reinterpret_cast<uintptr_t>(a_scale) & 3u) || (reinterpret_cast<uintptr_t>(w_scale) & 3u))
        return SPEC_ERR_ALIGN;
    return SPEC_OK;
}

// The LM-head variant's own arguments (the GEMM operands are checked by
// check_gemm with N = V, y = logits, bf16 out).
spec_status check_logit_stats(int64_t M, int64_t V, float temperature, const void* logits, int64_t ld_logits,
                              const float* stats, int64_t ld_stats, int64_t n_groups) {
    (void)V; (void)logits; (void)ld_logits;
    if (!isfinite(temperature) || temperature < 0.0f) return SPEC_ERR_VALUE;
    if (ld_stats < n_groups) return SPEC_ERR_SHAPE;
    if (M == 0) return SPEC_OK;
    if (!stats) return SPEC_ERR_NULL;
    if (reinterpret_cast<uintptr_t>(stats) & 7u) return SPEC_ERR_ALIGN;
    return SPEC_OK;
}

spec_status check_accept_stats(const float* target_stats, int64_t n_stats, int64_t ld_stats, int64_t B) {
    if (n_stats < 1 || ld_stats < n_stats) return SPEC_ERR_SHAPE;
    if (n_stats > 2147483647LL) return SPEC_ERR_UNSUPPORTED;
    if (B == 0) return SPEC_OK;
    if (!target_stats) return SPEC_ERR_NULL;
    if (reinterpret_cast<uintptr_t>(target_stats) & 7u) return SPEC_ERR_ALIGN;
    return SPEC_OK;
}

spec_status check_accept_tree(const void* target_logits, const int32_t* parents, const int32_t* tokens,
                              const float* uniforms, int64_t B, int64_t N, int64_t V, float temperature,
                              const int32_t* out_tokens, const int32_t* accepted_nodes,
                              const int32_t* num_accepted) {
    if (!isfinite(temperature) || temperature < 0.0f) return SPEC_ERR_VALUE;
    if (B < 0 || N < 1 || V < 1) return SPEC_ERR_SHAPE;
    if (N > 64 || V > 4194304LL || B > kMaxGridY) return SPEC_ERR_UNSUPPORTED;
    // the streaming kernels count (row, 4096-logit slice) items in 31 bits
    if (B * (N + 1) * ((V + 4095) / 4096) > 2147483647LL) return SPEC_ERR_UNSUPPORTED;
    if (B == 0) return SPEC_OK;
    if (!target_logits || !parents || !tokens || !out_tokens || !accepted_nodes || !num_accepted)
        return SPEC_ERR_NULL;
    if (temperature > 0.0f && !uniforms) return SPEC_ERR_NULL;
    if (reinterpret_cast<uintptr_t>(target_logits) & 1u) return SPEC_ERR_ALIGN;
    if ((reinterpret_cast<uintptr_t>(parents) & 3u) || (reinterpret_cast<uintptr_t>(tokens) & 3u) ||
        (reinterpret_cast<uintptr_t>(out_tokens) & 3u) || (reinterpret_cast<uintptr_t>(accepted_nodes) & 3u) ||
        (reinterpret_cast<uintptr_t>(num_accepted) & 3u) || (uniforms && (reinterpret_cast<uintptr_t>(uniforms) & 3u)))
        return SPEC_ERR_ALIGN;
    return SPEC_OK;
}

spec_status check_accept(const void* target_logits, const void* draft_logits, const int32_t* draft_tokens,
                         const float* uniforms, int64_t B, int64_t k, int64_t V, float temperature,
                         const int32_t* out_tokens, const int32_t* num_accepted) {
    (void)draft_logits;
    if (!isfinite(temperature) || temperature < 0.0f) return SPEC_ERR_VALUE;
    if (B < 0 || k < 1 || V < 1) return SPEC_ERR_SHAPE;
    if (k > 16 || V > 4194304LL) return SPEC_ERR_UNSUPPORTED;   // <= 256 sampling chunks of 16384
    if (B * (2 * k + 1) > kMaxGridY) return SPEC_ERR_UNSUPPORTED;
    if (B == 0) return SPEC_OK;
    if (!target_logits || !draft_tokens || !out_tokens || !num_accepted) return SPEC_ERR_NULL;
    if (temperature > 0.0f && !uniforms) return SPEC_ERR_NULL;
    if ((reinterpret_cast<uintptr_t>(target_logits) & 1u) ||
        (draft_logits && (reinterpret_cast<uintptr_t>(draft_logits) & 1u)))
        return SPEC_ERR_ALIGN;
    if ((reinterpret_cast<uintptr_t>(draft_tokens) & 3u) || (reinterpret_cast<uintptr_t>(out_tokens) & 3u) ||
        (reinterpret_cast<uintptr_t>(num_accepted) & 3u) ||
        (uniforms && (reinterpret_cast<uintptr_t>(uniforms) & 3u)))
        return SPEC_ERR_ALIGN;
    return SPEC_OK;
}

}  // namespace specfp8
