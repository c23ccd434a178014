// extern "C" entry points of libspecfp8.so: validate on the host, then
// enqueue the kernels on the caller's stream.  Nothing here allocates,
// frees or synchronizes.
#include <hip/hip_runtime.h>

#include "../../include/spec_fp8.h"
#include "kernels.hpp"
#include "validate.hpp"

namespace {

thread_local int g_last_hip_error = 0;

inline spec_status from_hip(hipError_t e) {
    if (e == hipSuccess) return SPEC_OK;
    g_last_hip_error = (int)e;
    return SPEC_ERR_HIP;
}

inline hipStream_t as_stream(void* s) { return reinterpret_cast<hipStream_t>(s); }

// One workgroup per (tile, K-split): the grid is an int.
inline bool grid_fits(const specfp8::GemmPlan& p) {
    return (int64_t)p.m_tiles * p.n_tiles * p.splits <= 2147483647LL;
}

}  // namespace

extern "C" {

spec_status spec_fp8_quantize(const void* x, int64_t rows, int64_t cols, int64_t ld_x,
                              spec_quant_input in_kind, spec_scale_mode mode, float* scales, uint8_t* q,
                              int64_t ld_q, void* stream) {
    const spec_status st = specfp8::check_quantize(x, rows, cols, ld_x, (int)in_kind, (int)mode, scales, q, ld_q);
    if (st != SPEC_OK || rows == 0) return st;
    return from_hip(specfp8::launch_quantize(reinterpret_cast<const uint16_t*>(x), rows, cols, ld_x, (int)in_kind,
                                             (int)mode, scales, q, ld_q, as_stream(stream)));
}

spec_status spec_silu_mul_bf16(const void* x, int64_t rows, int64_t cols, int64_t ld_x, void* h, int64_t ld_h,
                               void* stream) {
    const spec_status st = specfp8::check_silu_mul(x, rows, cols, ld_x, h, ld_h);
    if (st != SPEC_OK || rows == 0) return st;
    return from_hip(specfp8::launch_silu_mul(reinterpret_cast<const uint16_t*>(x), rows, cols, ld_x,
                                             reinterpret_cast<uint16_t*>(h), ld_h, as_stream(stream)));
}

spec_status spec_fp8_clip_count(const void* x, int64_t rows, int64_t cols, int64_t ld_x, const float* scale,
                               uint64_t* count, void* stream) {
    const spec_status st = specfp8::check_clip_count(x, rows, cols, ld_x, scale, count);
    if (st != SPEC_OK || rows == 0) return st;
    return from_hip(specfp8::launch_clip_count(reinterpret_cast<const uint16_t*>(x), rows, cols, ld_x, scale,
                                               reinterpret_cast<unsigned long long*>(count), as_stream(stream)));
}

spec_status spec_fp8_kv_cache_write(const void* k, int64_t ld_k, const void* v, int64_t ld_v,
                                    const int64_t* slot_mapping, int64_t T, int64_t H, int64_t D,
                                    int64_t num_slots, spec_scale_mode mode, float* k_scale, float* v_scale,
                                    uint8_t* k_cache, uint8_t* v_cache, void* stream) {
    const spec_status st = specfp8::check_kv_cache_write(k, ld_k, v, ld_v, slot_mapping, T, H, D, num_slots,
                                                         (int)mode, k_scale, v_scale, k_cache, v_cache);
    if (st != SPEC_OK || T == 0 || num_slots == 0) return st;
    return from_hip(specfp8::launch_kv_cache_write(
        reinterpret_cast<const uint16_t*>(k), ld_k, reinterpret_cast<const uint16_t*>(v), ld_v, slot_mapping, T, H,
        D, num_slots, mode == SPEC_SCALE_PER_TENSOR ? 1 : 0, k_scale, v_scale, k_cache, v_cache,
        as_stream(stream)));
}

size_t spec_fp8_gemm_workspace_bytes(int64_t M, int64_t N, int64_t K) {
    if (M <= 0 || N <= 0 || K <= 0 || K % 128 != 0) return 0;
    return specfp8::plan_gemm(M, N, K).workspace_bytes;
}

spec_status spec_fp8_gemm(const uint8_t* a, int64_t lda, const float* a_scale, spec_scale_mode a_mode,
                          const uint8_t* w, int64_t ldw, const float* w_scale, spec_scale_mode w_mode, int64_t M,
                          int64_t N, int64_t K, void* y, int64_t ldy, spec_out_dtype out_dtype, void* workspace,
                          size_t workspace_bytes, void* stream) {
    const spec_status st = specfp8::check_gemm(a, lda, a_scale, (int)a_mode, w, ldw, w_scale, (int)w_mode, M, N, K,
                                               y, ldy, (int)out_dtype);
    if (st != SPEC_OK || M == 0) return st;
    const specfp8::GemmPlan plan = specfp8::plan_gemm(M, N, K);
    if (!grid_fits(plan)) return SPEC_ERR_UNSUPPORTED;
    if (plan.workspace_bytes > 0) {
        if (!workspace || workspace_bytes < plan.workspace_bytes) return SPEC_ERR_WORKSPACE;
        if ((reinterpret_cast<uintptr_t>(workspace) & 15u) != 0) return SPEC_ERR_ALIGN;
    }
    return from_hip(specfp8::launch_gemm(plan, a, lda, a_scale, a_mode == SPEC_SCALE_PER_TENSOR, w, ldw, w_scale,
                                         w_mode == SPEC_SCALE_PER_TENSOR, M, N, K, y, ldy, out_dtype == SPEC_OUT_F32,
                                         workspace, as_stream(stream)));
}

size_t spec_logit_stats_count(int64_t M, int64_t V, int64_t K) {
    if (M <= 0 || V <= 0 || K <= 0 || K % 128 != 0) return 0;
    if (M > 2147483647LL || V > 2147483647LL || K > 2147483647LL) return 0;
    return (size_t)specfp8::plan_gemm(M, V, K, specfp8::kEpiStats).stat_groups;
}

spec_status spec_fp8_gemm_logit_stats(const uint8_t* a, int64_t lda, const float* a_scale, spec_scale_mode a_mode,
                                      const uint8_t* w, int64_t ldw, const float* w_scale, spec_scale_mode w_mode,
                                      int64_t M, int64_t V, int64_t K, float temperature, void* logits,
                                      int64_t ld_logits, float* stats, int64_t ld_stats, void* stream) {
    spec_status st = specfp8::check_gemm(a, lda, a_scale, (int)a_mode, w, ldw, w_scale, (int)w_mode, M, V, K, logits,
                                         ld_logits, SPEC_OUT_BF16);
    if (st != SPEC_OK) return st;
    const specfp8::GemmPlan plan = specfp8::plan_gemm(M > 0 ? M : 1, V, K, specfp8::kEpiStats);
    st = specfp8::check_logit_stats(M, V, temperature, logits, ld_logits, stats, ld_stats, plan.stat_groups);
    if (st != SPEC_OK || M == 0) return st;
    if (!grid_fits(plan) || !specfp8::gemm_strides_fit(plan.kind, lda, ldw)) return SPEC_ERR_UNSUPPORTED;
    const float c2 = temperature > 0.0f ? (float)(1.4426950408889634 / (double)temperature) : 0.0f;
    return from_hip(specfp8::launch_gemm(plan, a, lda, a_scale, a_mode == SPEC_SCALE_PER_TENSOR, w, ldw, w_scale,
                                         w_mode == SPEC_SCALE_PER_TENSOR, M, V, K, logits, ld_logits, 0, nullptr,
                                         as_stream(stream), temperature > 0.0f ? 1 : 2, c2,
                                         reinterpret_cast<float2*>(stats), ld_stats));
}

spec_status spec_fp8_gemm_silu_mul(const uint8_t* a, int64_t lda, const float* a_scale, spec_scale_mode a_mode,
                                   const uint8_t* w, int64_t ldw, const float* w_scale, spec_scale_mode w_mode,
                                   int64_t M, int64_t I, int64_t K, void* h, int64_t ldh, void* stream) {
    if (I <= 0) return SPEC_ERR_SHAPE;
    if (I % 8 != 0 || I > 1073741823LL) return SPEC_ERR_UNSUPPORTED;
    if (ldh < I) return SPEC_ERR_SHAPE;
    // the weight operand is [2I, K]; the output checks are those of a bf16 [M, I] result
    spec_status st = specfp8::check_gemm(a, lda, a_scale, (int)a_mode, w, ldw, w_scale, (int)w_mode, M, 2 * I, K, h,
                                         2 * I, SPEC_OUT_BF16);
    if (st != SPEC_OK || M == 0) return st;
    if (ldh % 8 != 0 || (reinterpret_cast<uintptr_t>(h) & 15u)) return SPEC_ERR_ALIGN;
    const specfp8::GemmPlan plan = specfp8::plan_gemm(M, 2 * I, K, specfp8::kEpiSilu);
    if (!grid_fits(plan)) return SPEC_ERR_UNSUPPORTED;
    return from_hip(specfp8::launch_gemm(plan, a, lda, a_scale, a_mode == SPEC_SCALE_PER_TENSOR, w, ldw, w_scale,
                                         w_mode == SPEC_SCALE_PER_TENSOR, M, 2 * I, K, h, ldh, 0, nullptr,
                                         as_stream(stream), 0, 0.0f, nullptr, 0, I));
}

size_t spec_verify_accept_workspace_bytes(int64_t B, int64_t k, int64_t V) {
    if (B <= 0 || k < 1 || V < 1) return 0;
    return specfp8::plan_accept(B, k, V).bytes;
}

spec_status spec_verify_accept(const void* target_logits, const void* draft_logits, const int32_t* draft_tokens,
                               const float* uniforms, int64_t B, int64_t k, int64_t V, float temperature,
                               int32_t* out_tokens, int32_t* num_accepted, void* workspace, size_t workspace_bytes,
                               void* stream) {
    const spec_status st = specfp8::check_accept(target_logits, draft_logits, draft_tokens, uniforms, B, k, V,
                                                 temperature, out_tokens, num_accepted);
    if (st != SPEC_OK || B == 0) return st;
    const specfp8::AcceptPlan plan = specfp8::plan_accept(B, k, V);
    if (!workspace || workspace_bytes < plan.bytes) return SPEC_ERR_WORKSPACE;
    if ((reinterpret_cast<uintptr_t>(workspace) & 15u) != 0) return SPEC_ERR_ALIGN;
    return from_hip(specfp8::launch_accept(plan, reinterpret_cast<const uint16_t*>(target_logits),
                                           reinterpret_cast<const uint16_t*>(draft_logits), draft_tokens, uniforms,
                                           B, k, V, temperature, out_tokens, num_accepted, workspace,
                                           as_stream(stream)));
}

spec_status spec_verify_accept_noalloc(const void* target_logits, const void* draft_logits,
                                       const int32_t* draft_tokens, const float* uniforms, int64_t B, int64_t k,
                                       int64_t V, float temperature, int32_t* out_tokens, int32_t* num_accepted,
                                       void* stream) {
    const spec_status st = specfp8::check_accept(target_logits, draft_logits, draft_tokens, uniforms, B, k, V,
                                                 temperature, out_tokens, num_accepted);
    if (st != SPEC_OK || B == 0) return st;
    const specfp8::AcceptPlan plan = specfp8::plan_accept(B, k, V);
    if (plan.bytes > specfp8::kAcceptScratchBytes) return SPEC_ERR_SCRATCH;
    void* ws = nullptr;
    const spec_status se = from_hip(specfp8::accept_scratch(&ws));
    if (se != SPEC_OK) return se;
    return from_hip(specfp8::launch_accept(plan, reinterpret_cast<const uint16_t*>(target_logits),
                                           reinterpret_cast<const uint16_t*>(draft_logits), draft_tokens, uniforms,
                                           B, k, V, temperature, out_tokens, num_accepted, ws,
                                           as_stream(stream)));
}

spec_status spec_verify_accept_stats(const void* target_logits, const float* target_stats, int64_t n_stats,
                                     int64_t ld_stats, const void* draft_logits, const int32_t* draft_tokens,
                                     const float* uniforms, int64_t B, int64_t k, int64_t V, float temperature,
                                     int32_t* out_tokens, int32_t* num_accepted, void* workspace,
                                     size_t workspace_bytes, void* stream) {
    spec_status st = specfp8::check_accept(target_logits, draft_logits, draft_tokens, uniforms, B, k, V, temperature,
                                           out_tokens, num_accepted);
    if (st != SPEC_OK) return st;
    st = specfp8::check_accept_stats(target_stats, n_stats, ld_stats, B);
    if (st != SPEC_OK || B == 0) return st;
    const specfp8::AcceptPlan plan = specfp8::plan_accept(B, k, V);
    if (!workspace || workspace_bytes < plan.bytes) return SPEC_ERR_WORKSPACE;
    if ((reinterpret_cast<uintptr_t>(workspace) & 15u) != 0) return SPEC_ERR_ALIGN;
    return from_hip(specfp8::launch_accept(plan, reinterpret_cast<const uint16_t*>(target_logits),
                                           reinterpret_cast<const uint16_t*>(draft_logits), draft_tokens, uniforms,
                                           B, k, V, temperature, out_tokens, num_accepted, workspace,
                                           as_stream(stream), reinterpret_cast<const float2*>(target_stats),
                                           n_stats, ld_stats));
}

size_t spec_verify_accept_tree_workspace_bytes(int64_t B, int64_t N, int64_t V) {
    if (B <= 0 || N < 1 || V < 1) return 0;
    return specfp8::plan_accept(B, N, V).bytes;
}

spec_status spec_verify_accept_tree(const void* target_logits, const int32_t* parents, const int32_t* tokens,
                                    const float* uniforms, int64_t B, int64_t N, int64_t V, float temperature,
                                    int32_t* out_tokens, int32_t* accepted_nodes, int32_t* num_accepted,
                                    void* workspace, size_t workspace_bytes, void* stream) {
    const spec_status st = specfp8::check_accept_tree(target_logits, parents, tokens, uniforms, B, N, V, temperature,
                                                      out_tokens, accepted_nodes, num_accepted);
    if (st != SPEC_OK || B == 0) return st;
    const specfp8::AcceptPlan plan = specfp8::plan_accept(B, N, V);
    if (!workspace || workspace_bytes < plan.bytes) return SPEC_ERR_WORKSPACE;
    if ((reinterpret_cast<uintptr_t>(workspace) & 15u) != 0) return SPEC_ERR_ALIGN;
    return from_hip(specfp8::launch_accept_tree(plan, reinterpret_cast<const uint16_t*>(target_logits), parents,
                                                tokens, uniforms, B, N, V, temperature, out_tokens, accepted_nodes,
                                                num_accepted, workspace, as_stream(stream)));
}

spec_status spec_tree_attention_mask(const int32_t* parents, int64_t B, int64_t N, uint64_t* mask, int32_t* depth,
                                     void* stream) {
    const spec_status st = specfp8::check_tree_mask(parents, B, N, mask, depth);
    if (st != SPEC_OK || B == 0) return st;
    return from_hip(specfp8::launch_tree_mask(parents, B, N, mask, depth, as_stream(stream)));
}

const char* spec_status_string(spec_status s) {
    switch (s) {
        case SPEC_OK: return "ok";
        case SPEC_ERR_NULL: return "required pointer is NULL";
        case SPEC_ERR_SHAPE: return "invalid shape or leading dimension";
        case SPEC_ERR_UNSUPPORTED: return "shape outside the supported fast path";
        case SPEC_ERR_ENUM: return "unknown enum value";
        case SPEC_ERR_ALIGN: return "misaligned pointer or leading dimension";
        case SPEC_ERR_WORKSPACE: return "workspace missing or too small";
        case SPEC_ERR_HIP: return "HIP launch failed";
        case SPEC_ERR_VALUE: return "scalar argument out of range";
        case SPEC_ERR_SCRATCH: return "call exceeds the library's fixed scratch buffer";
    }
    return "unknown status";
}

int spec_last_hip_error(void) { return g_last_hip_error; }

int spec_version(void) { return 510; }

}  // extern "C"
