// Host-only argument checks of the libspecfp8 C ABI.  No HIP here: every
// check runs before anything is enqueued, so argument errors never touch the
// device (and can be exercised on a machine without a GPU).
#pragma once

#include <stddef.h>
#include <stdint.h>

#include "../../include/spec_fp8.h"

namespace specfp8 {

spec_status check_quantize(const void* x, int64_t rows, int64_t cols, int64_t ld_x, int in_kind, int mode,
                           const float* scales, const void* q, int64_t ld_q);
spec_status check_silu_mul(const void* x, int64_t rows, int64_t cols, int64_t ld_x, const void* h,
                           int64_t ld_h);
spec_status check_clip_count(const void* x, int64_t rows, int64_t cols, int64_t ld_x, const float* scale,
                             const void* count);
spec_status check_gemm(const void* a, int64_t lda, const float* a_scale, int a_mode, const void* w,
                       int64_t ldw, const float* w_scale, int w_mode, int64_t M, int64_t N, int64_t K,
                       const void* y, int64_t ldy, int out_dtype);
spec_status check_kv_cache_write(const void* k, int64_t ld_k, const void* v, int64_t ld_v,
                                 const int64_t* slot_mapping, int64_t T, int64_t H, int64_t D, int64_t num_slots,
                                 int mode, const float* k_scale, const float* v_scale, const void* k_cache,
                                 const void* v_cache);
spec_status check_logit_stats(int64_t M, int64_t V, float temperature, const void* logits, int64_t ld_logits,
                              const float* stats, int64_t ld_stats, int64_t n_groups);
spec_status check_accept_stats(const float* target_stats, int64_t n_stats, int64_t ld_stats, int64_t B);
spec_status check_accept_tree(const void* target_logits, const int32_t* parents, const int32_t* tokens,
                              const float* uniforms, int64_t B, int64_t N, int64_t V, float temperature,
                              const int32_t* out_tokens, const int32_t* accepted_nodes,
                              const int32_t* num_accepted);
spec_status check_tree_mask(const int32_t* parents, int64_t B, int64_t N, const uint64_t* mask,
                            const int32_t* depth);
spec_status check_accept(const void* target_logits, const void* draft_logits, const int32_t* draft_tokens,
                         const float* uniforms, int64_t B, int64_t k, int64_t V, float temperature,
                         const int32_t* out_tokens, const int32_t* num_accepted);

}  // namespace specfp8
