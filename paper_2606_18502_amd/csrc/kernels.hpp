// Host-side launchers of the verify-path kernels (internal to libspecfp8).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace specfp8 {

// ---- quantize.hip
hipError_t launch_quantize(const uint16_t* x, int64_t rows, int64_t cols, int64_t ld_x, int in_kind,
                           int mode, float* scales, uint8_t* q, int64_t ld_q, hipStream_t stream);
hipError_t launch_silu_mul(const uint16_t* x, int64_t rows, int64_t cols, int64_t ld_x,
                           uint16_t* h, int64_t ld_h, hipStream_t stream);
// count += number of x values with |fl32(x * fl32(1/scale[0]))| > 448
hipError_t launch_clip_count(const uint16_t* x, int64_t rows, int64_t cols, int64_t ld_x, const float* scale,
                             unsigned long long* count, hipStream_t stream);

// ---- kvcache.hip
// Keys and values of T new tokens ([T][ld] bf16, H heads of D values each) to
// E4M3 codes in the slot-major caches [num_slots][H][D]; per-row scales go to
// [num_slots][H], a per-tensor scale is read from [0].
hipError_t launch_kv_cache_write(const uint16_t* k, int64_t ld_k, const uint16_t* v, int64_t ld_v,
                                 const int64_t* slot_mapping, int64_t T, int64_t H, int64_t D,
                                 int64_t num_slots, int per_tensor, float* k_scale, float* v_scale,
                                 uint8_t* k_cache, uint8_t* v_cache, hipStream_t stream);

// ---- gemm.hip
struct GemmPlan {
    int kind;              // tile configuration (plan.hpp, kTiles)
    int m_tiles, n_tiles;  // output tiles
    int splits;            // K-splits (1 = none)
    int reduce;            // kReduceLast when K is split (plan.hpp, GemmReduce)
    int group_m;           // > 1: tile order in groups of group_m M-tiles
    int krot_on;           // staggered K start per N-tile
    int64_t stat_groups;   // column groups per row of the epilogue statistics (n_tiles * waves across N)
    size_t part_off;       // byte offset of the partial tiles in the workspace (tickets before it)
    size_t workspace_bytes;
};
// Epilogue of a plan: plain (K may be split), logit statistics, or the
// SiLU-gated output; the last two keep one workgroup per output tile.
enum GemmEpilogue { kEpiPlain = 0, kEpiStats = 1, kEpiSilu = 2 };
GemmPlan plan_gemm(int64_t M, int64_t N, int64_t K, int epilogue = kEpiPlain);
// The plan for an explicit tile kind and K split (plan_gemm's choices are
// made through it; also used to compare configurations).
GemmPlan plan_gemm_as(int64_t M, int64_t N, int64_t K, int kind, int splits, int epilogue = kEpiPlain);
// Whether the kernel of tile kind `kind` can address operands with these row
// strides: the in-place-refill kernels need a tile's rows of A and of W to
// span at most 4 GiB ((BM - 1) lda + 128 and (BN - 1) ldw + 128 <= 2^32);
// the others take any stride.
bool gemm_strides_fit(int kind, int64_t lda, int64_t ldw);
// stats_mode 0: plain GEMM; 1/2: also the per-(row, column group) statistics
// of the bf16 output (softmax in base 2 with c2 = log2(e)/T, or argmax) into
// stats [M][ld_stats]; requires p.splits == 1.
hipError_t launch_gemm(const GemmPlan& p, const uint8_t* a, int64_t lda, const float* sa, int a_per_tensor,
                       const uint8_t* w, int64_t ldw, const float* sw, int w_per_tensor, int64_t M,
                       int64_t N, int64_t K, void* y, int64_t ldy, int out_f32, void* workspace,
                       hipStream_t stream, int stats_mode = 0, float c2 = 0.0f, float2* stats = nullptr,
                       int64_t ld_stats = 0, int64_t silu_inter = 0);
// SiLU-gated output: N = 2I weight rows [gate; up], y = h [M, ldy] bf16 with
// I = silu_inter columns; the plan comes from plan_gemm(M, 2I, K, kEpiSilu).

// ---- accept.hip
struct AcceptPlan {
    int64_t chunk;         // vocabulary elements per sampling workgroup
    int64_t nchunk;        // sampling chunks per row
    int64_t schunk;        // vocabulary elements per statistics item (one wave)
    int64_t nschunk;       // statistics items per row
    size_t stats_off, fine_off, ctr_off, zx_off, bytes;
};
AcceptPlan plan_accept(int64_t B, int64_t k, int64_t V);
// tstats (optional): the target rows' statistics [B*(k+1)][ld_tstats], n_tstats
// entries per row, in the form the GEMM epilogue writes for this temperature.
hipError_t launch_accept(const AcceptPlan& p, const uint16_t* zt, const uint16_t* zd, const int32_t* x,
                         const float* u, int64_t B, int64_t k, int64_t V, float temperature,
                         int32_t* out_tokens, int32_t* num_accepted, void* workspace, hipStream_t stream,
                         const float2* tstats = nullptr, int64_t n_tstats = 0, int64_t ld_tstats = 0);

// Device address of the library's fixed acceptance scratch on the current
// device (looked up once per device); kAcceptScratchBytes long.
constexpr size_t kAcceptScratchBytes = (size_t)16 << 20;
hipError_t accept_scratch(void** ptr);

// Token-tree verification (N nodes per sequence, N+1 target rows); the plan
// is plan_accept(B, N, V).
hipError_t launch_accept_tree(const AcceptPlan& p, const uint16_t* zt, const int32_t* parent, const int32_t* x,
                              const float* u, int64_t B, int64_t N, int64_t V, float temperature,
                              int32_t* out_tokens, int32_t* accepted_nodes, int32_t* num_accepted, void* workspace,
                              hipStream_t stream);

// ---- tree_mask.hip
// Ancestor-or-self masks (bit j = node j) and depths of B trees of N <= 64
// nodes, parents int32 [B][N]; mask uint64 [B][N], depth int32 [B][N].
hipError_t launch_tree_mask(const int32_t* parents, int64_t B, int64_t N, uint64_t* mask, int32_t* depth,
                            hipStream_t stream);

}  // namespace specfp8
