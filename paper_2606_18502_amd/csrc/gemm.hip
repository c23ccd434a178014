// W8A8 FP8 GEMM for gfx950: Y = (A W^T) * sa[m] * sw[n], fp32 accumulation.
//
// Operands are E4M3 bytes, both K-contiguous (A [M,K] activations, W [N,K]
// weights).  The inner product runs on the CDNA4 matrix cores:
// v_mfma_f32_16x16x128_f8f6f4 multiplies a 16x128 by a 128x16 E4M3 tile into
// 16x16 fp32 accumulators (E4M3 products are exact; the hardware accumulates
// in fp32).  W takes the instruction's "row" operand and A its "column"
// operand, so the 4 accumulators a lane holds are 4 consecutive output
// channels n of one token row m, and the epilogue writes them as one 8-byte
// (bf16) or 16-byte (fp32) store.
//
// Data movement per K-step of 128 bytes:
//  * the workgroup's A tile (BM rows) and W tile (BN rows) are copied from
//    global memory straight into LDS with global_load_lds_dwordx4 (no VGPR
//    staging): one wave instruction moves 8 rows x 128 bytes = 1 KiB;
//  * inside LDS each 128-byte row holds its eight 16-byte chunks in XOR-
//    swizzled slots (slot = chunk ^ swz(row)); the swizzle is applied on the
//    global side, so global reads stay fully coalesced, and the MFMA operand
//    reads (ds_read_b128, lane l reading logical chunk 2(l/16) + h of row
//    l % 16) put the lanes that one LDS cycle serves on distinct banks -- no
//    conflicts (see swz);
//  * STAGES buffers rotate so that STAGES-1 K-steps of loads are in flight
//    while the current one is multiplied.
//
// K is split across workgroups (split-K) when there are fewer output tiles
// than compute units.  The fp32 partial tiles are then added in split order
// (deterministic) by the last workgroup of each tile to finish (a ticket per
// tile), which then applies the epilogue.
// Workgroup ids are remapped so that the tiles and K-splits that share
// operands run on the same XCD (blocks are dealt round-robin to the 8 XCDs),
// which keeps re-read operand bytes in that XCD's L2.
//
// Epilogue variants (a template argument, so each is its own kernel):
//  0  the scaled output, bf16 or fp32 (after the split-K reduction);
//  1  bf16 logits plus per-row softmax statistics of the stored values over
//     each wave's columns (the LM head of the verify pass);
//  2  bf16 logits plus per-row (max, lowest column) over each wave's columns;
//  3  the SiLU-gated FFN output h = bf16(silu(gate) * up) from a weight tile
//     whose 16-row blocks pair 8 gate rows with the matching 8 up rows.
#include <float.h>

#include <utility>

#include "device_common.hpp"
#include "kernels.hpp"
#include "plan.hpp"

namespace specfp8 {

typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v4f __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void* lds_ptr_t;

namespace {

constexpr int kBK = kGemmBK;   // bytes (= E4M3 elements) of K per step
constexpr int kXcds = 8;

struct GemmArgs {
    const uint8_t* a;
    const uint8_t* w;
    const float* sa;
    const float* sw;
    void* y;
    uint64_t* part;   // split K: per tile and split, the threads' accumulators (two 8-byte halves each)
    unsigned int* tickets;   // split K: one per tile, zero between calls
    float2* stats;    // [M][ld_stats] column-group statistics of the bf16 output (stats_mode != 0)
    int64_t lda, ldw, ldy, ld_stats;
    int M, N, K;
    int a_per_tensor, w_per_tensor, out_f32;
    int m_tiles, n_tiles, splits, ksteps;
    int stats_mode;   // 0: none; 1: (max t, sum 2^(t - max)), t = z * c2; 2: (max z, lowest column)
    float c2;
    int silu_inter;   // > 0: SiLU-gated output of I = silu_inter columns from W = [gate; up] (N = 2I)
    int group_m;      // > 1: tiles are ordered in groups of group_m M-tiles that walk the N-tiles together
    int krot_on;      // 1: workgroups of different N-tiles start K at staggered steps
};

// Weight row of logical output column n.  With the SiLU-gated epilogue every
// 16-row block of the weight tile pairs 8 gate rows with the matching 8 up
// rows (logical block b holds gate c, up c for c = 8b .. 8b+7), so that one
// lane exchange brings each h column's gate and up accumulators together.
__device__ __forceinline__ int w_row(const GemmArgs& g, int n) {
    if (g.silu_inter == 0) return n;
    const int c = (n >> 4) * 8 + (n & 7);
    return (n & 8) ? g.silu_inter + c : c;
}

__device__ __forceinline__ int xcd_remap(int b, int total) {
    // Blocks are dealt to XCDs round-robin (block b -> XCD b % 8).  Give each
    // XCD a contiguous range of logical ids.
    const int xcd = b % kXcds, idx = b / kXcds;
    const int per = total / kXcds, rem = total % kXcds;
    return xcd * per + (xcd < rem ? xcd : rem) + idx;
}

template <int WTM, int WTN, int WM, int WN, int STAGES>
struct GemmCfg {
    static constexpr int kWaves = WM * WN;
    static constexpr int kThreads = 64 * kWaves;
    static constexpr int BM = 16 * WTM * WM;
    static constexpr int BN = 16 * WTN * WN;
    static constexpr int kRows = BM + BN;
    static constexpr int kGroups = kRows / 8;                // 1 KiB load groups per stage
    static constexpr int kGroupsPerWave = kGroups / kWaves;  // load instructions per wave and stage
    static constexpr int kStageBytes = kRows * kBK;
    static constexpr int kLdsBytes = STAGES * kStageBytes;
    static_assert(kRows % 16 == 0, "tile rows must be multiples of 16");
    static_assert(kGroups % kWaves == 0, "every wave issues the same number of loads per stage");
    static_assert((STAGES - 1) * kGroupsPerWave < 64, "vmcnt range");
    static constexpr int kKind = tile_kind_of(WTM, WTN, WM, WN, STAGES);
    static_assert(kKind >= 0, "a tile of the kind table");
    static constexpr int kReadSpan8 = kTiles[kKind].rspan8;   // schedule of a K-step (kind table)
    static constexpr int kLoadSpan8 = kTiles[kKind].lspan8;
    static_assert(kReadSpan8 >= 1 && kReadSpan8 <= 8 && kLoadSpan8 >= 1 && kLoadSpan8 <= 8, "spans in eighths");
};

// LDS swizzle.  gfx950's LDS has 64 banks of 4 bytes (256 bytes per cycle),
// so a ds_read_b128 takes at least 4 cycles, 16 lanes per cycle; the lanes
// served together are l and l + 16 for l % 16 < 8 (lanes 0-7 with 16-23,
// 8-15 with 24-31, 32-39 with 48-55, 40-47 with 56-63): a control kernel
// reading 16 contiguous bytes per lane counts no conflict, and the operand
// read counted 4 conflict cycles of 8 under a swizzle that only kept lanes
// 0-15 apart.  Rows are 128 bytes, so rows r and r^1 share a 256-byte bank
// line (their chunks land in the two halves); lanes l and l + 16 read rows
// 0-7 (or 8-15) at chunks differing by 2, so the XOR masks of the four row
// pairs must form a set F with F and F ^ 2 disjoint: F = {0, 1, 4, 5}.  Every
// cycle's 16 lanes then hit 16 different 16-byte bank groups.
__device__ __forceinline__ int swz(int row) { return (0x5410 >> (4 * ((row >> 1) & 3))) & 0xf; }

// Load group i (of kGroupsPerWave) of this wave for the stage at `stage`.
template <class C>
__device__ __forceinline__ void issue_group(const GemmArgs& g, char* stage, int m0, int n0, int64_t kbyte,
                                            int wave, int lane, int i) {
    const int r_in = lane >> 3;       // row within the 8-row group
    const int slot = lane & 7;        // LDS slot this lane fills
    const int grp = wave + i * C::kWaves;
    const int row = grp * 8 + r_in;
    const int chunk = slot ^ swz(row);   // logical 16-byte chunk loaded into it
    const uint8_t* src;
    if (row < C::BM) {
        int m = m0 + row;
        m = m < g.M ? m : g.M - 1;
        src = g.a + (int64_t)m * g.lda + kbyte + chunk * 16;
    } else {
        int n = n0 + row - C::BM;
        n = w_row(g, n < g.N ? n : g.N - 1);
        src = g.w + (int64_t)n * g.ldw + kbyte + chunk * 16;
    }
    __builtin_amdgcn_global_load_lds((const void*)src, (lds_ptr_t)(stage + grp * 1024), 16, 0, 0);
}

template <class C>
__device__ __forceinline__ void issue_stage(const GemmArgs& g, char* stage, int m0, int n0,
                                            int64_t kbyte, int wave, int lane) {
#pragma unroll
    for (int i = 0; i < C::kGroupsPerWave; ++i) issue_group<C>(g, stage, m0, n0, kbyte, wave, lane, i);
}

// Placement of the per-step work between the MFMAs of a K-step of the roll
// kernel (numerator over 8 of the step's MFMA count): the stage refill loads
// go out over the first kRollLoadSpan8/8 of the MFMAs.  (The other kernel
// takes its spans from the kind table.)
constexpr int kRollLoadSpan8 = 4;

// vmcnt(N) with lgkmcnt/expcnt left alone (vmcnt field: bits [3:0] and [15:14]).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint32_t lds_addr(const void* p) {
    return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
}

// MFMA operand of one lane: the two logical 16-byte chunks 2kg, 2kg+1 of
// `row`, each in its swizzled slot.  The LDS reads are issued as inline asm so
// that the compiler does not treat them as readers of the direct-to-LDS loads
// still in flight for other stages (it would drain them all); completion is
// awaited explicitly.
__device__ __forceinline__ u32x4 lds_half(uint32_t stage, int row, int chunk) {
    const uint32_t a = stage + (uint32_t)row * kBK + ((uint32_t)(chunk ^ swz(row)) << 4);
    u32x4 v;
    asm volatile("ds_read_b128 %0, %1" : "=v"(v) : "v"(a));
    return v;
}

__device__ __forceinline__ v8i lds_frag(uint32_t stage, int row, int kg) {
    const u32x4 lo = lds_half(stage, row, 2 * kg);
    const u32x4 hi = lds_half(stage, row, 2 * kg + 1);
    v8i r;
    r[0] = lo[0]; r[1] = lo[1]; r[2] = lo[2]; r[3] = lo[3];
    r[4] = hi[0]; r[5] = hi[1]; r[6] = hi[2]; r[7] = hi[3];
    return r;
}

// Wait until at most N LDS reads are outstanding (they complete in order);
// the fragment passes through an empty asm after the wait, so no use of it
// can be scheduled before the wait.
template <int N>
__device__ __forceinline__ void frag_ready(v8i& f) {
    static_assert(N >= 0 && N < 16, "lgkmcnt range");
    asm volatile("s_waitcnt lgkmcnt(%0)" ::"n"(N) : "memory");
    asm volatile("" : "+v"(f));
}

// Operand fragments of one K-step held in registers: WTM activation blocks
// and WTN weight blocks.
template <int WTM, int WTN>
struct Frags {
    v8i a[WTM];
    v8i w[WTN];
};

template <class C, int WTM, int WTN>
__device__ __forceinline__ void read_frags(Frags<WTM, WTN>& f, uint32_t st, int wm, int wn, int lane) {
    const int kg = lane >> 4;
    const int r16 = lane & 15;
#pragma unroll
    for (int j = 0; j < WTM; ++j) f.a[j] = lds_frag(st, (wm * WTM + j) * 16 + r16, kg);
#pragma unroll
    for (int i = 0; i < WTN; ++i) f.w[i] = lds_frag(st, C::BM + (wn * WTN + i) * 16 + r16, kg);
}

__device__ __forceinline__ void lds_wait_all() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }

// One K-step `it` on compile-time stage S with fragments `cur` (already read):
//   1. wait until the loads of step it+1 have landed (this wave), barrier (all waves);
//   2. refill stage S -- its data is already in `cur` in every wave -- with step it+STAGES;
//   3. issue the LDS reads of step it+1 into `nxt` while the MFMAs of step it run.
// Every stage is its own LDS object and every wait count is a compile-time
// constant, so the compiler does not drain the direct-to-LDS loads of other
// stages; past the end of the K range the refill re-loads the last K-step (in
// bounds, never multiplied), which keeps the number of loads in flight -- and
// so the wait -- uniform.
template <class C, int STAGES, int WTM, int WTN, int S>
__device__ __forceinline__ void kstep(const GemmArgs& g, char* const* stages, int it, int nk, int ks0, int krot,
                                      int m0, int n0, int wave, int lane, int wm, int wn, v4f (&acc)[WTN][WTM],
                                      Frags<WTM, WTN>& cur, Frags<WTM, WTN>& nxt) {
    wait_vmcnt<(STAGES - 2) * C::kGroupsPerWave>();
    __builtin_amdgcn_s_barrier();
    const int refill = min(it + STAGES, nk - 1);
    const int64_t kref = (int64_t)(ks0 + (refill + krot) % nk) * kBK;
    // MFMAs of step it, with the stage refill loads and the LDS reads of step
    // it+1 spread between them so neither queue fills and blocks MFMA issue.
    // Each group is fenced with sched_barrier to keep this order.  On the last
    // step the reads target the current stage (in bounds, results unused),
    // which keeps the sequence free of branches.
    const bool more = it + 1 < nk;
    const uint32_t st_next = lds_addr(stages[more ? (S + 1) % STAGES : S]);
    const int kg = lane >> 4;
    const int r16 = lane & 15;
    constexpr int kMfma = WTM * WTN;
    constexpr int kReads = 2 * (WTM + WTN);
    constexpr int kG = C::kGroupsPerWave;
    constexpr int kRSpan = (kMfma * C::kReadSpan8 + 7) / 8 > 0 ? (kMfma * C::kReadSpan8 + 7) / 8 : 1;
    constexpr int kLSpan = (kMfma * C::kLoadSpan8 + 7) / 8 > 0 ? (kMfma * C::kLoadSpan8 + 7) / 8 : 1;
#pragma unroll
    for (int t = 0; t < kMfma; ++t) {
        const int i = t / WTM, j = t % WTM;
#pragma unroll
        for (int q = 0; q < kG; ++q)
            if ((q * kLSpan) / kG == t) issue_group<C>(g, stages[S], m0, n0, kref, wave, lane, q);
        acc[i][j] = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(cur.w[i], cur.a[j], acc[i][j], 0, 0, 0, 0, 0, 0);
#pragma unroll
        for (int r = 0; r < kReads; ++r) {
            if ((r * kRSpan) / kReads == t) {
                const int f = r / 2, h = r & 1;
                const int row = f < WTM ? (wm * WTM + f) * 16 + r16 : C::BM + (wn * WTN + f - WTM) * 16 + r16;
                const u32x4 v = lds_half(st_next, row, 2 * kg + h);
                v8i& dst = f < WTM ? nxt.a[f] : nxt.w[f - WTM];
                dst[4 * h + 0] = v[0];
                dst[4 * h + 1] = v[1];
                dst[4 * h + 2] = v[2];
                dst[4 * h + 3] = v[3];
            }
        }
        __builtin_amdgcn_sched_barrier(0);
    }
    lds_wait_all();
#pragma unroll
    for (int j = 0; j < WTM; ++j) asm volatile("" : "+v"(nxt.a[j]));
#pragma unroll
    for (int i = 0; i < WTN; ++i) asm volatile("" : "+v"(nxt.w[i]));
}

template <int WTM, int WTN>
__device__ __forceinline__ void load_scales(const GemmArgs& g, float (&sa_reg)[WTM], float (&sw_reg)[WTN][4], int m0,
                                            int n0, int wm, int wn, int lane) {
    const int kg0 = lane >> 4, r0 = lane & 15;
#pragma unroll
    for (int j = 0; j < WTM; ++j) {
        const int m = min(m0 + (wm * WTM + j) * 16 + r0, g.M - 1);
        sa_reg[j] = g.a_per_tensor ? g.sa[0] : g.sa[m];
    }
#pragma unroll
    for (int i = 0; i < WTN; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int n = w_row(g, min(n0 + (wn * WTN + i) * 16 + 4 * kg0 + r, g.N - 1));
            sw_reg[i][r] = g.w_per_tensor ? g.sw[0] : g.sw[n];
        }
}

__device__ __forceinline__ bool beats(float v, int i, float bv, int bi) {
    return v > bv || (v == bv && i < bi);
}

// Online (max, sum 2^(t - max)) of one more value t: one exponential of
// -|t - m| per value, the running sum rescaled when the maximum moves.  The
// running max starts at the finite sentinel -FLT_MAX, so that t = -inf (a
// column past the edge) adds exactly 0 without a branch.
__device__ __forceinline__ void online_add(float& m, float& s, float t) {
    const float d = t - m;
    const float e = __builtin_amdgcn_exp2f(-fabsf(d));
    const bool up = d > 0.0f;
    s = up ? fmaf(s, e, 1.0f) : s + e;
    m = up ? t : m;
}

// Merge of two (max, sum) pairs; (-inf, 0) is the empty pair.
__device__ __forceinline__ void online_merge(float& m, float& s, float om, float os) {
    const float M = fmaxf(m, om);
    if (M == -INFINITY) return;
    s = (m == -INFINITY ? 0.0f : s * __builtin_amdgcn_exp2f(m - M)) +
        (om == -INFINITY ? 0.0f : os * __builtin_amdgcn_exp2f(om - M));
    m = M;
}

// Statistics epilogues (STATS 1: (max t, sum 2^(t - max)) of t = fl32(z *
// c2); STATS 2: (max z, lowest column)) of the bf16 values a lane stores, per
// row block j of its wave tile: start values, then 4 consecutive columns
// n..n+3 at a time (a lane visits its columns in increasing order, so a
// strict comparison keeps the lowest column of a tie; columns past the edge
// count as absent).
template <int WTM, int STATS>
__device__ __forceinline__ void stats_init(float (&sm)[WTM], float (&ss)[WTM]) {
#pragma unroll
    for (int j = 0; j < WTM; ++j) {
        sm[j] = STATS == 1 ? -FLT_MAX : -INFINITY;
        ss[j] = STATS == 2 ? __int_as_float(0x7fffffff) : 0.0f;
    }
}

template <int STATS, bool EDGE>
__device__ __forceinline__ void stats_add4(const GemmArgs& g, const uint32_t (&bits)[4], int n, float& sm, float& ss) {
    if constexpr (STATS == 1) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const float t = bf16_to_f32(bits[r]) * g.c2;
            online_add(sm, ss, (!EDGE || n + r < g.N) ? t : -INFINITY);
        }
    } else if constexpr (STATS == 2) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const float z = bf16_to_f32(bits[r]);
            const bool gt = (!EDGE || n + r < g.N) && z > sm;
            sm = gt ? z : sm;
            ss = gt ? __int_as_float(n + r) : ss;
        }
    }
}

// The 4 lanes r16 + 16 kg that share a row combine their statistics by two
// xor shuffles in a fixed order; lane kg = 0 stores the row's entry of
// column group `col` (rows from mrow0 + 16 j + r16).  Empty groups store
// (-inf, 0) (STATS 1) or (-inf, INT_MAX bits) (STATS 2).
template <int WTM, int STATS>
__device__ __forceinline__ void stats_store(const GemmArgs& g, const float (&sm)[WTM], const float (&ss)[WTM], int mrow0,
                                            int lane, int64_t col) {
    const int kg = lane >> 4;
    const int r16 = lane & 15;
#pragma unroll
    for (int j = 0; j < WTM; ++j) {
        float m1 = sm[j], s1 = ss[j];
        if (STATS == 1 && m1 == -FLT_MAX) m1 = -INFINITY;      // no column of this group in this lane
#pragma unroll
        for (int o = 16; o <= 32; o <<= 1) {
            const float m2 = __shfl_xor(m1, o, 64);
            const float s2 = __shfl_xor(s1, o, 64);
            if (STATS == 2) {
                if (beats(m2, __float_as_int(s2), m1, __float_as_int(s1))) { m1 = m2; s1 = s2; }
            } else {
                online_merge(m1, s1, m2, s2);
            }
        }
        const int m = mrow0 + j * 16 + r16;
        if (kg == 0 && m < g.M) g.stats[(int64_t)m * g.ld_stats + col] = make_float2(m1, s1);
    }
}

// The 16x16 blocks of one wave's tile.  EDGE: the tile crosses the last row
// or column, so every store (and every statistic) is bounds-checked.
template <int WTM, int WTN, int STATS, bool EDGE>
__device__ __forceinline__ void store_blocks(const GemmArgs& g, const v4f (&acc)[WTN][WTM],
                                             const float (&sa_reg)[WTM], const float (&sw_reg)[WTN][4], int m0,
                                             int n0, int wm, int wn, int lane, float (&sm)[WTM], float (&ss)[WTM]) {
    const int kg = lane >> 4;
    const int r16 = lane & 15;
    if (STATS == 0 && g.out_f32) {
#pragma unroll
        for (int j = 0; j < WTM; ++j) {
            const int m = m0 + (wm * WTM + j) * 16 + r16;
            float* row = reinterpret_cast<float*>(g.y) + (int64_t)m * g.ldy;
#pragma unroll
            for (int i = 0; i < WTN; ++i) {
                const int n = n0 + (wn * WTN + i) * 16 + 4 * kg;
                float y[4];
#pragma unroll
                for (int r = 0; r < 4; ++r) y[r] = (acc[i][j][r] * sa_reg[j]) * sw_reg[i][r];
                if (!EDGE || n + 3 < g.N) {
                    if (!EDGE || m < g.M) *reinterpret_cast<float4*>(row + n) = make_float4(y[0], y[1], y[2], y[3]);
                } else if (m < g.M) {
                    for (int r = 0; r < 4 && n + r < g.N; ++r) row[n + r] = y[r];
                }
            }
        }
        return;
    }
#pragma unroll
    for (int j = 0; j < WTM; ++j) {
        const int m = m0 + (wm * WTM + j) * 16 + r16;
        uint16_t* row = reinterpret_cast<uint16_t*>(g.y) + (int64_t)m * g.ldy;
#pragma unroll
        for (int i = 0; i < WTN; ++i) {
            const int n = n0 + (wn * WTN + i) * 16 + 4 * kg;
            uint32_t bits[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) bits[r] = f32_to_bf16_rne((acc[i][j][r] * sa_reg[j]) * sw_reg[i][r]);
            if constexpr (STATS == 3) {
                // lanes 16 kg + r16 with kg < 2 hold the gate of h columns
                // (n - n0') / 2 + 4 kg + r (n0' = the block's first logical
                // column), lanes with kg >= 2 the matching up values
                float h[4];
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const float y = bf16_to_f32(bits[r]);
                    const float other = __shfl_xor(y, 32, 64);
                    h[r] = silu_mul_bf16(y, other);
                }
                const int hc = (n0 + (wn * WTN + i) * 16) / 2 + 4 * kg;    // first h column of this lane
                if (kg < 2 && (!EDGE || (m < g.M && hc < g.silu_inter))) {
                    uint16_t* hrow = reinterpret_cast<uint16_t*>(g.y) + (int64_t)m * g.ldy;
                    uint2 o;
                    o.x = (__float_as_uint(h[0]) >> 16) | (__float_as_uint(h[1]) & 0xffff0000u);
                    o.y = (__float_as_uint(h[2]) >> 16) | (__float_as_uint(h[3]) & 0xffff0000u);
                    *reinterpret_cast<uint2*>(hrow + hc) = o;
                }
                continue;
            }
            stats_add4<STATS, EDGE>(g, bits, n, sm[j], ss[j]);
            if (!EDGE || n + 3 < g.N) {
                if (!EDGE || m < g.M) {
                    uint2 o;
                    o.x = bits[0] | (bits[1] << 16);
                    o.y = bits[2] | (bits[3] << 16);
                    *reinterpret_cast<uint2*>(row + n) = o;
                }
            } else if (m < g.M) {
                for (int r = 0; r < 4 && n + r < g.N; ++r) row[n + r] = (uint16_t)bits[r];
            }
        }
    }
}

// Epilogue: lane holds D[n = 4*(lane/16) + r][m = lane%16] of each 16x16
// block; the scales were fetched into registers before the main loop.  Tiles
// wholly inside the output take the unchecked path.
//
// STATS 3 (SiLU-gated output, no K split): the tile's weight rows pair gate
// and up rows (w_row), and each lane pair kg, kg ^ 2 of a block exchanges its
// bf16-rounded values, so lanes kg < 2 store h = bf16(silu(gate) * up) for 4
// consecutive h columns: exactly what the bf16 output followed by the
// SiLU-gated quantize's input step gives for the same accumulators.
//
// STATS 1, 2 (bf16 output, no K split): the statistics of the stored values of
// each row over the columns this wave holds (column group nt * WN + wn), for
// the acceptance test of the logits: STATS 1 keeps (max t, sum 2^(t - max))
// of t = fl32(z * c2) online while the row's values are stored; STATS 2 keeps
// (max z, lowest column).  The 4 lanes r16 + 16 kg that share a row are then
// combined by two xor shuffles in a fixed order.  Empty groups store (-inf,
// 0) (STATS 1) or (-inf, INT_MAX bits) (STATS 2).
template <int WTM, int WTN, int WN, int STATS>
__device__ __forceinline__ void store_tile(const GemmArgs& g, const v4f (&acc)[WTN][WTM], const float (&sa_reg)[WTM],
                                           const float (&sw_reg)[WTN][4], int m0, int n0, int wm, int wn, int lane,
                                           int nt, int BM, int BN) {
    float sm[WTM], ss[WTM];      // STATS 1: running max and sum; STATS 2: best value and (int bits) its column
    stats_init<WTM, STATS>(sm, ss);
    if (m0 + BM <= g.M && n0 + BN <= g.N)
        store_blocks<WTM, WTN, STATS, false>(g, acc, sa_reg, sw_reg, m0, n0, wm, wn, lane, sm, ss);
    else
        store_blocks<WTM, WTN, STATS, true>(g, acc, sa_reg, sw_reg, m0, n0, wm, wn, lane, sm, ss);
    if constexpr (STATS == 1 || STATS == 2)
        stats_store<WTM, STATS>(g, sm, ss, m0 + wm * WTM * 16, lane, (int64_t)nt * WN + wn);
}

__device__ __forceinline__ uint64_t pack2(float lo, float hi) {
    return ((uint64_t)__float_as_uint(hi) << 32) | (uint64_t)__float_as_uint(lo);
}

// Split-K reduced in the kernel.  Every workgroup of a split
// tile stores its fp32 partial tile with device-coherent stores (relaxed
// agent-scope atomics: written through the non-coherent caches, so a
// workgroup on any XCD reads them), waits until all of them are
// acknowledged, then takes the tile's ticket.  The workgroup that takes the
// last ticket -- every other partial is then already acknowledged -- reloads
// them with device-coherent loads issued after the ticket returned, and adds
// all of them in split order, its own from registers, so the sums do not
// depend on which workgroup arrives last.  It returns the ticket to zero for
// the next call.  Each thread stores and reloads exactly the accumulators it
// holds (one float4 per 16x16 block, as two 8-byte halves in separate
// 512-byte rows, so every store and load instruction of a wave is contiguous).
// Returns false in the workgroups that are not last (they are done).
template <int WTM, int WTN, int NT>
__device__ __forceinline__ bool reduce_last(const GemmArgs& g, v4f (&acc)[WTN][WTM], int tile, int split, int tid,
                                            int* s_flag) {
    constexpr int kBlocks = WTM * WTN;
    uint64_t* const base = g.part + (size_t)tile * g.splits * kBlocks * 2 * NT;
    {
        uint64_t* const mine = base + (size_t)split * kBlocks * 2 * NT + tid;
#pragma unroll
        for (int i = 0; i < WTN; ++i)
#pragma unroll
            for (int j = 0; j < WTM; ++j) {
                uint64_t* p = mine + (size_t)(i * WTM + j) * 2 * NT;
                __hip_atomic_store(p, pack2(acc[i][j][0], acc[i][j][1]), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                __hip_atomic_store(p + NT, pack2(acc[i][j][2], acc[i][j][3]), __ATOMIC_RELAXED,
                                   __HIP_MEMORY_SCOPE_AGENT);
            }
    }
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    if (tid == 0) {
        const unsigned int t = __hip_atomic_fetch_add(g.tickets + tile, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        const int last = t == (unsigned int)(g.splits - 1);
        if (last) __hip_atomic_store(g.tickets + tile, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        *s_flag = last;
    }
    __syncthreads();
    if (!*s_flag) return false;
    v4f tot[WTN][WTM];
    for (int z = 0; z < g.splits; ++z) {
        v4f part[WTN][WTM];
        if (z == split) {
#pragma unroll
            for (int i = 0; i < WTN; ++i)
#pragma unroll
                for (int j = 0; j < WTM; ++j) part[i][j] = acc[i][j];
        } else {
            const uint64_t* src = base + (size_t)z * kBlocks * 2 * NT + tid;
            uint64_t lo[WTN][WTM], hi[WTN][WTM];
#pragma unroll
            for (int i = 0; i < WTN; ++i)
#pragma unroll
                for (int j = 0; j < WTM; ++j) {
                    const uint64_t* p = src + (size_t)(i * WTM + j) * 2 * NT;
                    lo[i][j] = __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    hi[i][j] = __hip_atomic_load(p + NT, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                }
#pragma unroll
            for (int i = 0; i < WTN; ++i)
#pragma unroll
                for (int j = 0; j < WTM; ++j)
                    part[i][j] = v4f{__uint_as_float((uint32_t)lo[i][j]), __uint_as_float((uint32_t)(lo[i][j] >> 32)),
                                     __uint_as_float((uint32_t)hi[i][j]), __uint_as_float((uint32_t)(hi[i][j] >> 32))};
        }
#pragma unroll
        for (int i = 0; i < WTN; ++i)
#pragma unroll
            for (int j = 0; j < WTM; ++j) tot[i][j] = z == 0 ? part[i][j] : tot[i][j] + part[i][j];
    }
#pragma unroll
    for (int i = 0; i < WTN; ++i)
#pragma unroll
        for (int j = 0; j < WTM; ++j) acc[i][j] = tot[i][j];
    return true;
}

template <int WTM, int WTN, int WM, int WN, int STAGES, int STATS, bool REDUCE_LAST>
__global__ __launch_bounds__(64 * WM * WN) void gemm_fp8_kernel(GemmArgs g) {
    using C = GemmCfg<WTM, WTN, WM, WN, STAGES>;
    static_assert(STAGES >= 2 && STAGES <= 4, "2..4 stages");
    __shared__ __attribute__((aligned(1024))) char lds0[C::kStageBytes];
    __shared__ __attribute__((aligned(1024))) char lds1[C::kStageBytes];
    __shared__ __attribute__((aligned(1024))) char lds2[STAGES > 2 ? C::kStageBytes : 16];
    __shared__ __attribute__((aligned(1024))) char lds3[STAGES > 3 ? C::kStageBytes : 16];
    char* const stages[4] = {lds0, lds1, lds2, lds3};

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = wave % WM;
    const int wn = wave / WM;

    const int total = g.m_tiles * g.n_tiles * g.splits;
    const int logical = xcd_remap(blockIdx.x, total);
    // consecutive logical ids: K-splits of a tile, then M-tiles of an N-tile
    const int split = logical % g.splits;
    const int tile = logical / g.splits;
    int mt, nt;
    if (g.group_m > 1) {
        // Large M: a group of group_m M-tiles walks the N-tiles, so the tiles
        // that run at once on one XCD form a group_m x (CUs / group_m) block
        // and re-read each other's operand rows from that XCD's L2.
        const int per_group = g.group_m * g.n_tiles;
        const int first = (tile / per_group) * g.group_m;
        const int gm = min(g.group_m, g.m_tiles - first);
        const int in = tile - (tile / per_group) * per_group;
        mt = first + in % gm;
        nt = in / gm;
    } else {
        mt = tile % g.m_tiles;
        nt = tile / g.m_tiles;
    }
    const int m0 = mt * C::BM;
    const int n0 = nt * C::BN;

    const int ks_per = (g.ksteps + g.splits - 1) / g.splits;
    const int ks0 = split * ks_per;
    const int ks1 = min(g.ksteps, ks0 + ks_per);
    const int nk = ks1 - ks0;
    // Workgroups that share an activation tile walk K from different
    // starting points, so they do not all request the same bytes at once.
    const int krot = g.krot_on ? (nt * 7 + split) % nk : 0;

    v4f acc[WTN][WTM];
#pragma unroll
    for (int i = 0; i < WTN; ++i)
#pragma unroll
        for (int j = 0; j < WTM; ++j) acc[i][j] = v4f{0.f, 0.f, 0.f, 0.f};

    // prologue: all STAGES stages in flight, then the fragments of step 0
#pragma unroll
    for (int s = 0; s < STAGES; ++s)
        issue_stage<C>(g, stages[s], m0, n0, (int64_t)(ks0 + (min(s, nk - 1) + krot) % nk) * kBK, wave, lane);
    // The epilogue's scales, fetched now so their latency hides behind the
    // main loop (rows and columns past the edge read a valid neighbour).
    float sa_reg[WTM];
    float sw_reg[WTN][4];
    load_scales<WTM, WTN>(g, sa_reg, sw_reg, m0, n0, wm, wn, lane);
    Frags<WTM, WTN> f0, f1;
    wait_vmcnt<(STAGES - 1) * C::kGroupsPerWave>();
    __builtin_amdgcn_s_barrier();
    read_frags<C>(f0, lds_addr(stages[0]), wm, wn, lane);
    lds_wait_all();
#pragma unroll
    for (int j = 0; j < WTM; ++j) asm volatile("" : "+v"(f0.a[j]));
#pragma unroll
    for (int i = 0; i < WTN; ++i) asm volatile("" : "+v"(f0.w[i]));

    // the loop body covers lcm(STAGES, 2) steps so that both the stage and the
    // register set of every step are compile-time constants
#define SPEC_STEP(S, CUR, NXT)                                                                              \
    if (base + (S) < nk)                                                                                    \
        kstep<C, STAGES, WTM, WTN, (S) % STAGES>(g, stages, base + (S), nk, ks0, krot, m0, n0, wave, lane, wm, \
                                                 wn, acc, CUR, NXT);
    constexpr int U = (STAGES % 2 == 0) ? STAGES : 2 * STAGES;
    static_assert(U <= 8, "the loop body below spells out at most 8 steps");
    for (int base = 0; base < nk; base += U) {
        SPEC_STEP(0, f0, f1)
        SPEC_STEP(1, f1, f0)
        if constexpr (U > 2) {
            SPEC_STEP(2, f0, f1)
            SPEC_STEP(3, f1, f0)
        }
        if constexpr (U > 4) {
            SPEC_STEP(4, f0, f1)
            SPEC_STEP(5, f1, f0)
        }
        if constexpr (U > 6) {
            SPEC_STEP(6, f0, f1)
            SPEC_STEP(7, f1, f0)
        }
    }
#undef SPEC_STEP
    wait_vmcnt<0>();   // no direct-to-LDS write may outlive the workgroup

    if constexpr (STATS == 0 && REDUCE_LAST) {
        if (g.splits > 1) {
            __shared__ int s_last;
            if (!reduce_last<WTM, WTN, C::kThreads>(g, acc, tile, split, tid, &s_last)) return;
        }
    }
    store_tile<WTM, WTN, WN, STATS>(g, acc, sa_reg, sw_reg, m0, n0, wm, wn, lane, nt, C::BM, C::BN);
}

// ---- long prompts: 256-wide tiles, operand fragments refilled in place ------
//
// At large M every CU runs several tiles, and its time follows the operand
// bytes it streams (its data path, not its matrix cores, sets the pace).  A
// 256x224 or 256x256 tile (2x2 waves of 128x112 or 128x128) streams 22-27%
// fewer operand bytes per output than 160x224.  Its 224-256 accumulators per
// lane leave no room for a second set of operand fragments, so each fragment
// is refilled with the next K-step's data as soon as its last MFMA of the
// current step has issued: the MFMAs run W-block-major, so a W fragment dies
// after its WTM MFMAs and the A fragments during the last W block.  Two LDS
// stages (60 or 64 KiB): the loads of step it+2 go out while step it
// multiplies.  The loads take the uniform-base form: the K-step's base
// addresses are scalars and each lane keeps one 32-bit offset per load group
// for the whole K loop (the plan takes this kernel only when M * lda and
// N * ldw fit in 32 bits).
constexpr int kRollDelay = 2;   // MFMAs between a fragment's last use and its refill

template <int WTM, int WTN>
struct RollCfg {
    static constexpr int kThreads = 256;                  // 2 x 2 waves
    static constexpr int BM = 32 * WTM;
    static constexpr int BN = 32 * WTN;
    static constexpr int kRows = BM + BN;
    static constexpr int kGroupsPerWave = kRows / 32;     // 8-row (1 KiB) load groups per wave and stage
    static constexpr int kStageBytes = kRows * kBK;
    // group q of wave w covers rows 8 (w + 4 q) ..: activation rows for q < WTM
    static_assert(BM / 8 == 4 * WTM, "the first WTM groups of every wave load A");
};

// Load group q of this wave for a stage: the group's 8 rows x 128 bytes go
// from base + off (base: the K-step's first byte of A or W, a scalar; off:
// this lane's row and chunk) to LDS at m0 = the group's 1 KiB.  Written as
// inline asm to get the scalar-base form; the issuing code waits for it with
// explicit vmcnt waits.
__device__ __forceinline__ void roll_load(const uint8_t* base, uint32_t off, uint32_t lds) {
    asm volatile("s_nop 0\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(off), "s"(base), "{m0}"(lds) : "memory");
}

// ds_read_b128 at vaddr + OFF (OFF < 64 KiB, an immediate).
template <int OFF>
__device__ __forceinline__ u32x4 lds_read_imm(uint32_t vaddr) {
    static_assert(OFF >= 0 && OFF < 65536, "ds offset range");
    u32x4 v;
    asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(v) : "v"(vaddr), "n"(OFF));
    return v;
}

// The 16x16 operand block b (16 rows from the wave's first row of A or W, plus
// 16 b) of this lane: row r16 = lane % 16 of the block, logical chunks
// 2 kg, 2 kg + 1 (kg = lane / 16).  All blocks of a wave share the row bits
// that decide the swizzle, so each lane's two addresses are fixed per stage
// (base[0], base[1]) and the block is an immediate offset of 16 rows x 128.
template <int B>
__device__ __forceinline__ v8i roll_frag(const uint32_t (&base)[2]) {
    const u32x4 lo = lds_read_imm<B * 2048>(base[0]);
    const u32x4 hi = lds_read_imm<B * 2048>(base[1]);
    return __builtin_bit_cast(v8i, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
}

template <int WTM, int WTN, int N>
struct RollRead {
    // fragment N of the step order: W blocks 0 .. WTN-1, then A blocks
    __device__ __forceinline__ static void run(Frags<WTM, WTN>& f, const uint32_t (&wb)[2], const uint32_t (&ab)[2]) {
        if constexpr (N < WTN) f.w[N] = roll_frag<N>(wb);
        else f.a[N - WTN] = roll_frag<N - WTN>(ab);
    }
};

// f(std::integral_constant<int, I>{}) for I = 0 .. N-1, in order, each I a
// compile-time constant (an immediate LDS offset, a fragment index).
template <class F, int... I>
__device__ __forceinline__ void static_for_seq(F&& f, std::integer_sequence<int, I...>) {
    (f(std::integral_constant<int, I>{}), ...);
}
template <int N, class F>
__device__ __forceinline__ void static_for(F&& f) {
    static_for_seq(f, std::make_integer_sequence<int, N>{});
}

// One K-step `it` on stage S.  LOADS: refill stage S with step it+2 (there is
// one); NEXT: refill the fragments with step it+1 (there is one).  ab/wb: this
// lane's A and W read bases in stage S ^ 1.
template <class R, int WTM, int WTN, int S, bool LOADS, bool NEXT>
__device__ __forceinline__ void roll_step(const uint8_t* a0, const uint8_t* w0, int it, int nk, int krot,
                                          const uint32_t (&off)[R::kGroupsPerWave], uint32_t lds_stage,
                                          const uint32_t (&ab)[2], const uint32_t (&wb)[2], v4f (&acc)[WTN][WTM],
                                          Frags<WTM, WTN>& f) {
    wait_vmcnt<0>();                      // step it+1 has landed (this wave's loads) ...
    __builtin_amdgcn_s_barrier();         // ... and every wave's; every wave has read step it from stage S
    const int64_t kref = (int64_t)((it + 2 + krot) % nk) * kBK;
    const uint8_t* abase = a0 + kref;
    const uint8_t* wbase = w0 + kref;
    constexpr int kMfma = WTM * WTN;
    constexpr int kG = R::kGroupsPerWave;
    constexpr int kLSpan = (kMfma * kRollLoadSpan8 + 7) / 8;
    // refill order: W block i after its last MFMA (i WTM + WTM - 1), A block j
    // after its last one ((WTN - 1) WTM + j), each kRollDelay MFMAs later
    auto refill = [&](auto td_c) {
        constexpr int td = decltype(td_c)::value;
        if constexpr (td % WTM == WTM - 1 && td / WTM < WTN - 1) RollRead<WTM, WTN, td / WTM>::run(f, wb, ab);
        if constexpr (td >= (WTN - 1) * WTM) RollRead<WTM, WTN, WTN + td - (WTN - 1) * WTM>::run(f, wb, ab);
    };
    static_for<kMfma>([&](auto tc) {
        constexpr int t = decltype(tc)::value;
        constexpr int i = t / WTM, j = t % WTM;
        if constexpr (LOADS) {
            static_for<kG>([&](auto qc) {
                constexpr int q = decltype(qc)::value;
                if constexpr ((q * kLSpan) / kG == t) roll_load(q < WTM ? abase : wbase, off[q], lds_stage + q * 4096);
            });
        }
        acc[i][j] = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(f.w[i], f.a[j], acc[i][j], 0, 0, 0, 0, 0, 0);
        if constexpr (NEXT && t >= kRollDelay) refill(std::integral_constant<int, t - kRollDelay>{});
        __builtin_amdgcn_sched_barrier(0);
    });
    if constexpr (NEXT) {
        // the fragments whose last MFMAs issued just now (wait states first,
        // so that those MFMAs have read their operands)
        asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7\n\ts_nop 7" ::: "memory");
        static_for<kRollDelay>([&](auto dc) { refill(std::integral_constant<int, kMfma - kRollDelay + decltype(dc)::value>{}); });
        RollRead<WTM, WTN, WTN - 1>::run(f, wb, ab);
        lds_wait_all();
#pragma unroll
        for (int j = 0; j < WTM; ++j) asm volatile("" : "+v"(f.a[j]));
#pragma unroll
        for (int i = 0; i < WTN; ++i) asm volatile("" : "+v"(f.w[i]));
    }
}

// fp32 epilogue of the in-place-refill tiles (never split): W block by W
// block, each block's 4 weight scales per lane loaded just before use, so
// that few registers besides the accumulators are live.  The arithmetic is
// store_blocks': y = fl32(fl32(acc * sa) * sw).
template <int WTM, int WTN, bool EDGE>
__device__ __forceinline__ void roll_store_f32(const GemmArgs& g, const v4f (&acc)[WTN][WTM],
                                               const float (&sa_reg)[WTM], int m0, int n0, int wm, int wn, int lane) {
    const int kg = lane >> 4;
    const int r16 = lane & 15;
#pragma unroll
    for (int i = 0; i < WTN; ++i) {
        const int n = n0 + (wn * WTN + i) * 16 + 4 * kg;
        float sw[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) sw[r] = g.w_per_tensor ? g.sw[0] : g.sw[min(n + r, g.N - 1)];
#pragma unroll
        for (int j = 0; j < WTM; ++j) {
            const int m = m0 + (wm * WTM + j) * 16 + r16;
            if (EDGE && m >= g.M) continue;
            float y[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) y[r] = (acc[i][j][r] * sa_reg[j]) * sw[r];
            float* row = reinterpret_cast<float*>(g.y) + (int64_t)m * g.ldy;
            if (!EDGE || n + 3 < g.N) *reinterpret_cast<float4*>(row + n) = make_float4(y[0], y[1], y[2], y[3]);
            else
                for (int r = 0; r < 4 && n + r < g.N; ++r) row[n + r] = y[r];
        }
    }
}

// bf16 epilogue of the in-place-refill tiles through LDS: each wave puts its
// 16 WTM x 16 WTN bf16 block into LDS (y = fl32(fl32(acc * sa) * sw), then
// RNE), then writes it out row by row with 16-byte stores, so every row
// segment leaves the CU as whole cache lines at once.  (Written from the MFMA
// layout directly, a row's line is filled 32 bytes at a time across the whole
// epilogue and can be evicted, and written back, several times while the
// other workgroups of the XCD stream their operands.)  LDS rows of 256 bytes
// (the staging then fills both stages exactly) swap their 16-byte chunks by
// row; other rows get a 16-byte pad; either way the 8-byte writes of a wave
// and the 16-byte reads hit distinct banks.  The caller has passed a
// workgroup barrier after the K loop, so no stage is still read.  EDGE: the
// tile crosses the last row or column: weight scales are read clamped, and
// rows >= M and columns >= N are neither stored nor counted.
//
// STATS 1, 2 (the LM head): after its stores, every lane reads back from LDS
// the 4 WTN consecutive columns kg * 4 WTN ... of row 16 j + r16 of its wave
// block, for every row block j, and forms their statistics: STATS 1 the
// maximum t = fl32(z * c2) first, then the sum of 2^(t - max); STATS 2 the
// maximum z and its lowest column (columns visited in increasing order, a
// strict comparison).  stats_store then combines the 4 lanes of a row, so
// each wave writes the statistics of its 16 WTN columns (one column group).
template <int WTM, int WTN, int STATS, bool EDGE>
__device__ __forceinline__ void roll_store_lds(const GemmArgs& g, const v4f (&acc)[WTN][WTM], const float (&sa_reg)[WTM],
                                               int m0, int n0, int wm, int wn, int wave, int lane, char* lds,
                                               int64_t col_group) {
    constexpr int kRowBytes = 32 * WTN;                   // 16 WTN bf16 columns
    constexpr bool kSwap = kRowBytes == 256;
    constexpr int kPitch = kSwap ? 256 : kRowBytes + 16;
    constexpr int kRows = 16 * WTM;                       // rows per wave
    static_assert(4 * kRows * kPitch <= 2 * RollCfg<WTM, WTN>::kStageBytes, "staging fits the two stages");
    auto at = [](int row, int byte) {
        return (uint32_t)(row * kPitch + (kSwap ? ((((byte >> 4) ^ (row & 15)) << 4) | (byte & 15)) : byte));
    };
    const int kg = lane >> 4;
    const int r16 = lane & 15;
    const uint32_t base = lds_addr(lds) + (uint32_t)(wave * kRows * kPitch);
#pragma unroll
    for (int i = 0; i < WTN; ++i) {
        const int n = n0 + (wn * WTN + i) * 16 + 4 * kg;
        float sw[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) sw[r] = g.w_per_tensor ? g.sw[0] : g.sw[EDGE ? min(n + r, g.N - 1) : n + r];
#pragma unroll
        for (int j = 0; j < WTM; ++j) {
            uint32_t bits[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) bits[r] = f32_to_bf16_rne((acc[i][j][r] * sa_reg[j]) * sw[r]);
            const uint32_t a = base + at(j * 16 + r16, i * 32 + kg * 8);
            const uint32_t lo = bits[0] | (bits[1] << 16), hi = bits[2] | (bits[3] << 16);
            asm volatile("ds_write_b64 %0, %1" ::"v"(a), "v"((uint64_t)lo | ((uint64_t)hi << 32)) : "memory");
        }
    }
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");   // this wave's block is in LDS (only it reads it back)
    constexpr int kChunks = kRowBytes / 16;                // 16-byte chunks per row
    const int64_t row0 = m0 + wm * kRows;
    const int col0 = n0 + wn * WTN * 16;
    // one 16-byte chunk of 8 columns: whole, or (EDGE) the columns below N.
    // Where a wave's row segments are whole 128-byte lines (256 and 384
    // bytes: the 256x256 and 160x384 tiles), whole chunks are stored
    // nontemporally: the output (82 MB of logits for an LM head) would
    // otherwise be allocated in, and written back through, the caches the
    // operand streams use (LM head 221 -> 216 us, with statistics 225 ->
    // 218 us; the acceptance that reads the logits next measured the same,
    // its greedy argmax pass 1.6 us slower).  The 224-byte segments of the
    // 256x224 tile start mid-line; stored nontemporally, the lines they share
    // were written 1.15 times, so they are stored normally.
    constexpr bool kNontemporal = kRowBytes % 128 == 0;
    auto put = [&](int c, const u32x4& v) {
        const int64_t m = row0 + c / kChunks;
        const int n = col0 + (c % kChunks) * 8;
        uint16_t* dst = reinterpret_cast<uint16_t*>(g.y) + m * g.ldy + n;
        if (!EDGE || (m < g.M && n + 7 < g.N)) {
            if constexpr (kNontemporal) __builtin_nontemporal_store(v, reinterpret_cast<u32x4*>(dst));
            else *reinterpret_cast<u32x4*>(dst) = v;
        } else if (m < g.M) {
            const uint32_t w[4] = {v[0], v[1], v[2], v[3]};
            for (int e = 0; e < 8 && n + e < g.N; ++e) dst[e] = (uint16_t)(w[e >> 1] >> (16 * (e & 1)));
        }
    };
    constexpr int kPerLane = kRows * kChunks / 64;         // chunks per lane, 4 at a time
    static_assert(kRows * kChunks % 64 == 0, "chunks per lane");
    constexpr int kFull = kPerLane / 4 * 4;
#pragma unroll 1
    for (int k0 = 0; k0 < kFull; k0 += 4) {
        u32x4 v[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int c = (k0 + u) * 64 + lane;
            asm volatile("ds_read_b128 %0, %1" : "=v"(v[u]) : "v"(base + at(c / kChunks, (c % kChunks) * 16)));
        }
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
#pragma unroll
        for (int u = 0; u < 4; ++u) asm volatile("" : "+v"(v[u]));   // no use moves above the wait
#pragma unroll
        for (int u = 0; u < 4; ++u) put((k0 + u) * 64 + lane, v[u]);
    }
#pragma unroll
    for (int k = kFull; k < kPerLane; ++k) {
        const int c = k * 64 + lane;
        u32x4 v;
        asm volatile("ds_read_b128 %0, %1" : "=v"(v) : "v"(base + at(c / kChunks, (c % kChunks) * 16)));
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
        asm volatile("" : "+v"(v));
        put(c, v);
    }
    if constexpr (STATS == 1 || STATS == 2) {
        static_assert(WTN % 2 == 0, "a lane's columns are whole 16-byte chunks");
        constexpr int kLaneCols = 4 * WTN;
        constexpr int kLaneChunks = kLaneCols / 8;
        const int c0 = col0 + kg * kLaneCols;              // this lane's first column
        float sm[WTM], ss[WTM];
#pragma unroll 1
        for (int j = 0; j < WTM; ++j) {
            u32x4 v[kLaneChunks];
#pragma unroll
            for (int q = 0; q < kLaneChunks; ++q)
                asm volatile("ds_read_b128 %0, %1"
                             : "=v"(v[q])
                             : "v"(base + at(j * 16 + r16, kg * kLaneCols * 2 + q * 16)));
            asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
            // the values are read only now: no use may move above the wait
#pragma unroll
            for (int q = 0; q < kLaneChunks; ++q) asm volatile("" : "+v"(v[q]));
            auto z_of = [&](int q, int e) {
                return __uint_as_float(((e & 1) ? v[q][e >> 1] : v[q][e >> 1] << 16) & 0xffff0000u);
            };
            if constexpr (STATS == 1) {
                float zmax = -INFINITY;
#pragma unroll
                for (int q = 0; q < kLaneChunks; ++q)
#pragma unroll
                    for (int e = 0; e < 8; ++e)
                        if (!EDGE || c0 + q * 8 + e < g.N) zmax = fmaxf(zmax, z_of(q, e));
                const float M = zmax * g.c2;                 // = max t (c2 > 0; rounding is monotone)
                float s = 0.0f;
                if (zmax != -INFINITY) {
#pragma unroll
                    for (int q = 0; q < kLaneChunks; ++q)
#pragma unroll
                        for (int e = 0; e < 8; ++e)
                            if (!EDGE || c0 + q * 8 + e < g.N)
                                s += __builtin_amdgcn_exp2f(z_of(q, e) * g.c2 - M);
                }
                sm[j] = M;
                ss[j] = s;
            } else {
                float best = -INFINITY;
                int bi = 0x7fffffff;
#pragma unroll
                for (int q = 0; q < kLaneChunks; ++q)
#pragma unroll
                    for (int e = 0; e < 8; ++e) {
                        const float z = z_of(q, e);
                        const bool gt = (!EDGE || c0 + q * 8 + e < g.N) && z > best;
                        best = gt ? z : best;
                        bi = gt ? c0 + q * 8 + e : bi;
                    }
                sm[j] = best;
                ss[j] = __int_as_float(bi);
            }
        }
        stats_store<WTM, STATS>(g, sm, ss, (int)row0, lane, col_group);
    }
}

// STATS 1, 2: the statistics epilogue of the LM head (bf16 logits plus their
// per-(row, wave column group) statistics, as gemm_fp8_kernel's), with the
// same logits as STATS 0.
template <int WTM, int WTN, int STATS>
__global__ __launch_bounds__(256) void gemm_fp8_roll_kernel(GemmArgs g) {
    using R = RollCfg<WTM, WTN>;
    __shared__ __attribute__((aligned(1024))) char lds[2 * R::kStageBytes];   // two stages; the epilogue's staging
    char* const lds0 = lds;
    char* const lds1 = lds + R::kStageBytes;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave % 2;
    const int wn = wave / 2;

    const int total = g.m_tiles * g.n_tiles;
    const int tile = xcd_remap(blockIdx.x, total);
    int mt, nt;
    if (g.group_m > 1) {
        const int per_group = g.group_m * g.n_tiles;
        const int first = (tile / per_group) * g.group_m;
        const int gm = min(g.group_m, g.m_tiles - first);
        const int in = tile - (tile / per_group) * per_group;
        mt = first + in % gm;
        nt = in / gm;
    } else {
        mt = tile % g.m_tiles;
        nt = tile / g.m_tiles;
    }
    const int m0 = mt * R::BM;
    const int n0 = nt * R::BN;
    const int nk = g.ksteps;
    const int krot = g.krot_on ? (nt * 7) % nk : 0;

    // per-lane offsets of the load groups from the tile's first operand rows
    // (rows past the edge re-read the last row); a tile spans less than
    // 4 GiB of either operand (the host checks), the whole operand may not
    const uint8_t* const a0 = g.a + (int64_t)m0 * g.lda;
    const uint8_t* const w0 = g.w + (int64_t)n0 * g.ldw;
    uint32_t off[R::kGroupsPerWave];
#pragma unroll
    for (int q = 0; q < R::kGroupsPerWave; ++q) {
        const int row = (wave + 4 * q) * 8 + (lane >> 3);
        const int chunk = (lane & 7) ^ swz(row);
        if (q < WTM) {
            const int m = min(m0 + row, g.M - 1);
            off[q] = (uint32_t)(m - m0) * (uint32_t)g.lda + (uint32_t)(chunk * 16);
        } else {
            const int n = min(n0 + row - R::BM, g.N - 1);
            off[q] = (uint32_t)(n - n0) * (uint32_t)g.ldw + (uint32_t)(chunk * 16);
        }
    }
    // LDS: the group's 1 KiB of each stage (m0 of the loads), and this lane's
    // operand read bases in each stage
    const uint32_t st[2] = {lds_addr(lds0), lds_addr(lds1)};
    const uint32_t ld0 = st[0] + (uint32_t)wave * 1024, ld1 = st[1] + (uint32_t)wave * 1024;
    const int kg = lane >> 4, r16 = lane & 15;
    uint32_t ab[2][2], wb[2][2];
#pragma unroll
    for (int s = 0; s < 2; ++s)
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const uint32_t in_row = (uint32_t)(r16 * kBK + (((2 * kg + h) ^ swz(r16)) << 4));
            ab[s][h] = st[s] + (uint32_t)(wm * WTM * 16 * kBK) + in_row;
            wb[s][h] = st[s] + (uint32_t)((R::BM + wn * WTN * 16) * kBK) + in_row;
        }

    v4f acc[WTN][WTM];
#pragma unroll
    for (int i = 0; i < WTN; ++i)
#pragma unroll
        for (int j = 0; j < WTM; ++j) acc[i][j] = v4f{0.f, 0.f, 0.f, 0.f};

    // prologue: steps 0 and 1 in flight, then the fragments of step 0
#pragma unroll
    for (int s = 0; s < 2; ++s) {
        const int64_t kb = (int64_t)((min(s, nk - 1) + krot) % nk) * kBK;
#pragma unroll
        for (int q = 0; q < R::kGroupsPerWave; ++q)
            roll_load(q < WTM ? a0 + kb : w0 + kb, off[q], (s ? ld1 : ld0) + q * 4096);
    }
    wait_vmcnt<R::kGroupsPerWave>();
    __builtin_amdgcn_s_barrier();
    Frags<WTM, WTN> f;
    static_for<WTM + WTN>([&](auto nc) { RollRead<WTM, WTN, decltype(nc)::value>::run(f, wb[0], ab[0]); });
    lds_wait_all();
#pragma unroll
    for (int j = 0; j < WTM; ++j) asm volatile("" : "+v"(f.a[j]));
#pragma unroll
    for (int i = 0; i < WTN; ++i) asm volatile("" : "+v"(f.w[i]));

    // steady state in pairs of steps (stage 0, stage 1) that both refill
    // their stage, then the last pair (the plan takes this kernel only for an
    // even number of K-steps), so no step is behind a branch
#define SPEC_ROLL(S, LOADS, NEXT, IT) \
    roll_step<R, WTM, WTN, S, LOADS, NEXT>(a0, w0, IT, nk, krot, off, S ? ld1 : ld0, ab[S ^ 1], wb[S ^ 1], acc, f)
    for (int it = 0; it + 2 < nk; it += 2) {
        SPEC_ROLL(0, true, true, it);
        SPEC_ROLL(1, true, true, it + 1);
    }
    SPEC_ROLL(0, false, true, nk - 2);
    SPEC_ROLL(1, false, false, nk - 1);
#undef SPEC_ROLL
    wait_vmcnt<0>();

    float sa_reg[WTM];
#pragma unroll
    for (int j = 0; j < WTM; ++j)
        sa_reg[j] = g.a_per_tensor ? g.sa[0] : g.sa[min(m0 + (wm * WTM + j) * 16 + r16, g.M - 1)];
    const bool edge = m0 + R::BM > g.M || n0 + R::BN > g.N;
    if (STATS == 0 && g.out_f32) {
        if (edge) roll_store_f32<WTM, WTN, true>(g, acc, sa_reg, m0, n0, wm, wn, lane);
        else roll_store_f32<WTM, WTN, false>(g, acc, sa_reg, m0, n0, wm, wn, lane);
    } else {
        __builtin_amdgcn_s_barrier();     // every wave is done reading the stages
        const int64_t col_group = (int64_t)nt * 2 + wn;
        if (edge) roll_store_lds<WTM, WTN, STATS, true>(g, acc, sa_reg, m0, n0, wm, wn, wave, lane, lds, col_group);
        else roll_store_lds<WTM, WTN, STATS, false>(g, acc, sa_reg, m0, n0, wm, wn, wave, lane, lds, col_group);
    }
}

// ---- tile configurations (plan.hpp, kTiles) ----------------------------------

// The statistics epilogues are separate instantiations, so the plain GEMMs'
// register allocation does not carry them (and the 160x224 tile, whose
// statistics variant would spill, has none: the plan never asks for it).
template <int KIND, bool WITH_STATS = true, bool REDUCE_LAST = true>
hipError_t launch_cfg(GemmArgs g, hipStream_t stream) {
    constexpr int WTM = kTiles[KIND].wtm, WTN = kTiles[KIND].wtn, WM = kTiles[KIND].wm, WN = kTiles[KIND].wn;
    constexpr int STAGES = kTiles[KIND].stages;
    using C = GemmCfg<WTM, WTN, WM, WN, STAGES>;
    static_assert(C::BM == tile_bm(KIND) && C::BN == tile_bn(KIND), "tile table");
    const int total = g.m_tiles * g.n_tiles * g.splits;
    if (g.silu_inter > 0) {
        hipLaunchKernelGGL((gemm_fp8_kernel<WTM, WTN, WM, WN, STAGES, 3, false>), dim3(total), dim3(C::kThreads), 0,
                           stream, g);
        return hipGetLastError();
    }
    if constexpr (WITH_STATS) {
        if (g.stats_mode == 1) {
            hipLaunchKernelGGL((gemm_fp8_kernel<WTM, WTN, WM, WN, STAGES, 1, false>), dim3(total), dim3(C::kThreads), 0,
                               stream, g);
            return hipGetLastError();
        }
        if (g.stats_mode == 2) {
            hipLaunchKernelGGL((gemm_fp8_kernel<WTM, WTN, WM, WN, STAGES, 2, false>), dim3(total), dim3(C::kThreads), 0,
                               stream, g);
            return hipGetLastError();
        }
    }
    if (g.stats_mode != 0) return hipErrorInvalidValue;
    if (!REDUCE_LAST && g.splits > 1) return hipErrorInvalidValue;
    hipLaunchKernelGGL((gemm_fp8_kernel<WTM, WTN, WM, WN, STAGES, 0, REDUCE_LAST>), dim3(total), dim3(C::kThreads), 0,
                       stream, g);
    return hipGetLastError();
}

template <int KIND>
hipError_t launch_roll(const GemmArgs& g, hipStream_t stream) {
    constexpr int WTM = kTiles[KIND].wtm, WTN = kTiles[KIND].wtn;
    static_assert(kTiles[KIND].roll && kTiles[KIND].wm == 2 && kTiles[KIND].wn == 2 && kTiles[KIND].stages == 2,
                  "roll tiles are 2x2 waves over 2 stages");
    static_assert(RollCfg<WTM, WTN>::BM == tile_bm(KIND) && RollCfg<WTM, WTN>::BN == tile_bn(KIND), "tile table");
    if (g.splits != 1 || g.silu_inter != 0 || g.ksteps < 2 || g.ksteps % 2 != 0) return hipErrorInvalidValue;
    const dim3 grid(g.m_tiles * g.n_tiles);
    if constexpr (KIND == kRollStatsKind) {
        if (g.stats_mode == 1 && !g.out_f32) {
            hipLaunchKernelGGL((gemm_fp8_roll_kernel<WTM, WTN, 1>), grid, dim3(256), 0, stream, g);
            return hipGetLastError();
        }
        if (g.stats_mode == 2 && !g.out_f32) {
            hipLaunchKernelGGL((gemm_fp8_roll_kernel<WTM, WTN, 2>), grid, dim3(256), 0, stream, g);
            return hipGetLastError();
        }
    }
    if (g.stats_mode != 0) return hipErrorInvalidValue;
    hipLaunchKernelGGL((gemm_fp8_roll_kernel<WTM, WTN, 0>), grid, dim3(256), 0, stream, g);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_gemm(const GemmPlan& p, const uint8_t* a, int64_t lda, const float* sa, int a_per_tensor,
                       const uint8_t* w, int64_t ldw, const float* sw, int w_per_tensor, int64_t M,
                       int64_t N, int64_t K, void* y, int64_t ldy, int out_f32, void* workspace,
                       hipStream_t stream, int stats_mode, float c2, float2* stats, int64_t ld_stats,
                       int64_t silu_inter) {
    if (!gemm_strides_fit(p.kind, lda, ldw)) {
        // the in-place-refill kernels address a tile's operand rows with 32-bit
        // offsets: strides too long for that take the 160x224 kernel, plain
        // output only (its statistics layout would differ; the host refuses
        // such a statistics call before it gets here)
        if (stats_mode != 0 || silu_inter != 0) return hipErrorInvalidValue;
        const GemmPlan q = plan_gemm_as(M, N, K, 2, 1, kEpiPlain);
        return launch_gemm(q, a, lda, sa, a_per_tensor, w, ldw, sw, w_per_tensor, M, N, K, y, ldy, out_f32,
                           workspace, stream, stats_mode, c2, stats, ld_stats, silu_inter);
    }
    GemmArgs g;
    g.stats = stats; g.ld_stats = ld_stats; g.stats_mode = stats_mode; g.c2 = c2;
    g.silu_inter = (int)silu_inter;
    g.a = a; g.w = w; g.sa = sa; g.sw = sw; g.y = y;
    char* ws = reinterpret_cast<char*>(workspace);
    g.tickets = reinterpret_cast<unsigned int*>(ws);
    g.part = reinterpret_cast<uint64_t*>(ws ? ws + p.part_off : nullptr);
    g.lda = lda; g.ldw = ldw; g.ldy = ldy;
    g.M = (int)M; g.N = (int)N; g.K = (int)K;
    g.a_per_tensor = a_per_tensor; g.w_per_tensor = w_per_tensor; g.out_f32 = out_f32;
    g.m_tiles = p.m_tiles; g.n_tiles = p.n_tiles; g.splits = p.splits; g.ksteps = (int)(K / kBK);
    g.group_m = p.group_m;
    g.krot_on = p.krot_on;
    hipError_t e;
    switch (p.kind) {
        case 0: e = launch_cfg<0>(g, stream); break;
        case 1: e = launch_cfg<1>(g, stream); break;
        case 2: e = launch_cfg<2, false, false>(g, stream); break;
        case 3: e = launch_cfg<3>(g, stream); break;
        case 4: e = launch_cfg<4>(g, stream); break;
        case 5: e = launch_cfg<5>(g, stream); break;
        case 6: e = launch_cfg<6>(g, stream); break;
        case 7: e = launch_cfg<7>(g, stream); break;
        case 8: e = launch_cfg<8>(g, stream); break;
        case 9: e = launch_roll<9>(g, stream); break;
        case 10: e = launch_roll<10>(g, stream); break;
        case 11: e = launch_roll<11>(g, stream); break;
        default: return hipErrorInvalidValue;
    }
    static_assert(kTileKinds == 12, "every tile kind has a case");
    return e;
}

}  // namespace specfp8
