// Host-side planners: tile shape, K split and workspace layout of the FP8
// GEMM, and the workspace layout of the acceptance.  Plain C++ (no HIP), so
// the argument checks and plans can also be built and exercised on a host
// without a GPU.
#include "kernels.hpp"
#include "plan.hpp"

namespace specfp8 {

namespace {

inline size_t align256(size_t x) { return (x + 255) / 256 * 256; }

// A CU's operand rows per K-step over the whole GEMM: the rounds of tiles the
// 256 CUs run, times a tile's rows (BM + BN).  A CU streams its operand bytes
// at a rate no tile shape changes, so this orders tile shapes by time.
int64_t rows_per_cu(int64_t M, int64_t N, int kind) {
    const int64_t tiles = ((M + tile_bm(kind) - 1) / tile_bm(kind)) * ((N + tile_bn(kind) - 1) / tile_bn(kind));
    return ((tiles + 255) / 256) * (int64_t)(tile_bm(kind) + tile_bn(kind));
}

}  // namespace

GemmPlan plan_gemm_as(int64_t M, int64_t N, int64_t K, int kind, int splits, int epilogue) {
    GemmPlan p{};
    if (kind < 0 || kind >= kTileKinds) kind = 2;
    // the statistics epilogues never split K; the 160x224 tile has no
    // statistics variant (it would spill), 160x192 takes its place
    if (epilogue == kEpiStats && kind == 2) kind = 4;
    // the in-place-refill kernels have the plain epilogue only (kRollStatsKind
    // also the statistics one) and no K split
    if (kTiles[kind].roll && epilogue != kEpiPlain && !(epilogue == kEpiStats && kind == kRollStatsKind))
        kind = epilogue == kEpiStats ? 4 : 2;
    if (kTiles[kind].roll) splits = 1;
    if (epilogue != kEpiPlain) splits = 1;
    p.kind = kind;
    const int bm = tile_bm(kind), bn = tile_bn(kind);
    p.m_tiles = (int)((M + bm - 1) / bm);
    p.n_tiles = (int)((N + bn - 1) / bn);
    const int64_t tiles = (int64_t)p.m_tiles * p.n_tiles;
    // the 160x224 kernel has no in-kernel reduction (its registers are
    // full), and a tile without a ticket cannot be reduced: no K split
    if (kind == 2 || tiles > (int64_t)(kGemmTicketBytes / sizeof(unsigned int))) splits = 1;
    const int ksteps = (int)(K / kGemmBK);
    if (splits > ksteps) splits = ksteps;
    if (splits < 1) splits = 1;
    // every split must own at least one K-step after ceil division
    while (splits > 1 && (int64_t)((ksteps + splits - 1) / splits) * (splits - 1) >= ksteps) --splits;
    p.splits = splits;
    p.reduce = splits > 1 ? kReduceLast : kReduceNone;
    // Many M-tiles (long prompts): tiles in groups of 4 M-tiles with K walked
    // in step, so the 32 tiles an XCD runs at once re-read 4 activation and
    // 8 weight tiles from its L2 (5-8% at M = 4096).  Few M-tiles keep the
    // staggered K start, which spreads the requests for shared rows.
    p.group_m = 1;
    p.krot_on = 1;
    if (p.m_tiles >= 8 && splits == 1) {
        p.group_m = 4;
        p.krot_on = 0;
    }
    p.stat_groups = (int64_t)p.n_tiles * kTiles[kind].wn;
    p.part_off = kGemmTicketBytes;
    p.workspace_bytes =
        splits > 1 ? p.part_off + align256((size_t)tiles * splits * (size_t)bm * bn * sizeof(float)) : 0;
    return p;
}

bool gemm_strides_fit(int kind, int64_t lda, int64_t ldw) {
    if (kind < 0 || kind >= kTileKinds || !kTiles[kind].roll) return true;
    const uint64_t lim = 1ull << 32;
    return (uint64_t)(tile_bm(kind) - 1) * (uint64_t)lda + kGemmBK <= lim &&
           (uint64_t)(tile_bn(kind) - 1) * (uint64_t)ldw + kGemmBK <= lim;
}

GemmPlan plan_gemm(int64_t M, int64_t N, int64_t K, int epilogue) {
    const int ksteps = (int)(K / kGemmBK);
    int splits = 1;
    // Tile shapes by measurement on MI355X (M = B*(k+1) verify rows).
    if (M <= 80) {
        // Draft and small verify batches: a weight stream with a fixed cost
        // per workgroup.  Very wide N (gate|up) fills the chip unsplit;
        // otherwise 64x64 tiles with K split until about 256 workgroups run
        // (one round of the CUs: at M = 80 the long-K down projection took
        // 25.2 us split in 4, 512 workgroups, and 23.6 us split in 2),
        // keeping >= 8 K-steps per split.  The last workgroup of a tile adds
        // its partial tiles: one launch fewer, 1-2 us per GEMM here.
        if (N >= 192 * 64) return plan_gemm_as(M, N, K, M <= 64 ? 8 : 1, 1, epilogue);
        const int64_t tiles = ((M + 63) / 64) * ((N + 63) / 64);
        splits = (int)(256 / tiles);
        const int max_split = ksteps / 8 > 0 ? ksteps / 8 : 1;
        if (splits > max_split) splits = max_split;
        if (splits > 16) splits = 16;
        return plan_gemm_as(M, N, K, 0, splits, epilogue);
    }
    if (M <= 320) {
        // wide N: one 160x224 tile per CU (gate|up), or 160x192 for an LM
        // head (160x224 with a ragged last tile where N % 192 != 0); where the
        // tiles take several rounds of the CUs (an LM head), the 160x384
        // in-place-refill tile streams fewer operand rows per CU
        if (N % 224 == 0 && N >= 224 * 64 && rows_per_cu(M, N, 2) <= rows_per_cu(M, N, 11))
            return plan_gemm_as(M, N, K, 2, 1, epilogue);
        if (N >= 192 * 64) {
            // the plain epilogue takes the fewest rows per CU among 160x192
            // (160x224 where it divides N better), 160x224 and 160x384; the
            // statistics epilogue takes the same tile where it has one
            // (160x384), else 160x192 (160x224 where it divides N better)
            int stats_kind = (N % 192 == 0) ? 4 : 2;
            int plain_kind = stats_kind;
            if (rows_per_cu(M, N, 2) < rows_per_cu(M, N, plain_kind)) plain_kind = 2;
            if (ksteps >= 2 && ksteps % 2 == 0 && rows_per_cu(M, N, 11) < rows_per_cu(M, N, plain_kind))
                plain_kind = 11;
            if (plain_kind == kRollStatsKind) stats_kind = kRollStatsKind;
            GemmPlan p = plan_gemm_as(M, N, K, epilogue == kEpiPlain ? plain_kind : stats_kind, 1, epilogue);
            // Both walk K in order, so that the logits stored with their
            // statistics are the plain GEMM's bit for bit also where the two
            // take different tiles (a staggered K start gained nothing
            // measurable on the LM head).
            if (plain_kind != stats_kind || plain_kind == kRollStatsKind) p.krot_on = 0;
            return p;
        }
        // Short N (QKV, O, down).  A CU streams its operand rows at a rate
        // that no tile shape or wave count tried raised (~35 GB/s per CU at
        // every shape of the verify step), so a CU's time follows the operand
        // bytes it streams; a K split pays when it brings idle CUs in, and its
        // partial tiles are added by the last workgroup of each tile.  Sweeps
        // (cold weights) chose: long K (down, 14336 -> 4096) 80x128 tiles with
        // K split in 2; N <= 4096 (O) 160x64 split in 2; else (QKV) 64x128
        // unsplit.
        if (K >= 2 * N) return plan_gemm_as(M, N, K, 1, 2, epilogue);
        if (N <= 4096) return plan_gemm_as(M, N, K, 7, 2, epilogue);
        return plan_gemm_as(M, N, K, 8, 1, epilogue);
    }
    // Long prompts.  A CU's time is its operand bytes: per tile (BM + BN)
    // rows per K-step, times the rounds of tiles every CU runs.  The 256-wide
    // in-place-refill tiles stream fewer rows per output; take the kind with
    // the fewest rows per CU (an even number of K-steps is required by them).
    int best = 2;
    if (M >= 1024 && epilogue == kEpiPlain && ksteps >= 2 && ksteps % 2 == 0) {
        for (int kind : {9, 10})
            if (rows_per_cu(M, N, kind) < rows_per_cu(M, N, best)) best = kind;
    }
    return plan_gemm_as(M, N, K, best, 1, epilogue);
}

AcceptPlan plan_accept(int64_t B, int64_t k, int64_t V) {
    AcceptPlan p{};
    p.chunk = kAcceptChunk;
    p.nchunk = (V + kAcceptChunk - 1) / kAcceptChunk;
    p.schunk = kAcceptSlice;
    p.nschunk = (V + kAcceptSlice - 1) / kAcceptSlice;
    const int64_t R = 2 * k + 1;
    p.stats_off = 0;
    p.fine_off = align256((size_t)B * R * p.nschunk * 8);     // after a float2 per (row, slice)
    p.ctr_off = p.fine_off + align256((size_t)B * p.nchunk * kAcceptThreads * sizeof(double));
    p.zx_off = p.ctr_off + align256((size_t)B * sizeof(unsigned int));
    p.bytes = p.zx_off + align256((size_t)B * k * 8);                // a float2 per (sequence, draft)
    if (B == 0) p.bytes = 0;
    return p;
}

}  // namespace specfp8
