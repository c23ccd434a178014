// Launch geometry shared by the host-side planners (plan.cpp) and the
// kernels (gemm.hip, accept.hip).  Host-only code: no HIP here.
#pragma once

#include <stddef.h>
#include <stdint.h>

namespace specfp8 {

// ---- FP8 GEMM tiles ---------------------------------------------------------
// A tile is a WM x WN grid of waves, each wave holding WTM x WTN blocks of
// 16x16 outputs; STAGES LDS buffers rotate through the K-loop (deeper
// pipelines, 6 stages of 64x128 or 8 of 64x64, measured no faster).  roll: the
// kernel whose operand fragments are refilled in place (one fragment set;
// never split in K; plain epilogue only, but for kRollStatsKind, which also
// has the statistics epilogue).  rspan8, lspan8: the K-step schedule of the
// non-roll kernel, numerators over 8 of the step's MFMAs: the next step's LDS
// operand reads go out over the first rspan8/8 of them and the stage refill
// loads over the first lspan8/8 (chosen by cold same-run sweeps: spreading the
// refills over the whole step took down at M = 320 from 45.8 to 42.8 us and
// gate|up from 48.3 to 46.7 us; the short-N tiles measured best at 5/8, 4/8).
struct TileShape {
    int wtm, wtn, wm, wn, stages, roll, rspan8, lspan8;
};

// kind  BM x BN   waves (wave tile)     stages  LDS      used for
//  0    64 x 64   2x2 (32x32)           4       64 KiB   M <= 80 (K split)
//  1    80 x 128  1x2 (80x64)           4       104 KiB  M <= 80 wide N; M <= 320 long K (split)
//  2   160 x 224  2x2 (80x112)          3       144 KiB  M <= 320 wide N, large M
//  3   256 x 128  2x2 (128x64)          3       144 KiB
//  4   160 x 192  2x2 (80x96)           3       132 KiB  wide N with statistics
//  5   160 x 128  2x2 (80x64)           4       144 KiB
//  6   320 x 64   4x1 (80x64)           3       144 KiB
//  7   160 x 64   2x2 (80x32)           4       112 KiB  M <= 320, N <= 4096 (split)
//  8    64 x 128  2x2 (32x64)           4        96 KiB  M <= 64 wide N; M <= 320 short N
//  9   256 x 224  2x2 (128x112), roll   2       120 KiB  large M
// 10   256 x 256  2x2 (128x128), roll   2       128 KiB  large M
// 11   160 x 384  2x2 (80x192), roll    2       136 KiB  M <= 320, very wide N (LM head, with statistics)
constexpr TileShape kTiles[] = {
    {2, 2, 2, 2, 4, 0, 5, 4}, {5, 4, 1, 2, 4, 0, 6, 8}, {5, 7, 2, 2, 3, 0, 6, 8}, {8, 4, 2, 2, 3, 0, 5, 4},
    {5, 6, 2, 2, 3, 0, 5, 4}, {5, 4, 2, 2, 4, 0, 5, 4}, {5, 4, 4, 1, 3, 0, 5, 4}, {5, 2, 2, 2, 4, 0, 5, 4},
    {2, 4, 2, 2, 4, 0, 5, 4}, {8, 7, 2, 2, 2, 1, 5, 4}, {8, 8, 2, 2, 2, 1, 5, 4}, {5, 12, 2, 2, 2, 1, 5, 4},
};
constexpr int kTileKinds = sizeof(kTiles) / sizeof(kTiles[0]);
// The in-place-refill tile that also has the statistics epilogue (LM head).
constexpr int kRollStatsKind = 11;
constexpr int tile_bm(int k) { return 16 * kTiles[k].wtm * kTiles[k].wm; }
constexpr int tile_bn(int k) { return 16 * kTiles[k].wtn * kTiles[k].wn; }
constexpr int tile_threads(int k) { return 64 * kTiles[k].wm * kTiles[k].wn; }
// The non-roll kind with this wave grid and pipeline depth, or -1.
constexpr int tile_kind_of(int wtm, int wtn, int wm, int wn, int stages) {
    for (int k = 0; k < kTileKinds; ++k)
        if (!kTiles[k].roll && kTiles[k].wtm == wtm && kTiles[k].wtn == wtn && kTiles[k].wm == wm &&
            kTiles[k].wn == wn && kTiles[k].stages == stages)
            return k;
    return -1;
}

constexpr int kGemmBK = 128;   // bytes (= E4M3 elements) of K per step

// Split-K reduction: every workgroup of a split tile stores its partial tile
// in the workspace, and the last of them to arrive (an atomic ticket per
// tile) adds all of them in split order and writes the output.  The tickets
// live in the first kGemmTicketBytes of the workspace, which must be zero
// before the first call and which every call leaves zero again.  Plans with
// more tiles than tickets, and the 160x224 tile (no registers left for the
// reduction), do not split K.
enum GemmReduce { kReduceNone = 0, kReduceLast = 1 };
constexpr size_t kGemmTicketBytes = 16384;   // 4096 tile tickets

// ---- acceptance ---------------------------------------------------------------
constexpr int kAcceptThreads = 256;
constexpr int kAcceptVecs = 8;                                           // 16-byte vectors per lane per item
constexpr int64_t kAcceptSlice = (int64_t)64 * kAcceptVecs * 8;          // 4096 logits per wave item
constexpr int kAcceptPerThread = kAcceptVecs * 8;                        // 64 logits per thread (sampling)
constexpr int64_t kAcceptChunk = (int64_t)kAcceptThreads * kAcceptPerThread;   // 16384 logits per sampling block

}  // namespace specfp8
