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
//    swizzled slots (slot = chunk ^ (row & 7)); the swizzle is applied on the
//    global side, so global reads stay fully coalesced, and the MFMA operand
//    reads (ds_read_b128, 8 lanes on 8 different rows, same logical chunk)
//    hit 8 distinct slots -- no bank conflicts;
//  * STAGES buffers rotate so that STAGES-1 K-steps of loads are in flight
//    while the current one is multiplied.
//
// K is split across workgroups (split-K) when there are fewer output tiles
// than compute units; partial fp32 tiles then go to a workspace and a second
// kernel adds them in split order (deterministic) and applies the epilogue.
// Workgroup ids are remapped so that the tiles and K-splits that share
// operands run on the same XCD (blocks are dealt round-robin to the 8 XCDs),
// which keeps re-read operand bytes in that XCD's L2.
#include "device_common.hpp"
#include "kernels.hpp"

#ifdef SPECFP8_TUNING
#include <stdio.h>
#include <stdlib.h>
#endif


namespace specfp8 {

typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v4f __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void* lds_ptr_t;

namespace {

constexpr int kBK = 128;     // bytes (= E4M3 elements) of K per step
constexpr int kXcds = 8;

struct GemmArgs {
    const uint8_t* a;
    const uint8_t* w;
    const float* sa;
    const float* sw;
    void* y;
    float* partial;   // [splits][M][ldp] when splits > 1
    int64_t lda, ldw, ldy, ldp;
    int M, N, K;
    int a_per_tensor, w_per_tensor, out_f32;
    int m_tiles, n_tiles, splits, ksteps;
};

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
    static_assert((STAGES - 2) * kGroupsPerWave < 64, "vmcnt range");
};

template <class C>
__device__ __forceinline__ void issue_stage(const GemmArgs& g, char* stage, int m0, int n0,
                                            int64_t kbyte, int wave, int lane) {
    const int r_in = lane >> 3;       // row within the 8-row group
    const int slot = lane & 7;        // LDS slot this lane fills
    const int chunk = slot ^ r_in;    // logical 16-byte chunk loaded into it
#pragma unroll
    for (int i = 0; i < C::kGroupsPerWave; ++i) {
        const int grp = wave + i * C::kWaves;
        const int row = grp * 8 + r_in;
        const uint8_t* src;
        if (row < C::BM) {
            int m = m0 + row;
            m = m < g.M ? m : g.M - 1;
            src = g.a + (int64_t)m * g.lda + kbyte + chunk * 16;
        } else {
            int n = n0 + row - C::BM;
            n = n < g.N ? n : g.N - 1;
            src = g.w + (int64_t)n * g.ldw + kbyte + chunk * 16;
        }
        __builtin_amdgcn_global_load_lds((const void*)src, (lds_ptr_t)(stage + grp * 1024), 16, 0, 0);
    }
}

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
// awaited explicitly by frag_wait().
__device__ __forceinline__ v8i lds_frag(uint32_t stage, int row, int kg) {
    const int sw = row & 7;
    const uint32_t base = stage + (uint32_t)row * kBK;
    const uint32_t a0 = base + ((uint32_t)((2 * kg) ^ sw) << 4);
    const uint32_t a1 = base + ((uint32_t)((2 * kg + 1) ^ sw) << 4);
    u32x4 lo, hi;
    asm volatile("ds_read_b128 %0, %1" : "=v"(lo) : "v"(a0));
    asm volatile("ds_read_b128 %0, %1" : "=v"(hi) : "v"(a1));
    v8i r;
    r[0] = lo[0]; r[1] = lo[1]; r[2] = lo[2]; r[3] = lo[3];
    r[4] = hi[0]; r[5] = hi[1]; r[6] = hi[2]; r[7] = hi[3];
    return r;
}

// Wait for every outstanding LDS read; each fragment passes through an empty
// asm after the wait, so no use of it can be scheduled before the wait.
template <int N>
__device__ __forceinline__ void frag_wait(v8i (&f)[N]) {
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
#pragma unroll
    for (int i = 0; i < N; ++i) asm volatile("" : "+v"(f[i]));
}

// One K-step on compile-time stage S: wait for its loads, barrier, refill the
// stage consumed one step earlier, multiply.  Every stage is its own LDS
// object and every wait count is a compile-time constant, so the compiler can
// tell that the direct-to-LDS loads still in flight target other stages and
// does not drain them before the LDS reads of this one.  Past the end of the
// K range the refill re-loads the last K-step (in bounds, never multiplied),
// which keeps the number of loads in flight -- and so the wait -- uniform.
template <class C, int STAGES, int WTM, int WTN, int S>
__device__ __forceinline__ void kstep(const GemmArgs& g, char* const* stages, int it, int nk, int ks0, int m0,
                                      int n0, int wave, int lane, int wm, int wn, v4f (&acc)[WTN][WTM]) {
    wait_vmcnt<(STAGES - 2) * C::kGroupsPerWave>();
    __builtin_amdgcn_s_barrier();
    const int nxt = min(it + STAGES - 1, nk - 1);
    issue_stage<C>(g, stages[(S + STAGES - 1) % STAGES], m0, n0, (int64_t)(ks0 + nxt) * kBK, wave, lane);
    const uint32_t st = lds_addr(stages[S]);
    const int kg = lane >> 4;
    const int r16 = lane & 15;
    v8i frag[WTM + WTN];
#pragma unroll
    for (int j = 0; j < WTM; ++j) frag[j] = lds_frag(st, (wm * WTM + j) * 16 + r16, kg);
#pragma unroll
    for (int i = 0; i < WTN; ++i) frag[WTM + i] = lds_frag(st, C::BM + (wn * WTN + i) * 16 + r16, kg);
    frag_wait(frag);
#pragma unroll
    for (int i = 0; i < WTN; ++i)
#pragma unroll
        for (int j = 0; j < WTM; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(frag[WTM + i], frag[j], acc[i][j], 0, 0,
                                                                         0, 0, 0, 0);
}

template <int WTM, int WTN, int WM, int WN, int STAGES>
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
    const int mt = tile % g.m_tiles;
    const int nt = tile / g.m_tiles;
    const int m0 = mt * C::BM;
    const int n0 = nt * C::BN;

    const int ks_per = (g.ksteps + g.splits - 1) / g.splits;
    const int ks0 = split * ks_per;
    const int ks1 = min(g.ksteps, ks0 + ks_per);
    const int nk = ks1 - ks0;

    v4f acc[WTN][WTM];
#pragma unroll
    for (int i = 0; i < WTN; ++i)
#pragma unroll
        for (int j = 0; j < WTM; ++j) acc[i][j] = v4f{0.f, 0.f, 0.f, 0.f};

    // prologue: STAGES-1 stages in flight
#pragma unroll
    for (int s = 0; s < STAGES - 1; ++s)
        issue_stage<C>(g, stages[s], m0, n0, (int64_t)(ks0 + min(s, nk - 1)) * kBK, wave, lane);

    for (int base = 0; base < nk; base += STAGES) {
        kstep<C, STAGES, WTM, WTN, 0>(g, stages, base, nk, ks0, m0, n0, wave, lane, wm, wn, acc);
        if (base + 1 < nk) kstep<C, STAGES, WTM, WTN, 1>(g, stages, base + 1, nk, ks0, m0, n0, wave, lane, wm, wn, acc);
        if constexpr (STAGES > 2)
            if (base + 2 < nk) kstep<C, STAGES, WTM, WTN, 2>(g, stages, base + 2, nk, ks0, m0, n0, wave, lane, wm, wn, acc);
        if constexpr (STAGES > 3)
            if (base + 3 < nk) kstep<C, STAGES, WTM, WTN, 3>(g, stages, base + 3, nk, ks0, m0, n0, wave, lane, wm, wn, acc);
    }
    wait_vmcnt<0>();   // no direct-to-LDS write may outlive the workgroup

    const int kg = lane >> 4;
    const int r16 = lane & 15;
    // epilogue: lane holds D[n = 4*(lane/16) + r][m = lane%16] of each 16x16 block
#pragma unroll
    for (int i = 0; i < WTN; ++i) {
        const int n = n0 + (wn * WTN + i) * 16 + 4 * kg;
        if (n >= g.N) continue;
#pragma unroll
        for (int j = 0; j < WTM; ++j) {
            const int m = m0 + (wm * WTM + j) * 16 + r16;
            if (m >= g.M) continue;
            const v4f a = acc[i][j];
            if (g.splits > 1) {
                float* dst = g.partial + ((int64_t)split * g.M + m) * g.ldp + n;
                *reinterpret_cast<float4*>(dst) = make_float4(a[0], a[1], a[2], a[3]);
                continue;
            }
            const float sa = g.a_per_tensor ? g.sa[0] : g.sa[m];
            float y[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const float sw = g.w_per_tensor ? g.sw[0] : g.sw[n + r < g.N ? n + r : g.N - 1];
                y[r] = (a[r] * sa) * sw;
            }
            if (g.out_f32) {
                float* dst = reinterpret_cast<float*>(g.y) + (int64_t)m * g.ldy + n;
                if (n + 3 < g.N) {
                    *reinterpret_cast<float4*>(dst) = make_float4(y[0], y[1], y[2], y[3]);
                } else {
                    for (int r = 0; r < 4 && n + r < g.N; ++r) dst[r] = y[r];
                }
            } else {
                uint16_t* dst = reinterpret_cast<uint16_t*>(g.y) + (int64_t)m * g.ldy + n;
                if (n + 3 < g.N) {
                    uint2 o;
                    o.x = f32_to_bf16_rne(y[0]) | (f32_to_bf16_rne(y[1]) << 16);
                    o.y = f32_to_bf16_rne(y[2]) | (f32_to_bf16_rne(y[3]) << 16);
                    *reinterpret_cast<uint2*>(dst) = o;
                } else {
                    for (int r = 0; r < 4 && n + r < g.N; ++r) dst[r] = (uint16_t)f32_to_bf16_rne(y[r]);
                }
            }
        }
    }
}

// Sum the split-K partials in split order, then scale and convert.
__global__ __launch_bounds__(256) void splitk_reduce_kernel(GemmArgs g) {
    const int64_t quads = (int64_t)((g.N + 3) / 4);
    const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= (int64_t)g.M * quads) return;
    const int m = (int)(idx / quads);
    const int n = (int)(idx % quads) * 4;
    float4 s = *reinterpret_cast<const float4*>(g.partial + (int64_t)m * g.ldp + n);
    for (int z = 1; z < g.splits; ++z) {
        const float4 p = *reinterpret_cast<const float4*>(g.partial + ((int64_t)z * g.M + m) * g.ldp + n);
        s.x += p.x; s.y += p.y; s.z += p.z; s.w += p.w;
    }
    const float a[4] = {s.x, s.y, s.z, s.w};
    const float sa = g.a_per_tensor ? g.sa[0] : g.sa[m];
    float y[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        const float sw = g.w_per_tensor ? g.sw[0] : g.sw[n + r < g.N ? n + r : g.N - 1];
        y[r] = (a[r] * sa) * sw;
    }
    if (g.out_f32) {
        float* dst = reinterpret_cast<float*>(g.y) + (int64_t)m * g.ldy + n;
        if (n + 3 < g.N) {
            *reinterpret_cast<float4*>(dst) = make_float4(y[0], y[1], y[2], y[3]);
        } else {
            for (int r = 0; r < 4 && n + r < g.N; ++r) dst[r] = y[r];
        }
    } else {
        uint16_t* dst = reinterpret_cast<uint16_t*>(g.y) + (int64_t)m * g.ldy + n;
        if (n + 3 < g.N) {
            uint2 o;
            o.x = f32_to_bf16_rne(y[0]) | (f32_to_bf16_rne(y[1]) << 16);
            o.y = f32_to_bf16_rne(y[2]) | (f32_to_bf16_rne(y[3]) << 16);
            *reinterpret_cast<uint2*>(dst) = o;
        } else {
            for (int r = 0; r < 4 && n + r < g.N; ++r) dst[r] = (uint16_t)f32_to_bf16_rne(y[r]);
        }
    }
}

// ---- tile configurations -------------------------------------------------
// kind  BM x BN   waves (wave tile)     stages  LDS
//  0    64 x 64   2x2 (32x32)           4       64 KiB   small M
//  1    80 x 128  1x2 (80x64)           4       104 KiB  M <= 80
//  2   320 x 128  4x2 (80x64)           2       112 KiB
//  3   256 x 128  2x2 (128x64)          3       144 KiB  large M
//  4   320 x 64   4x2 (80x32)           3       144 KiB
//  5   160 x 128  2x2 (80x64)           4       144 KiB
//  6   320 x 32   4x1 (80x32)           3       132 KiB
//  7   160 x 64   2x2 (80x32)           4       112 KiB
using Cfg0 = GemmCfg<2, 2, 2, 2, 4>;
using Cfg1 = GemmCfg<5, 4, 1, 2, 4>;
using Cfg2 = GemmCfg<5, 4, 4, 2, 2>;
using Cfg3 = GemmCfg<8, 4, 2, 2, 3>;
using Cfg4 = GemmCfg<5, 2, 4, 2, 3>;
using Cfg5 = GemmCfg<5, 4, 2, 2, 4>;
using Cfg6 = GemmCfg<5, 2, 4, 1, 3>;
using Cfg7 = GemmCfg<5, 2, 2, 2, 4>;

constexpr int kCfgBM[8] = {Cfg0::BM, Cfg1::BM, Cfg2::BM, Cfg3::BM, Cfg4::BM, Cfg5::BM, Cfg6::BM, Cfg7::BM};
constexpr int kCfgBN[8] = {Cfg0::BN, Cfg1::BN, Cfg2::BN, Cfg3::BN, Cfg4::BN, Cfg5::BN, Cfg6::BN, Cfg7::BN};

template <class C, int WTM, int WTN, int WM, int WN, int STAGES>
hipError_t launch_cfg(GemmArgs g, hipStream_t stream) {
    auto kern = gemm_fp8_kernel<WTM, WTN, WM, WN, STAGES>;
    const int total = g.m_tiles * g.n_tiles * g.splits;
    hipLaunchKernelGGL(kern, dim3(total), dim3(C::kThreads), 0, stream, g);
    return hipGetLastError();
}

}  // namespace

GemmPlan plan_gemm(int64_t M, int64_t N, int64_t K) {
    GemmPlan p{};
    if (M <= 64) p.kind = 0;
    else if (M <= 80) p.kind = 1;
    else if (M <= 160) p.kind = 5;
    else if (M <= 640) p.kind = 2;
    else p.kind = 3;
    const int ksteps = (int)(K / kBK);
    int splits = 0;
#ifdef SPECFP8_TUNING
    // tuning builds only: SPECFP8_GEMM_PLAN="kind:splits" overrides the choice
    if (const char* env = getenv("SPECFP8_GEMM_PLAN")) {
        int k = -1, sp = 0;
        if (sscanf(env, "%d:%d", &k, &sp) >= 1 && k >= 0 && k < 8) { p.kind = k; splits = sp; }
    }
#endif
    const int bm = kCfgBM[p.kind], bn = kCfgBN[p.kind];
    p.m_tiles = (int)((M + bm - 1) / bm);
    p.n_tiles = (int)((N + bn - 1) / bn);
    const int tiles = p.m_tiles * p.n_tiles;
    if (splits <= 0) {
        // Split K only when fewer than half of the 256 compute units would
        // get a tile, and never beyond one wave of workgroups: every split
        // adds an M x N fp32 partial that is written and read back.
        splits = 1;
        if (2 * tiles <= 256) splits = 256 / tiles;
        const int max_split = ksteps / 4 > 0 ? ksteps / 4 : 1;   // >= 4 K-steps per split
        if (splits > max_split) splits = max_split;
        if (splits > 16) splits = 16;
    }
    if (splits > ksteps) splits = ksteps;
    if (splits < 1) splits = 1;
    // every split must own at least one K-step after ceil division
    while (splits > 1 && (int64_t)((ksteps + splits - 1) / splits) * (splits - 1) >= ksteps) --splits;
    p.splits = splits;
    p.ldp = (N + 3) / 4 * 4;
    p.workspace_bytes = splits > 1 ? (size_t)splits * (size_t)M * (size_t)p.ldp * sizeof(float) : 0;
    return p;
}

hipError_t launch_gemm(const GemmPlan& p, const uint8_t* a, int64_t lda, const float* sa, int a_per_tensor,
                       const uint8_t* w, int64_t ldw, const float* sw, int w_per_tensor, int64_t M,
                       int64_t N, int64_t K, void* y, int64_t ldy, int out_f32, void* workspace,
                       hipStream_t stream) {
    GemmArgs g;
    g.a = a; g.w = w; g.sa = sa; g.sw = sw; g.y = y;
    g.partial = reinterpret_cast<float*>(workspace);
    g.lda = lda; g.ldw = ldw; g.ldy = ldy; g.ldp = p.ldp;
    g.M = (int)M; g.N = (int)N; g.K = (int)K;
    g.a_per_tensor = a_per_tensor; g.w_per_tensor = w_per_tensor; g.out_f32 = out_f32;
    g.m_tiles = p.m_tiles; g.n_tiles = p.n_tiles; g.splits = p.splits; g.ksteps = (int)(K / kBK);
    hipError_t e;
    switch (p.kind) {
        case 0: e = launch_cfg<Cfg0, 2, 2, 2, 2, 4>(g, stream); break;
        case 1: e = launch_cfg<Cfg1, 5, 4, 1, 2, 4>(g, stream); break;
        case 2: e = launch_cfg<Cfg2, 5, 4, 4, 2, 2>(g, stream); break;
        case 3: e = launch_cfg<Cfg3, 8, 4, 2, 2, 3>(g, stream); break;
        case 4: e = launch_cfg<Cfg4, 5, 2, 4, 2, 3>(g, stream); break;
        case 5: e = launch_cfg<Cfg5, 5, 4, 2, 2, 4>(g, stream); break;
        case 6: e = launch_cfg<Cfg6, 5, 2, 4, 1, 3>(g, stream); break;
        default: e = launch_cfg<Cfg7, 5, 2, 2, 2, 4>(g, stream); break;
    }
    if (e != hipSuccess || p.splits == 1) return e;
    const int64_t work = M * ((N + 3) / 4);
    hipLaunchKernelGGL(splitk_reduce_kernel, dim3((unsigned)((work + 255) / 256)), dim3(256), 0, stream, g);
    return hipGetLastError();
}

}  // namespace specfp8
