// Acceptance test of the speculative-decoding verify step.
//
// Greedy (T == 0):
//   greedy_partial_kernel  (row, slice) items -> max logit and its lowest index
//   greedy_final_kernel    b -> argmax per position, longest matching prefix
// Speculative sampling (T > 0):
//   stoch_stats_kernel     (row, slice) items -> slice max m and sum 2^(t - m) of
//                          t = z * log2(e)/T (the tempered logit in base 2), for
//                          target rows 0..k and draft rows 0..k-1
//   stoch_sample_kernel    (chunk, b) -> every block merges the slice statistics
//                          of its sequence in slice order, takes the (identical)
//                          accept/reject decisions and sums the residual
//                          distribution over its chunk's 64-element ranges;
//                          the last block of the sequence to finish (an atomic
//                          ticket) locates the range holding u*R, scans it in
//                          vocabulary order and writes the tokens.
//
// Two variants reuse these kernels:
//   target statistics given (the LM head's epilogue wrote them): the streaming
//     kernel reads only the draft rows, and the merges read the given entries
//     for the target rows (clear_tickets_kernel when nothing is streamed);
//   token trees: the streaming kernels run over the N+1 target rows of every
//     sequence, then tree_greedy_kernel / tree_sample_kernel walk the tree
//     (see the token-tree section below).
//
// The two streaming kernels run a persistent grid in which every WAVE walks
// (row, slice) items of 4096 logits with the loads of its next item in flight
// while it reduces the current one, so HBM sees one continuous stream of
// 2 bytes per logit and no item needs a workgroup barrier.  Items are strided
// over the waves, so at any moment the chip reads one contiguous stretch of
// the logit tensors.  The sample kernel re-reads only the row(s) of the
// position where sampling happens (<= 2 rows per sequence), with every load of
// a thread issued before it computes.  All reductions use a fixed order, so
// results are deterministic.
#include <atomic>
#include <mutex>

#include "device_common.hpp"
#include "kernels.hpp"
#include "plan.hpp"

// Fixed acceptance scratch for callers that cannot allocate
// (spec_verify_accept_noalloc).  Each GPU holds its own copy at its own
// address; host code reaches it only through the address accept_scratch()
// looks up, never through this name (a host-side stand-in).
static __device__ __align__(256) unsigned char scratch[specfp8::kAcceptScratchBytes];

namespace specfp8 {

namespace {

constexpr int kAThreads = kAcceptThreads;
constexpr int kWavesPerBlock = kAThreads / kWave;
constexpr int kVecs = kAcceptVecs;                     // 16-byte vectors per lane per item
constexpr int64_t kSlice = kAcceptSlice;               // 4096 logits per wave item
constexpr int kPerThread = kAcceptPerThread;           // 64 logits per thread (sample kernel)
constexpr int64_t kChunk = kAcceptChunk;               // 16384 logits per sample block
static_assert(kSlice == (int64_t)kWave * kVecs * 8 && kChunk == (int64_t)kAThreads * kPerThread, "accept geometry");
constexpr int kMaxChunks = kAThreads;                 // V <= 2^22: one chunk per thread
constexpr int kStreamWavesPerCU = 12;

struct AcceptArgs {
    const uint16_t* zt;
    const uint16_t* zd;
    const int32_t* x;
    const float* u;
    int32_t* out;
    int32_t* num;
    const int32_t* parent; // token tree: parent node of each node, -1 for the root's candidates (tree mode)
    int32_t* nodes;        // token tree: accepted node indices [B][k] (tree mode)
    float2* stats;         // [B][Rs][nslice] statistics of the streamed rows
    const float2* tst;     // target rows' statistics from the LM-head epilogue, or null
    int64_t ldtst;         // row stride of tst (entries)
    uint32_t ntst;         // entries per target row in tst
    float2* tsm;           // [B][k+1] tst merged to one entry per row by the statistics kernel, or null
    float2* zx;            // [B][k] (target, draft) logits at the draft tokens, gathered by the statistics
                           // kernel for the sampling kernel (chain mode with a statistics pass), or null
    uint32_t sw;           // streaming waves of the statistics grid (the first sw waves)
    double* finem;         // [B][nchunk][256] residual mass per 64-element range
    unsigned int* ctr;     // [B]
    int64_t V, nchunk;
    uint32_t nslice, items;   // slices per row; rows * nslice (< 2^31)
    int B, k;
    uint32_t R;            // rows per sequence whose statistics are merged (k+1, or 2k+1 with draft logits)
    uint32_t Rs;           // of these, the rows the statistics kernel streams (R, or R - (k+1) with tst)
    uint32_t rt0;          // first streamed row within the sequence (0, or k+1 with tst)
    float c2;              // log2(e) / T
};

// Statistics entries of row r (0..R-1) of sequence b: the target rows from
// the LM-head epilogue when given, else (and for draft rows) the streamed ones.
__device__ __forceinline__ const float2* row_stats(const AcceptArgs& a, int b, int r, uint32_t& n) {
    if ((uint32_t)r < a.rt0) {
        if (a.tsm) {
            n = 1;
            return a.tsm + (int64_t)b * (a.k + 1) + r;
        }
        n = a.ntst;
        return a.tst + ((int64_t)b * (a.k + 1) + r) * a.ldtst;
    }
    n = a.nslice;
    return a.stats + ((int64_t)b * a.Rs + (r - (int)a.rt0)) * a.nslice;
}

using Raw = uint4[kVecs];

// Slice layout: vector j of lane l starts at element e0 + (j * 64 + l) * 8, so
// one load instruction of a wave reads 1 KiB contiguous.
__device__ __forceinline__ int64_t slice_vec(int64_t e0, int j, int lane) {
    return e0 + ((int64_t)j * kWave + lane) * 8;
}

// Issue the loads of one slice (vector path only).  Out-of-range vectors load
// the last full vector of the slice instead (always in bounds, V % 8 == 0);
// their values are masked where they are used.  The loads are nontemporal:
// the statistics pass reads each logit once, and cache-allocating loads of
// 148 MB would push the model's weights and the dirty outputs of the layer
// out of the Infinity Cache (measured in the verify step: the statistics pass
// 31.1 -> 27.0 us, the next gate|up and down GEMMs ~1 us faster each; the
// sampling kernel's re-read of the residual rows then comes from HBM).
typedef unsigned int stream_u32x4 __attribute__((ext_vector_type(4)));
template <bool VEC>
__device__ __forceinline__ void load_slice(const uint16_t* __restrict__ row, int64_t e0, int64_t e1, int lane,
                                           Raw& raw) {
    if (!VEC) return;
#pragma unroll
    for (int j = 0; j < kVecs; ++j) {
        const int64_t e = min(slice_vec(e0, j, lane), e1 - 8);
        const stream_u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const stream_u32x4*>(row + e));
        raw[j] = make_uint4(v.x, v.y, v.z, v.w);
    }
}

// Element e + q of a group of 8 starting at e < e1 exists.  With vector
// loads, V and every range end are multiples of 8, so the whole group does.
template <bool VEC>
__device__ __forceinline__ bool in8(int64_t e, int q, int64_t e1) { return VEC || e + q < e1; }

// 8 values starting at e (< e1): from the loaded vector, or element-wise when
// V is not a multiple of 8 (no vector loads then).  Elements >= e1 read `fill`.
template <bool VEC>
__device__ __forceinline__ void vals8(const uint16_t* __restrict__ row, const uint4& raw, int64_t e, int64_t e1,
                                      float fill, float out[8]) {
    if (VEC) {
        unpack8(raw, out);
    } else {
#pragma unroll
        for (int q = 0; q < 8; ++q) out[q] = (e + q < e1) ? bf16_to_f32(row[e + q]) : fill;
    }
}

// Workgroups of the streaming kernels: at most kStreamWavesPerCU waves per
// compute unit, the items spread so that every wave takes the same count (but
// the last).  Past one workgroup per CU the count is rounded up to a whole
// number of workgroups per CU, so every CU streams the same share: a CU
// holding one workgroup more than its neighbours sets the kernel's end
// (measured on the C4 workload: 3.6 workgroups per CU 27.9 us, exactly 3 per
// CU 25.8 us).  Waves past the last item return at once.
inline unsigned stream_blocks(int64_t items, int cus) {
    const int64_t cap = (int64_t)cus * kStreamWavesPerCU;
    const int64_t per = (items + cap - 1) / cap;
    const int64_t waves = (items + per - 1) / per;
    int64_t blocks = (waves + kWavesPerBlock - 1) / kWavesPerBlock;
    if (blocks > cus) blocks = (blocks + cus - 1) / cus * cus;
    return (unsigned)blocks;
}

// Persistent wave loop over items it = gw, gw + GW, ...: the slice of item
// it + GW is loaded while item it is reduced (two register buffers).  The
// wave id is read from the first lane, so the item, row and slice indices are
// known to be wave-uniform and their arithmetic runs on the scalar unit
// (C4 stochastic acceptance 46.4 -> 46.1 us).
// Only the first a.sw waves of the grid stream (workgroups past them do side
// work).
template <bool VEC, class RowOf, class Body>
__device__ __forceinline__ void stream_items(const AcceptArgs& a, RowOf row_of, Body body) {
    const int lane = threadIdx.x & (kWave - 1);
    const uint32_t gw = blockIdx.x * kWavesPerBlock + (uint32_t)__builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
    const uint32_t GW = a.sw;
    auto lo = [&](uint32_t it) { return (int64_t)(it % a.nslice) * kSlice; };
    auto hi = [&](uint32_t it) { return min(lo(it) + kSlice, a.V); };
    auto clampi = [&](uint32_t it) { return it < a.items ? it : a.items - 1; };
    if (gw >= GW || gw >= a.items) return;
    Raw r0, r1;
    load_slice<VEC>(row_of(gw / a.nslice), lo(gw), hi(gw), lane, r0);
    for (uint32_t it = gw; it < a.items; it += 2 * GW) {
        const uint32_t n1 = clampi(it + GW), n2 = clampi(it + 2 * GW);
        load_slice<VEC>(row_of(n1 / a.nslice), lo(n1), hi(n1), lane, r1);
        body(it, r0);
        load_slice<VEC>(row_of(n2 / a.nslice), lo(n2), hi(n2), lane, r0);
        if (it + GW < a.items) body(it + GW, r1);
    }
}

// ------------------------------------------------------------------ greedy

__device__ __forceinline__ bool better(float v, int i, float bv, int bi) {
    return v > bv || (v == bv && i < bi);
}

// Lane maximum of the logits of one slice (8-element groups, v_max3 pairs).
// Missing elements (non-vector path past e1) read NaN, which fmaxf ignores.
template <bool VEC, bool FULL>
__device__ __forceinline__ float slice_max(const uint16_t* z, const Raw& raw, int64_t e0, int64_t e1, int lane) {
    float zm = -INFINITY;
#pragma unroll
    for (int j = 0; j < kVecs; ++j) {
        const int64_t e = slice_vec(e0, j, lane);
        if (FULL || e < e1) {
            float v[8];
            vals8<VEC>(z, raw[j], e, e1, __builtin_nanf(""), v);
#pragma unroll
            for (int q = 0; q < 8; q += 2) zm = fmaxf(fmaxf(zm, v[q]), v[q + 1]);
        }
    }
    return zm;
}

// (max logit, lowest index holding it) of one slice, reduced over the wave.
template <bool VEC, bool FULL>
__device__ __forceinline__ float2 slice_argmax(const uint16_t* z, const Raw& raw, int64_t e0, int64_t e1, int lane) {
    const float M = wave_max(slice_max<VEC, FULL>(z, raw, e0, e1, lane));
    // lowest index of M in the lane: scan backwards, the last hit wins
    int bi = 0x7fffffff;
#pragma unroll
    for (int j = kVecs - 1; j >= 0; --j) {
        const int64_t e = slice_vec(e0, j, lane);
        if (FULL || e < e1) {
            float v[8];
            vals8<VEC>(z, raw[j], e, e1, __builtin_nanf(""), v);
#pragma unroll
            for (int q = 7; q >= 0; --q) bi = (v[q] == M) ? (int)(e + q) : bi;
        }
    }
    return make_float2(M, __int_as_float(wave_min_i32(bi)));
}

template <bool VEC>
__global__ __launch_bounds__(kAThreads) void greedy_partial_kernel(AcceptArgs a) {
    const int lane = threadIdx.x & (kWave - 1);
    auto row_of = [&](uint32_t row) { return a.zt + (int64_t)row * a.V; };
    stream_items<VEC>(a, row_of, [&](uint32_t it, const Raw& raw) {
        const uint32_t row = it / a.nslice, c = it % a.nslice;
        const uint16_t* z = row_of(row);
        const int64_t e0 = (int64_t)c * kSlice, e1 = min(e0 + kSlice, a.V);
        const float2 r = (VEC && e1 - e0 == kSlice) ? slice_argmax<VEC, true>(z, raw, e0, e1, lane)
                                                    : slice_argmax<VEC, false>(z, raw, e0, e1, lane);
        if (lane == 0) a.stats[(int64_t)row * a.nslice + c] = r;
    });
}

// Entry `lane` of row r's (max logit, lowest index) statistics, or the
// neutral (-inf, INT_MAX) past the row's entries.
__device__ __forceinline__ float2 argmax_entry(const AcceptArgs& a, int b, int r, int lane) {
    uint32_t nst;
    const float2* st = row_stats(a, b, r, nst);
    return (uint32_t)lane < nst ? st[lane] : make_float2(-INFINITY, __int_as_float(0x7fffffff));
}

// Merged (max logit, lowest index) of row r of sequence b, for lanes of one
// wave; `first` is the row's entry `lane` (argmax_entry), loaded beforehand.
// The order of `better` is total, so the merge order does not matter.
__device__ __forceinline__ int merged_argmax(const AcceptArgs& a, int b, int r, int lane, float2 first) {
    uint32_t nst;
    const float2* st = row_stats(a, b, r, nst);
    float bv = first.x;
    int bi = __float_as_int(first.y);
    // the entries past the first 64 (many when they come from the LM-head
    // epilogue: 668 per row at V = 128256), 16 per lane per round trip
    for (int64_t c0 = lane + 64; c0 < nst; c0 += 16 * 64) {
        float2 pv[16];
#pragma unroll
        for (int q = 0; q < 16; ++q) {
            const int64_t c = c0 + q * 64;
            pv[q] = c < nst ? st[c] : make_float2(-INFINITY, __int_as_float(0x7fffffff));
        }
#pragma unroll
        for (int q = 0; q < 16; ++q) {
            const int pi = __float_as_int(pv[q].y);
            if (better(pv[q].x, pi, bv, bi)) { bv = pv[q].x; bi = pi; }
        }
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
        const float ov = __shfl_xor(bv, o, 64);
        const int oi = __shfl_xor(bi, o, 64);
        if (better(ov, oi, bv, bi)) { bv = ov; bi = oi; }
    }
    return bi;
}

__global__ __launch_bounds__(1024) void greedy_final_kernel(AcceptArgs a) {
    __shared__ int g[17], s_x[16];
    const int b = blockIdx.x;
    const int t = threadIdx.x, lane = t & 63, wv = t >> 6;
    // the drafts are loaded first, so their round trip overlaps the merge
    const int32_t xt = t < a.k ? a.x[(int64_t)b * a.k + t] : 0;
    // wave wv merges positions wv, wv+16, ... (one round for k < 16); lanes
    // stride over the slices
    const int nw = (int)(blockDim.x >> 6);
    for (int pos = wv; pos <= a.k; pos += nw) {
        const int bi = merged_argmax(a, b, pos, lane, argmax_entry(a, b, pos, lane));
        if (lane == 0) g[pos] = bi;
    }
    if (t < a.k) s_x[t] = xt;
    __syncthreads();
    if (t <= a.k) {
        // a_b = number of leading drafts equal to the target argmax
        int acc = a.k;
        for (int i = 0; i < a.k; ++i)
            if (s_x[i] != g[i]) { acc = i; break; }
        int32_t* out = a.out + (int64_t)b * (a.k + 1);
        out[t] = t < acc ? g[t] : (t == acc ? g[acc] : -1);
        if (t == 0) a.num[b] = acc;
    }
}

// ------------------------------------------------------------- stochastic

// (m, sum 2^(t - m)) of t = z * c2 over one slice, reduced over the wave:
// the wave maximum first (c2 > 0, so max t = fl(max z * c2)), then one
// exponential per element with the wave's m, so no partial sum is rescaled.
template <bool VEC, bool FULL>
__device__ __forceinline__ float2 slice_stats(const uint16_t* z, const Raw& raw, int64_t e0, int64_t e1, int lane,
                                              float c2) {
    const float M = wave_max(slice_max<VEC, FULL>(z, raw, e0, e1, lane)) * c2;
    float s = 0.0f;
    if (M != -INFINITY) {
#pragma unroll
        for (int j = 0; j < kVecs; ++j) {
            const int64_t e = slice_vec(e0, j, lane);
            if (FULL || e < e1) {
                float v[8];
                vals8<VEC>(z, raw[j], e, e1, -INFINITY, v);
#pragma unroll
                for (int q = 0; q < 8; ++q) s += __builtin_amdgcn_exp2f(fmaf(v[q], c2, -M));
            }
        }
    }
    return make_float2(M, wave_sum(s));
}

// Online merge of (max, sum 2^(t - max)) pairs.
__device__ __forceinline__ void merge_ms(float& m, float& z, float om, float oz) {
    if (om == -INFINITY) return;
    if (om > m) {
        z = (m == -INFINITY ? 0.0f : z * exp2f(m - om)) + oz;
        m = om;
    } else {
        z += oz * exp2f(om - m);
    }
}

// (M, Z) of the n statistics entries st[0..n) merged over one wave: lane l
// merges entries l, l + 64, l + 128, ... in that order (`first` is its entry
// l, loaded by the caller, or (-inf, 0) past n), then the wave combines the
// lanes.  A row given as its single merged entry gives back that entry
// exactly (the other lanes add zeros).
__device__ __forceinline__ float2 merge_row_ms(const float2* st, uint32_t n, int lane, float2 first) {
    float m = -INFINITY, z = 0.0f;
    merge_ms(m, z, first.x, first.y);
    // loads issued 8 per lane before they are merged, in entry order
    for (int64_t q0 = lane + kWave; q0 < n; q0 += 8 * kWave) {
        float2 v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int64_t q = q0 + u * kWave;
            v[u] = q < n ? st[q] : make_float2(-INFINITY, 0.0f);
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) merge_ms(m, z, v[u].x, v[u].y);
    }
    const float M = wave_max(m);
    const float Z = wave_sum(m == -INFINITY ? 0.0f : z * exp2f(m - M));
    return make_float2(M, Z);
}

template <bool VEC>
__global__ __launch_bounds__(kAThreads) void stoch_stats_kernel(AcceptArgs a) {
    const int lane = threadIdx.x & (kWave - 1);
    if (a.tsm) {
        // Target statistics from the LM-head epilogue (many entries per row):
        // merged here to one entry per row, so that every sampling block
        // reads one entry per target row.  The waves with the highest ids
        // hold the fewest items (often none), so they take the merges.
        const uint32_t gw = blockIdx.x * kWavesPerBlock + (threadIdx.x >> 6);
        const uint32_t GW = gridDim.x * kWavesPerBlock;
        const uint32_t rows = (uint32_t)a.B * (uint32_t)(a.k + 1);
        for (uint32_t m = GW - 1 - gw; m < rows; m += GW) {
            const float2* st = a.tst + (int64_t)m * a.ldtst;
            const float2 first = (uint32_t)lane < a.ntst ? st[lane] : make_float2(-INFINITY, 0.0f);
            const float2 r = merge_row_ms(st, a.ntst, lane, first);
            if (lane == 0) a.tsm[m] = r;
        }
    }
    auto row_of = [&](uint32_t row) -> const uint16_t* {
        const int64_t b = row / a.Rs;
        const int r = (int)(a.rt0 + row % a.Rs);
        return (r <= a.k) ? a.zt + (b * (a.k + 1) + r) * a.V : a.zd + (b * a.k + (r - a.k - 1)) * a.V;
    };
    // The logits at the draft tokens, which the sampling kernel's accept
    // tests need, are gathered by the workgroups past the streaming ones (64
    // (sequence, draft) pairs per wave), so the sampling kernel reads them in
    // one round trip with the statistics instead of two dependent ones (the
    // draft ids, then the logits at them).
    const uint32_t gwave = blockIdx.x * kWavesPerBlock + (threadIdx.x >> 6);
    if (a.zx && gwave >= a.sw) {
        const uint32_t pz = (gwave - a.sw) * kWave + (uint32_t)lane;
        if (pz < (uint32_t)a.B * (uint32_t)a.k) {
            const int32_t xg = a.x[pz];
            float gt = 0.0f, gd = 0.0f;
            if (xg >= 0 && xg < a.V) {
                const int64_t b = pz / (uint32_t)a.k, i = pz % (uint32_t)a.k;
                gt = bf16_to_f32(a.zt[(b * (a.k + 1) + i) * a.V + xg]);
                if (a.zd) gd = bf16_to_f32(a.zd[(b * a.k + i) * a.V + xg]);
            }
            a.zx[pz] = make_float2(gt, gd);
        }
        return;
    }
    stream_items<VEC>(a, row_of, [&](uint32_t it, const Raw& raw) {
        const uint32_t row = it / a.nslice, c = it % a.nslice;
        const uint16_t* z = row_of(row);
        const int64_t e0 = (int64_t)c * kSlice, e1 = min(e0 + kSlice, a.V);
        if (c == 0 && (row % a.Rs) == 0 && lane == 0) a.ctr[row / a.Rs] = 0u;   // ticket of the sample kernel
        const float2 r = (VEC && e1 - e0 == kSlice) ? slice_stats<VEC, true>(z, raw, e0, e1, lane, a.c2)
                                                    : slice_stats<VEC, false>(z, raw, e0, e1, lane, a.c2);
        if (lane == 0) a.stats[(int64_t)row * a.nslice + c] = r;
    });
}

// Residual (or bonus) distribution at the sampled position j.
struct Dist {
    const uint16_t* zt_row;   // target row j
    const uint16_t* zd_row;   // draft row j, or null (one-hot drafts / bonus)
    float mt, inv_zt;         // merged max and 1/sum of the target row
    float md, inv_zd;
    int64_t skip;             // element forced to zero (one-hot draft), -1 if none
    int64_t kill0;            // token tree: bit i of `kill` zeroes element kill0 + i (rejected candidates)
    uint64_t kill;
};

__device__ __forceinline__ bool killed(const Dist& d, int64_t e) {
    const uint64_t i = (uint64_t)(e - d.kill0);
    return i < 64 && ((d.kill >> i) & 1ull);
}

// Probabilities of the 8 elements at e (< e1) from loaded vectors: with a
// draft row (HAS_D) the residual max(0, p - q), else p with element `skip`
// (the one-hot draft token, or -1) set to zero.
template <bool VEC, bool HAS_D>
__device__ __forceinline__ void dist8(const Dist& d, float c2, const uint4& rt, const uint4& rd, int64_t e,
                                      int64_t e1, float r[8]) {
    float zt[8];
    vals8<VEC>(d.zt_row, rt, e, e1, 0.0f, zt);
    if constexpr (HAS_D) {
        float zd[8];
        vals8<VEC>(d.zd_row, rd, e, e1, 0.0f, zd);
#pragma unroll
        for (int q = 0; q < 8; ++q) {
            const float p = __builtin_amdgcn_exp2f(fmaf(zt[q], c2, -d.mt)) * d.inv_zt;
            const float qq = __builtin_amdgcn_exp2f(fmaf(zd[q], c2, -d.md)) * d.inv_zd;
            r[q] = in8<VEC>(e, q, e1) ? fmaxf(p - qq, 0.0f) : 0.0f;
        }
    } else {
#pragma unroll
        for (int q = 0; q < 8; ++q) {
            const float p = __builtin_amdgcn_exp2f(fmaf(zt[q], c2, -d.mt)) * d.inv_zt;
            r[q] = (in8<VEC>(e, q, e1) && e + q != d.skip && !killed(d, e + q)) ? p : 0.0f;
        }
    }
}

// The same probability for one element e < V (bit-identical to dist8).
template <bool HAS_D>
__device__ __forceinline__ float dist1(const Dist& d, float c2, int64_t e) {
    const float p = __builtin_amdgcn_exp2f(fmaf(bf16_to_f32(d.zt_row[e]), c2, -d.mt)) * d.inv_zt;
    if constexpr (HAS_D) {
        const float qq = __builtin_amdgcn_exp2f(fmaf(bf16_to_f32(d.zd_row[e]), c2, -d.md)) * d.inv_zd;
        return fmaxf(p - qq, 0.0f);
    } else {
        return (e != d.skip && !killed(d, e)) ? p : 0.0f;
    }
}

// Mass of the range [e0, e1) of at most 64 elements (e0 < e1), in double.
// The 8 vectors of the range are loaded before any is used.
template <bool VEC, bool HAS_D>
__device__ __forceinline__ double range_mass(const Dist& d, float c2, int64_t e0, int64_t e1) {
    Raw rt, rd;
    if (VEC) {
#pragma unroll
        for (int j = 0; j < kVecs; ++j) {
            const int64_t e = min(e0 + j * 8, e1 - 8);
            rt[j] = *reinterpret_cast<const uint4*>(d.zt_row + e);
            if (HAS_D) rd[j] = *reinterpret_cast<const uint4*>(d.zd_row + e);
        }
    }
    double m = 0.0;
#pragma unroll
    for (int j = 0; j < kVecs; ++j) {
        const int64_t e = e0 + j * 8;
        if (e < e1) {
            float r[8];
            dist8<VEC, HAS_D>(d, c2, rt[j], rd[j], e, e1, r);
            m += (((double)r[0] + (double)r[1]) + ((double)r[2] + (double)r[3])) +
                 (((double)r[4] + (double)r[5]) + ((double)r[6] + (double)r[7]));
        }
    }
    return m;
}

// Masses of the kAThreads ranges of kPerThread elements of chunk ch, read with
// coalesced loads: wave wv covers the chunk's elements [wv*4096, (wv+1)*4096)
// in kVecs loads of 512 (16 bytes per lane, consecutive lanes on consecutive
// 16-byte pieces, so one load instruction reads 1 KiB contiguous).  The 8 lanes
// that share a range add their sums by xor exchanges in a fixed order, and the
// first of them stores the mass of range wv*64 + j*8 + lane/8 into s_rm.  Called
// by the whole block; s_rm is complete after the caller's next barrier.
template <bool VEC, bool HAS_D>
__device__ __forceinline__ void chunk_masses(const Dist& d, float c2, int64_t ch, int64_t V, int t,
                                             double* s_rm) {
    static_assert(kChunk == (int64_t)kWavesPerBlock * kVecs * kWave * 8 && kPerThread == 8 * 8,
                  "a range is 8 lanes of one load");
    const int lane = t & (kWave - 1), wv = t / kWave;
    const int64_t base = ch * kChunk + (int64_t)wv * (kVecs * kWave * 8) + (int64_t)lane * 8;
    Raw rt, rd;
    if (VEC) {
#pragma unroll
        for (int j = 0; j < kVecs; ++j) {
            const int64_t e = base + (int64_t)j * kWave * 8;
            if (e < V) {
                rt[j] = *reinterpret_cast<const uint4*>(d.zt_row + e);
                if (HAS_D) rd[j] = *reinterpret_cast<const uint4*>(d.zd_row + e);
            }
        }
    }
#pragma unroll
    for (int j = 0; j < kVecs; ++j) {
        const int64_t e = base + (int64_t)j * kWave * 8;
        double m = 0.0;
        if (e < V) {
            float r[8];
            dist8<VEC, HAS_D>(d, c2, rt[j], rd[j], e, V, r);
            m = (((double)r[0] + (double)r[1]) + ((double)r[2] + (double)r[3])) +
                (((double)r[4] + (double)r[5]) + ((double)r[6] + (double)r[7]));
        }
        m += __shfl_xor(m, 1);
        m += __shfl_xor(m, 2);
        m += __shfl_xor(m, 4);
        if ((lane & 7) == 0) s_rm[wv * (kVecs * 8) + j * 8 + (lane >> 3)] = m;
    }
}

// Block-wide scan of one double per thread, in thread order: the thread's
// interval [lo, hi) of the running sum and the block total.  Intervals of
// consecutive threads tile exactly (hi of thread t is bit-identical to lo of
// thread t + 1), so a value in [0, total) has exactly one owner, and the
// owner's own value is positive.  `sh` holds kWavesPerBlock doubles.
__device__ __forceinline__ void block_scan_d(double v, double* sh, double& lo, double& hi, double& total) {
    const int lane = threadIdx.x & (kWave - 1), wv = threadIdx.x >> 6;
    double incl = v;
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
        const double y = __shfl_up(incl, o, kWave);
        if (lane >= o) incl += y;
    }
    double excl = __shfl_up(incl, 1, kWave);
    if (lane == 0) excl = 0.0;
    __syncthreads();                       // sh may still be read by a previous scan
    if (lane == kWave - 1) sh[wv] = incl;
    __syncthreads();
    double before = 0.0;
    for (int q = 0; q < wv; ++q) before += sh[q];
    double tot = before;
    for (int q = wv; q < kWavesPerBlock; ++q) tot += sh[q];
    lo = before + excl;
    hi = before + incl;
    total = tot;
}

// Owner of `target` among the block's intervals (base + [lo, hi)): writes the
// owner's index (always in [0, blockDim.x)) and base + lo to shared memory.
// If rounding left no owner (target at or past the end), the last thread with
// positive mass owns it; with no positive mass at all (non-finite logits),
// thread 0 does.
__device__ __forceinline__ void find_owner(double v, double lo, double hi, double base, double target, int* s_own,
                                           double* s_base, int* s_lastpos) {
    if (threadIdx.x == 0) { *s_own = -1; *s_lastpos = -1; }
    __syncthreads();
    const double blo = base + lo, bhi = base + hi;
    if (blo <= target && target < bhi) { *s_own = threadIdx.x; *s_base = blo; }
    if (v > 0.0) atomicMax(s_lastpos, (int)threadIdx.x);
    __syncthreads();
    const int lastpos = *s_lastpos;
    if (*s_own < 0 && (int)threadIdx.x == (lastpos >= 0 ? lastpos : 0)) { *s_own = threadIdx.x; *s_base = blo; }
    __syncthreads();
}

__device__ __forceinline__ void wait_stores() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

__device__ __forceinline__ void store_coherent(double* p, double v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ double load_coherent(const double* p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

constexpr int kRunRegs = 16;   // range masses a thread keeps in registers (nchunk <= 16: V <= 262144)

// The inverse-CDF search down to one 64-element range, by the whole last
// block of a sequence in one round trip: its residual masses fm[0 .. nchunk * 256),
// one per 64-element range in vocabulary order (range th of chunk ch at
// ch * 256 + th, stored by every block of the sequence), are read in runs of
// nchunk consecutive ranges per thread; the runs are summed in order and
// scanned across the block, which gives the total R; the thread whose run
// holds target = u * R walks it range by range.  Writes the chosen range
// (index into fm) to *s_rng and the mass before it to *s_base; where rounding
// leaves target past every interval, the last range with positive mass is
// taken, and range 0 where there is none (R == 0 or not finite).  Returns R.
__device__ __forceinline__ double locate_range(const double* fm, int64_t nchunk, float u, double* sh, int* s_own,
                                               double* s_base, int* s_lastpos, int* s_rng) {
    const int t = threadIdx.x;
    const int64_t r0 = (int64_t)t * nchunk;
    const bool in_regs = nchunk <= kRunRegs;
    double v[kRunRegs];
    double run = 0.0;
    if (in_regs) {
#pragma unroll
        for (int i = 0; i < kRunRegs; ++i) v[i] = i < nchunk ? load_coherent(fm + r0 + i) : 0.0;
#pragma unroll
        for (int i = 0; i < kRunRegs; ++i) run += v[i];
    } else {
        for (int64_t i = 0; i < nchunk; ++i) run += load_coherent(fm + r0 + i);
    }
    double lo, hi, R;
    block_scan_d(run, sh, lo, hi, R);
    const double target = (double)u * R;
    find_owner(run, lo, hi, 0.0, target, s_own, s_base, s_lastpos);
    if (t == *s_own) {
        double cum = *s_base, last_base = cum, pick_base = cum;
        int64_t pick = -1, lastpos = -1;
        auto visit = [&](int64_t i, double m) {
            const double nx = cum + m;
            if (m > 0.0) { lastpos = i; last_base = cum; }
            if (pick < 0 && cum <= target && target < nx) { pick = i; pick_base = cum; }
            cum = nx;
        };
        if (in_regs) {
#pragma unroll
            for (int i = 0; i < kRunRegs; ++i)
                if (i < nchunk) visit(i, v[i]);
        } else {
            for (int64_t i = 0; i < nchunk; ++i) visit(i, load_coherent(fm + r0 + i));
        }
        if (pick < 0) {
            pick = lastpos >= 0 ? lastpos : 0;
            pick_base = lastpos >= 0 ? last_base : *s_base;
        }
        *s_rng = R > 0.0 ? (int)(r0 + pick) : 0;
        *s_base = R > 0.0 ? pick_base : 0.0;
    }
    __syncthreads();
    return R;
}


// Sampling from the residual (or bonus) distribution of position j by inverse
// CDF in vocabulary order: every block stores the masses of its chunk's 256
// ranges of 64 elements (thread t owns range t); the last block of the
// sequence finds the range holding u*R (locate_range), then the element
// within the range (one lane each).
template <bool VEC>
__global__ __launch_bounds__(kAThreads) void stoch_sample_kernel(AcceptArgs a) {
    __shared__ float sM[33], sZ[33];
    __shared__ double s_rm[kAThreads];
    __shared__ int s_acc[16], s_x[16];
    __shared__ int s_j, s_last, s_rng;
    __shared__ float s_uk;
    __shared__ double sh[kWavesPerBlock];
    __shared__ int s_own, s_lastpos;
    __shared__ double s_base;
    const int64_t c = blockIdx.x;
    const int b = blockIdx.y;
    const int t = threadIdx.x;
    const int lane = t & 63, wv = t >> 6;
    const int k = a.k;

    // The operands of the accept tests are loaded first (draft id, then the
    // two logits at it), so their round trips overlap the statistics merge;
    // so are the resampling uniform and the drafts the outputs repeat.
    // With a statistics pass the logits at the draft tokens were gathered by
    // it, and load with the draft ids in one round trip.
    int32_t xi = -1;
    float zx_t = 0.0f, zx_d = 0.0f, ui = 0.0f;
    if (t <= k) ui = a.u[(int64_t)b * (k + 1) + t];
    if (t < k) {
        xi = a.x[(int64_t)b * k + t];
        if (a.zx) {
            const float2 g = a.zx[(int64_t)b * k + t];
            zx_t = g.x;
            zx_d = g.y;
        } else if (xi >= 0 && xi < a.V) {
            zx_t = bf16_to_f32(a.zt[((int64_t)b * (k + 1) + t) * a.V + xi]);
            if (a.zd) zx_d = bf16_to_f32(a.zd[((int64_t)b * k + t) * a.V + xi]);
        }
    }

    // 1. merge the slice statistics of every row of sequence b: wave wv takes
    //    rows wv, wv+4, ...; lanes stride over slices (the first slice of
    //    every row is loaded up front); fixed reduction order.
    constexpr int kRowsPerWave = (33 + kWavesPerBlock - 1) / kWavesPerBlock;   // R <= 2*16+1
    float2 first[kRowsPerWave];
#pragma unroll
    for (int i = 0; i < kRowsPerWave; ++i) {
        const int r = wv + i * kWavesPerBlock;
        first[i] = make_float2(-INFINITY, 0.0f);
        if (r < (int)a.R) {
            uint32_t nst;
            const float2* st = row_stats(a, b, r, nst);
            if ((uint32_t)lane < nst) first[i] = st[lane];
        }
    }
#pragma unroll
    for (int i = 0; i < kRowsPerWave; ++i) {
        const int r = wv + i * kWavesPerBlock;
        if (r < (int)a.R) {
            uint32_t nst;
            const float2* st = row_stats(a, b, r, nst);
            const float2 mz = merge_row_ms(st, nst, lane, first[i]);
            if (lane == 0) { sM[r] = mz.x; sZ[r] = mz.y; }
        }
    }
    if (t < k) s_x[t] = xi;
    if (t == k) s_uk = ui;
    __syncthreads();

    // 2. accept tests of the k drafts, evaluated in parallel (identical in
    //    every block of sequence b); the first rejection j is then a scan.
    //    t - M is formed exactly in double (bf16 * fp32 fits in 53 bits).
    if (t < k) {
        double p = 0.0, q = 0.0;
        if (xi >= 0 && xi < a.V) {
            p = exp2((double)zx_t * (double)a.c2 - (double)sM[t]) / (double)sZ[t];
            q = a.zd ? exp2((double)zx_d * (double)a.c2 - (double)sM[k + 1 + t]) / (double)sZ[k + 1 + t] : 1.0;
        }
        s_acc[t] = ((double)ui * q < p) ? 1 : 0;
    }
    __syncthreads();
    if (t == 0) {
        int j = k;
        for (int i = 0; i < k; ++i)
            if (!s_acc[i]) { j = i; break; }
        s_j = j;
    }
    __syncthreads();
    const int j = s_j;

    Dist d;
    d.zt_row = a.zt + ((int64_t)b * (k + 1) + j) * a.V;
    d.mt = sM[j];
    d.inv_zt = 1.0f / sZ[j];
    d.zd_row = nullptr;
    d.md = 0.0f;
    d.inv_zd = 0.0f;
    d.skip = -1;
    d.kill0 = 0;
    d.kill = 0;
    if (j < k) {
        if (a.zd) {
            d.zd_row = a.zd + ((int64_t)b * k + j) * a.V;
            d.md = sM[k + 1 + j];
            d.inv_zd = 1.0f / sZ[k + 1 + j];
        } else {
            d.skip = s_x[j];
        }
    }

    double* fm = a.finem + (int64_t)b * a.nchunk * kAThreads;   // range masses
    auto range_of = [&](int64_t ch, int th, int64_t& e0, int64_t& e1) {
        e0 = ch * kChunk + (int64_t)th * kPerThread;
        e1 = min(e0 + kPerThread, a.V);
    };
    // the mass of this thread's range of chunk ch (every thread of the block calls it)
    auto mass_of = [&](int64_t ch) {
        __syncthreads();                     // s_rm's previous readers are done
        if (d.zd_row) chunk_masses<VEC, true>(d, a.c2, ch, a.V, t, s_rm);
        else chunk_masses<VEC, false>(d, a.c2, ch, a.V, t, s_rm);
        __syncthreads();
        return s_rm[t];
    };

    // 3. this block's range masses, stored device-coherently (relaxed
    //    agent-scope atomic stores, written through the L2) and acknowledged
    //    before the ticket is taken; the last block reads them with
    //    device-coherent loads.  No agent-scope fence is needed (on this chip
    //    such a fence writes back and invalidates the XCD's whole L2).
    {
        const double m = mass_of(c);
        store_coherent(fm + c * kAThreads + t, m);
        wait_stores();
        __syncthreads();
        if (t == 0) {
            const unsigned int ticket = __hip_atomic_fetch_add(a.ctr + b, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            s_last = (ticket == (unsigned int)(a.nchunk - 1));
        }
        __syncthreads();
        if (!s_last) return;
    }

    // 4. last block of sequence b: the range of 64 elements holding u*R.
    double R = locate_range(fm, a.nchunk, s_uk, sh, &s_own, &s_base, &s_lastpos, &s_rng);
    if (!(R > 0.0)) {
        // The residual vanished (p_j == q_j wherever it is positive): sample
        // p_j itself.  This block recomputes every range mass.
        d.zd_row = nullptr;
        d.skip = -1;
        for (int64_t ch = 0; ch < a.nchunk; ++ch) store_coherent(fm + ch * kAThreads + t, mass_of(ch));
        wait_stores();
        __syncthreads();
        R = locate_range(fm, a.nchunk, s_uk, sh, &s_own, &s_base, &s_lastpos, &s_rng);
    }
    const double target = (double)s_uk * R;

    // Then the element within the range (wave 0, one element per lane).
    if (wv == 0) {
        int64_t e0, e1;
        range_of(s_rng / kAThreads, s_rng % kAThreads, e0, e1);
        const double base3 = s_base;
        const int64_t e = e0 + lane;
        const float r = e < e1 ? (d.zd_row ? dist1<true>(d, a.c2, e) : dist1<false>(d, a.c2, e)) : 0.0f;
        double incl = (double)r;
#pragma unroll
        for (int o = 1; o < kWave; o <<= 1) {
            const double y = __shfl_up(incl, o, kWave);
            if (lane >= o) incl += y;
        }
        double excl = __shfl_up(incl, 1, kWave);
        if (lane == 0) excl = 0.0;
        const unsigned long long own = __ballot(base3 + excl <= target && target < base3 + incl);
        const unsigned long long pos = __ballot(r > 0.0f);
        int pick;
        if (own) pick = __ffsll((long long)own) - 1;
        else if (pos) pick = 63 - __builtin_clzll(pos);          // rounding: last positive element
        else pick = 0;
        if (lane <= k) {
            int32_t* out = a.out + (int64_t)b * (k + 1);
            out[lane] = lane < j ? s_x[lane] : (lane == j ? (int)min(e0 + pick, a.V - 1) : -1);
            if (lane == 0) {
                a.num[b] = j;
                a.ctr[b] = 0u;
            }
        }
    }
}

// ------------------------------------------------------------- token tree
//
// Tree mode: the N drafted nodes of a sequence form a tree (parent[n] in
// [-1, n), -1 for candidates of the first new position); target row 0 scores
// the first new position and row n+1 the position after node n, so a
// sequence has N+1 target rows, whose statistics the streaming kernels above
// compute as for k = N.  The children of a node are its candidates, tested
// in index order.  A node whose parent is out of range is never reached.

constexpr int kMaxTree = 64;   // nodes per sequence


// Writes sequence b's outputs: the tokens of the accepted path, then the
// emitted token, -1 padded to N+1; the path's node indices, -1 padded to N.
__device__ __forceinline__ void tree_outputs(const AcceptArgs& a, int b, const int* path, const int* x, int depth,
                                             int token, int i0, int step) {
    const int N = a.k;
    for (int i = i0; i <= N; i += step) {
        a.out[(int64_t)b * (N + 1) + i] = i < depth ? x[path[i]] : (i == depth ? token : -1);
        if (i < N) a.nodes[(int64_t)b * N + i] = i < depth ? path[i] : -1;
    }
}

// Greedy walk (one block per sequence): the argmax of every row from its
// slice statistics, then from the root the first child whose token is the
// current row's argmax, until no child matches; that argmax is emitted.
__global__ __launch_bounds__(1024) void tree_greedy_kernel(AcceptArgs a) {
    __shared__ int g[kMaxTree + 1];
    __shared__ int s_par[kMaxTree], s_x[kMaxTree], s_path[kMaxTree];
    __shared__ int s_depth, s_tok;
    const int b = blockIdx.x;
    const int t = threadIdx.x, lane = t & 63, wv = t >> 6;
    const int N = a.k;
    // the tree and the first statistics entry of every row of the wave are
    // loaded before anything waits for them (one round trip for all); the
    // tree reaches shared memory after the merge
    int par = -2, xv = -1;
    if (t < N) {
        par = a.parent[(int64_t)b * N + t];
        xv = a.x[(int64_t)b * N + t];
    }
    // rows over the 16 waves: wave wv merges rows wv, wv+16, ...
    constexpr int kGreedyWaves = 1024 / kWave;
    constexpr int kRowsPerWaveG = (kMaxTree + 1 + kGreedyWaves - 1) / kGreedyWaves;
    float2 first[kRowsPerWaveG];
#pragma unroll
    for (int i = 0; i < kRowsPerWaveG; ++i) {
        const int r = wv + i * kGreedyWaves;
        first[i] = r <= N ? argmax_entry(a, b, r, lane) : make_float2(-INFINITY, __int_as_float(0x7fffffff));
    }
#pragma unroll
    for (int i = 0; i < kRowsPerWaveG; ++i) {
        const int r = wv + i * kGreedyWaves;
        if (r > N) break;
        const int bi = merged_argmax(a, b, r, lane, first[i]);
        if (lane == 0) g[r] = bi;
    }
    if (t < N) {
        s_par[t] = par;
        s_x[t] = xv;
    }
    __syncthreads();
    if (t == 0) {
        int cur = -1, depth = 0;
        for (;;) {
            const int gv = g[cur + 1];
            int nxt = -1;
            for (int n = cur + 1; n < N; ++n)
                if (s_par[n] == cur && s_x[n] == gv) { nxt = n; break; }
            if (nxt < 0) break;
            s_path[depth++] = nxt;
            cur = nxt;
        }
        s_depth = depth;
        s_tok = g[cur + 1];
    }
    __syncthreads();
    tree_outputs(a, b, s_path, s_x, s_depth, s_tok, t, blockDim.x);
    if (t == 0) a.num[b] = s_depth;
}

// Sampling walk, block (chunk c, sequence b).  Every block merges the row
// statistics, gets every candidate's target probability in parallel (one
// round trip for all of them) and walks the tree identically: at the current
// node, child n with token x is accepted iff u[n] (1 - S) < P(x), S the mass
// of the tokens already rejected there (a repeated token has P = 0); on
// acceptance the walk moves to n, else x is removed.  Where every child is
// rejected (or there is none) the final draw comes from P with the removed
// tokens zeroed: each block sums its chunk as for chains (the removed tokens
// of a 64-element range are a bit mask), and the last block of the sequence
// searches the chunk, the range and the element holding u[N] R.
template <bool VEC>
__global__ __launch_bounds__(kAThreads) void tree_sample_kernel(AcceptArgs a) {
    __shared__ float sM[kMaxTree + 1], sZ[kMaxTree + 1];
    __shared__ int s_par[kMaxTree], s_x[kMaxTree], s_path[kMaxTree], s_kill[kMaxTree];
    __shared__ double s_p[kMaxTree];
    __shared__ float s_u[kMaxTree + 1];
    __shared__ int s_f, s_depth, s_nkill, s_last, s_rng;
    __shared__ double sh[kWavesPerBlock];
    __shared__ int s_own, s_lastpos;
    __shared__ double s_base;
    const int64_t c = blockIdx.x;
    const int b = blockIdx.y;
    const int t = threadIdx.x;
    const int lane = t & 63, wv = t >> 6;
    const int N = a.k;

    // the tree, the uniforms, the first statistics entries and the
    // candidates' logits are loaded before anything waits for them, so their
    // round trips overlap (the logits' addresses need the tree); they reach
    // shared memory after the merge
    int par = -2, xv = -1;
    float uv = 0.0f;
    if (t < N) {
        par = a.parent[(int64_t)b * N + t];
        xv = a.x[(int64_t)b * N + t];
    }
    if (t <= N) uv = a.u[(int64_t)b * (N + 1) + t];
    // wave wv merges rows wv, wv+4, ...: the first entry of every one of its
    // rows is loaded before any is merged (one round trip for all of them),
    // then each lane merges its entries in index order
    constexpr int kTreeRowsPerWave = (kMaxTree + 1 + kWavesPerBlock - 1) / kWavesPerBlock;
    float2 first[kTreeRowsPerWave];
#pragma unroll
    for (int i = 0; i < kTreeRowsPerWave; ++i) {
        const int r = wv + i * kWavesPerBlock;
        first[i] = make_float2(-INFINITY, 0.0f);
        if (r <= N) {
            uint32_t nst;
            const float2* st = row_stats(a, b, r, nst);
            if ((uint32_t)lane < nst) first[i] = st[lane];
        }
    }
    float zx = 0.0f;
    bool ok = false;
    if (t < N) {
        ok = par >= -1 && par < t && xv >= 0 && xv < a.V;
        if (ok) zx = bf16_to_f32(a.zt[((int64_t)b * (N + 1) + par + 1) * a.V + xv]);
    }
#pragma unroll
    for (int i = 0; i < kTreeRowsPerWave; ++i) {
        const int r = wv + i * kWavesPerBlock;
        if (r > N) break;
        uint32_t nst;
        const float2* st = row_stats(a, b, r, nst);
        const float2 mz = merge_row_ms(st, nst, lane, first[i]);
        if (lane == 0) { sM[r] = mz.x; sZ[r] = mz.y; }
    }
    if (t < N) {
        s_par[t] = par;
        s_x[t] = xv;
    }
    if (t <= N) s_u[t] = uv;
    __syncthreads();
    // every candidate's probability under its parent's row; t - M is formed
    // exactly in double (bf16 * fp32 fits in 53 bits), as for chains
    if (t < N) s_p[t] = ok ? exp2((double)zx * (double)a.c2 - (double)sM[par + 1]) / (double)sZ[par + 1] : 0.0;
    __syncthreads();
    if (t == 0) {
        int cur = -1, depth = 0, nk = 0;
        for (;;) {
            double S = 0.0;
            int nxt = -1;
            nk = 0;
            for (int n = cur + 1; n < N; ++n) {
                if (s_par[n] != cur) continue;
                const int x = s_x[n];
                bool valid = x >= 0 && x < a.V;
                for (int i = 0; i < nk && valid; ++i) valid = s_kill[i] != x;
                const double px = valid ? s_p[n] : 0.0;
                if ((double)s_u[n] * (1.0 - S) < px) { nxt = n; break; }
                if (valid) {
                    s_kill[nk++] = x;
                    S += px;
                }
            }
            if (nxt < 0) break;
            s_path[depth++] = nxt;
            cur = nxt;
        }
        s_f = cur;
        s_depth = depth;
        s_nkill = nk;
    }
    __syncthreads();
    const int f = s_f;
    int nk = s_nkill;

    Dist d;
    d.zt_row = a.zt + ((int64_t)b * (N + 1) + f + 1) * a.V;
    d.mt = sM[f + 1];
    d.inv_zt = 1.0f / sZ[f + 1];
    d.zd_row = nullptr;
    d.md = 0.0f;
    d.inv_zd = 0.0f;
    d.skip = -1;
    auto killed_in = [&](int64_t e0, Dist& dd) {     // the removed tokens of the range [e0, e0 + 64)
        dd.kill0 = e0;
        dd.kill = 0;
        for (int i = 0; i < nk; ++i) {
            const uint64_t off = (uint64_t)((int64_t)s_kill[i] - e0);
            if (off < 64) dd.kill |= 1ull << off;
        }
    };
    double* fm = a.finem + (int64_t)b * a.nchunk * kAThreads;
    auto range_of = [&](int64_t ch, int th, int64_t& e0, int64_t& e1) {
        e0 = ch * kChunk + (int64_t)th * kPerThread;
        e1 = min(e0 + kPerThread, a.V);
    };
    auto mass_of = [&](int64_t ch) {
        int64_t e0, e1;
        range_of(ch, t, e0, e1);
        if (e0 >= a.V) return 0.0;
        Dist dd = d;
        killed_in(e0, dd);
        return range_mass<VEC, false>(dd, a.c2, e0, e1);
    };
    {
        store_coherent(fm + c * kAThreads + t, mass_of(c));
        wait_stores();
        __syncthreads();
        if (t == 0) {
            const unsigned int ticket = __hip_atomic_fetch_add(a.ctr + b, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            s_last = (ticket == (unsigned int)(a.nchunk - 1));
        }
        __syncthreads();
        if (!s_last) return;
    }
    double R = locate_range(fm, a.nchunk, s_u[N], sh, &s_own, &s_base, &s_lastpos, &s_rng);
    if (!(R > 0.0)) {
        // the removed tokens held all the mass: draw from P itself
        nk = 0;
        for (int64_t ch = 0; ch < a.nchunk; ++ch) store_coherent(fm + ch * kAThreads + t, mass_of(ch));
        wait_stores();
        __syncthreads();
        R = locate_range(fm, a.nchunk, s_u[N], sh, &s_own, &s_base, &s_lastpos, &s_rng);
    }
    const double target = (double)s_u[N] * R;
    if (wv == 0) {
        int64_t e0, e1;
        range_of(s_rng / kAThreads, s_rng % kAThreads, e0, e1);
        const double base3 = s_base;
        Dist dd = d;
        killed_in(e0, dd);
        const int64_t e = e0 + lane;
        const float r = e < e1 ? dist1<false>(dd, a.c2, e) : 0.0f;
        double incl = (double)r;
#pragma unroll
        for (int o = 1; o < kWave; o <<= 1) {
            const double y = __shfl_up(incl, o, kWave);
            if (lane >= o) incl += y;
        }
        double excl = __shfl_up(incl, 1, kWave);
        if (lane == 0) excl = 0.0;
        const unsigned long long own = __ballot(base3 + excl <= target && target < base3 + incl);
        const unsigned long long pos = __ballot(r > 0.0f);
        int pick;
        if (own) pick = __ffsll((long long)own) - 1;
        else if (pos) pick = 63 - __builtin_clzll(pos);
        else pick = 0;
        tree_outputs(a, b, s_path, s_x, s_depth, (int)min(e0 + pick, a.V - 1), lane, kWave);
        if (lane == 0) {
            a.num[b] = s_depth;
            a.ctr[b] = 0u;
        }
    }
}

// Clears the sample kernel's tickets when no statistics kernel runs (target
// statistics given and no draft logits to stream).
__global__ __launch_bounds__(256) void clear_tickets_kernel(unsigned int* ctr, int n) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) ctr[i] = 0u;
}

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mutex;
void* g_scratch_ptr[kMaxDevices] = {};
std::atomic<int> g_cus[kMaxDevices];

// Compute units of the current device (256 on MI355X), looked up once per
// device; the streaming grids are sized from it.
hipError_t device_cus(int* cus) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    int n = g_cus[dev].load(std::memory_order_relaxed);
    if (n <= 0) {
        e = hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev);
        if (e != hipSuccess) return e;
        if (n <= 0) return hipErrorInvalidDevice;
        g_cus[dev].store(n, std::memory_order_relaxed);
    }
    *cus = n;
    return hipSuccess;
}

}  // namespace

hipError_t accept_scratch(void** ptr) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    if (g_scratch_ptr[dev] == nullptr) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (p == nullptr) return hipErrorInvalidSymbol;
        g_scratch_ptr[dev] = p;
    }
    *ptr = g_scratch_ptr[dev];
    return hipSuccess;
}

hipError_t launch_accept(const AcceptPlan& p, const uint16_t* zt, const uint16_t* zd, const int32_t* x,
                         const float* u, int64_t B, int64_t k, int64_t V, float temperature,
                         int32_t* out_tokens, int32_t* num_accepted, void* workspace, hipStream_t stream,
                         const float2* tstats, int64_t n_tstats, int64_t ld_tstats) {
    int cus = 0;
    if (hipError_t e = device_cus(&cus); e != hipSuccess) return e;
    AcceptArgs a{};
    a.tst = tstats; a.ntst = (uint32_t)n_tstats; a.ldtst = ld_tstats; a.tsm = nullptr;
    char* ws = reinterpret_cast<char*>(workspace);
    a.zt = zt; a.zd = zd; a.x = x; a.u = u; a.out = out_tokens; a.num = num_accepted;
    a.stats = reinterpret_cast<float2*>(ws + p.stats_off);
    a.finem = reinterpret_cast<double*>(ws + p.fine_off);
    a.ctr = reinterpret_cast<unsigned int*>(ws + p.ctr_off);
    a.V = V; a.nchunk = p.nchunk; a.nslice = (uint32_t)p.nschunk; a.B = (int)B; a.k = (int)k;
    const bool vec = (V % 8 == 0) && ((uintptr_t)zt % 16 == 0) && (zd == nullptr || (uintptr_t)zd % 16 == 0);
    a.rt0 = tstats ? (uint32_t)(k + 1) : 0u;
    if (temperature == 0.0f) {
        a.R = (uint32_t)(k + 1);
        a.Rs = a.R - a.rt0;
        a.c2 = 0.0f;
        a.items = (uint32_t)(B * a.Rs * p.nschunk);
        if (a.items > 0) {
            const unsigned g1 = stream_blocks(a.items, cus);
            a.sw = g1 * kWavesPerBlock;
            if (vec) hipLaunchKernelGGL(greedy_partial_kernel<true>, dim3(g1), dim3(kAThreads), 0, stream, a);
            else hipLaunchKernelGGL(greedy_partial_kernel<false>, dim3(g1), dim3(kAThreads), 0, stream, a);
            hipError_t e = hipGetLastError();
            if (e != hipSuccess) return e;
        }
        // one wave per position (k + 1 <= 17 positions, at most 16 waves)
        const unsigned fw = (unsigned)(k + 1 < 16 ? k + 1 : 16);
        hipLaunchKernelGGL(greedy_final_kernel, dim3((unsigned)B), dim3(64 * fw), 0, stream, a);
        return hipGetLastError();
    }
    a.R = (uint32_t)((k + 1) + (zd ? k : 0));
    a.Rs = a.R - a.rt0;
    a.c2 = (float)(1.4426950408889634 / (double)temperature);
    a.items = (uint32_t)(B * a.Rs * p.nschunk);
    // with target statistics and streamed draft rows, the statistics kernel
    // merges the target rows' entries into the statistics area after the
    // streamed rows' (B*Rs*nslice + B*(k+1) <= B*R*nslice entries)
    if (tstats && a.items > 0) a.tsm = a.stats + (int64_t)B * a.Rs * p.nschunk;
    if (a.items > 0) {
        const unsigned g1 = stream_blocks(a.items, cus);
        a.sw = g1 * kWavesPerBlock;
        // workgroups past the streaming ones gather the logits at the draft
        // tokens, 64 (sequence, draft) pairs per wave
        a.zx = reinterpret_cast<float2*>(ws + p.zx_off);
        const unsigned gz = (unsigned)((B * k + kAThreads - 1) / kAThreads);
        if (vec) hipLaunchKernelGGL(stoch_stats_kernel<true>, dim3(g1 + gz), dim3(kAThreads), 0, stream, a);
        else hipLaunchKernelGGL(stoch_stats_kernel<false>, dim3(g1 + gz), dim3(kAThreads), 0, stream, a);
    } else {
        hipLaunchKernelGGL(clear_tickets_kernel, dim3((unsigned)((B + 255) / 256)), dim3(256), 0, stream, a.ctr,
                           (int)B);
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    dim3 g2((unsigned)p.nchunk, (unsigned)B);
    if (vec) hipLaunchKernelGGL(stoch_sample_kernel<true>, g2, dim3(kAThreads), 0, stream, a);
    else hipLaunchKernelGGL(stoch_sample_kernel<false>, g2, dim3(kAThreads), 0, stream, a);
    return hipGetLastError();
}

hipError_t launch_accept_tree(const AcceptPlan& p, const uint16_t* zt, const int32_t* parent, const int32_t* x,
                              const float* u, int64_t B, int64_t N, int64_t V, float temperature,
                              int32_t* out_tokens, int32_t* accepted_nodes, int32_t* num_accepted, void* workspace,
                              hipStream_t stream) {
    int cus = 0;
    if (hipError_t e = device_cus(&cus); e != hipSuccess) return e;
    AcceptArgs a{};
    char* ws = reinterpret_cast<char*>(workspace);
    a.zt = zt; a.zd = nullptr; a.x = x; a.u = u; a.out = out_tokens; a.num = num_accepted;
    a.parent = parent; a.nodes = accepted_nodes;
    a.stats = reinterpret_cast<float2*>(ws + p.stats_off);
    a.finem = reinterpret_cast<double*>(ws + p.fine_off);
    a.ctr = reinterpret_cast<unsigned int*>(ws + p.ctr_off);
    a.tst = nullptr; a.ntst = 0; a.ldtst = 0;
    a.V = V; a.nchunk = p.nchunk; a.nslice = (uint32_t)p.nschunk; a.B = (int)B; a.k = (int)N;
    a.R = a.Rs = (uint32_t)(N + 1);
    a.rt0 = 0;
    a.items = (uint32_t)(B * a.Rs * p.nschunk);
    const bool vec = (V % 8 == 0) && ((uintptr_t)zt % 16 == 0);
    const unsigned g1 = stream_blocks(a.items, cus);
    a.sw = g1 * kWavesPerBlock;
    if (temperature == 0.0f) {
        a.c2 = 0.0f;
        if (vec) hipLaunchKernelGGL(greedy_partial_kernel<true>, dim3(g1), dim3(kAThreads), 0, stream, a);
        else hipLaunchKernelGGL(greedy_partial_kernel<false>, dim3(g1), dim3(kAThreads), 0, stream, a);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        hipLaunchKernelGGL(tree_greedy_kernel, dim3((unsigned)B), dim3(1024), 0, stream, a);
        return hipGetLastError();
    }
    a.c2 = (float)(1.4426950408889634 / (double)temperature);
    if (vec) hipLaunchKernelGGL(stoch_stats_kernel<true>, dim3(g1), dim3(kAThreads), 0, stream, a);
    else hipLaunchKernelGGL(stoch_stats_kernel<false>, dim3(g1), dim3(kAThreads), 0, stream, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    dim3 g2((unsigned)p.nchunk, (unsigned)B);
    if (vec) hipLaunchKernelGGL(tree_sample_kernel<true>, g2, dim3(kAThreads), 0, stream, a);
    else hipLaunchKernelGGL(tree_sample_kernel<false>, g2, dim3(kAThreads), 0, stream, a);
    return hipGetLastError();
}

}  // namespace specfp8
