// FP8 KV-cache write: the new tokens' key and value heads, quantized to E4M3
// and scattered to their cache slots (section 3.2: an FP8 KV cache holds half
// the bytes of a bf16 one).
//
// The cache is slot-major, [num_slots][H][D] codes, which is the paged layout
// [blocks][block_size][H][D] for any block size (slot = block * block_size +
// offset).  One (token, head) row of D values is owned by a group of G lanes
// (G = D/8 rounded up to a power of two, at most 64): every lane holds 8 values
// from one 16-byte load, the group reduces max|v| with lane exchanges inside
// the wave, and each lane writes its 8 codes as one 8-byte store.  A wave
// therefore covers 64/G rows, a 256-thread block 256/G rows; blockIdx.y picks
// keys (0) or values (1).  Traffic is the algorithmic 2 bytes read and 1 byte
// written per element plus 4 bytes of scale per row in the per-row mode.
#include "device_common.hpp"
#include "kernels.hpp"

namespace specfp8 {

namespace {

constexpr int kKvThreads = 256;

struct KvSide {
    const uint16_t* x;   // bf16 [T][ld_x]; head h of token t at x + t*ld_x + h*D
    int64_t ld_x;
    float* scale;        // per-row: [num_slots][H] (written); per-tensor: [1] (read)
    uint8_t* cache;      // [num_slots][H][D]
};

struct KvArgs {
    KvSide side[2];
    const int64_t* slot;
    int64_t T, H, D, num_slots;
    int per_tensor;
};

template <int G>
__global__ __launch_bounds__(kKvThreads) void kv_cache_write_kernel(KvArgs a) {
    const KvSide s = blockIdx.y ? a.side[1] : a.side[0];
    const int j = threadIdx.x % G;                                   // lane in the row's group
    const int64_t row = (int64_t)blockIdx.x * (kKvThreads / G) + threadIdx.x / G;
    const int64_t rows = a.T * a.H;
    int64_t t = 0, h = 0, slot = -1;
    if (row < rows) {
        t = row / a.H;
        h = row - t * a.H;
        slot = a.slot[t];
    }
    const bool live = slot >= 0 && slot < a.num_slots;
    const bool mine = live && (int64_t)j * 8 < a.D;
    float v[8];
    float amax = 0.0f;
    if (mine) {
        const uint4 p = *reinterpret_cast<const uint4*>(s.x + t * s.ld_x + h * a.D + (int64_t)j * 8);
        unpack8(p, v);
#pragma unroll
        for (int e = 0; e < 8; ++e) amax = fmaxf(amax, fabsf(v[e]));
    }
    // max over the G lanes of the row; every lane of the wave takes part
#pragma unroll
    for (int o = G / 2; o >= 1; o /= 2) amax = fmaxf(amax, __shfl_xor(amax, o));
    float sc;
    if (a.per_tensor) {
        sc = s.scale[0];
    } else {
        sc = fmaxf((float)((double)amax / 448.0), 0x1p-100f);
        if (live && j == 0) s.scale[slot * a.H + h] = sc;
    }
    if (!mine) return;
    const float inv = (float)(1.0 / (double)sc);
    uint2 o;
    o.x = e4m3x4(v[0] * inv, v[1] * inv, v[2] * inv, v[3] * inv);
    o.y = e4m3x4(v[4] * inv, v[5] * inv, v[6] * inv, v[7] * inv);
    *reinterpret_cast<uint2*>(s.cache + (slot * a.H + h) * a.D + (int64_t)j * 8) = o;
}

}  // namespace

int64_t kv_group_lanes(int64_t D) {
    int64_t g = 1;
    while (g * 8 < D) g *= 2;
    return g;
}

hipError_t launch_kv_cache_write(const uint16_t* k, int64_t ld_k, const uint16_t* v, int64_t ld_v,
                                 const int64_t* slot_mapping, int64_t T, int64_t H, int64_t D,
                                 int64_t num_slots, int per_tensor, float* k_scale, float* v_scale,
                                 uint8_t* k_cache, uint8_t* v_cache, hipStream_t stream) {
    KvArgs a;
    a.side[0] = KvSide{k, ld_k, k_scale, k_cache};
    a.side[1] = KvSide{v, ld_v, v_scale, v_cache};
    a.slot = slot_mapping;
    a.T = T;
    a.H = H;
    a.D = D;
    a.num_slots = num_slots;
    a.per_tensor = per_tensor;
    const int64_t rows = T * H;
    const int64_t g = kv_group_lanes(D);
    const int64_t per_block = kKvThreads / g;
    dim3 grid((unsigned)((rows + per_block - 1) / per_block), 2), block(kKvThreads);
#define SPEC_KV_CASE(N)                                                                     \
    case N:                                                                                 \
        hipLaunchKernelGGL(kv_cache_write_kernel<N>, grid, block, 0, stream, a);            \
        break;
    switch (g) {
        SPEC_KV_CASE(1)
        SPEC_KV_CASE(2)
        SPEC_KV_CASE(4)
        SPEC_KV_CASE(8)
        SPEC_KV_CASE(16)
        SPEC_KV_CASE(32)
        default:
            hipLaunchKernelGGL(kv_cache_write_kernel<64>, grid, block, 0, stream, a);
    }
#undef SPEC_KV_CASE
    return hipGetLastError();
}

}  // namespace specfp8
