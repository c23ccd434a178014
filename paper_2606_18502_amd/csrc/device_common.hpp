// Device helpers shared by the verify-path kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace specfp8 {

constexpr int kWave = 64;

// bf16 bit pattern -> fp32 (exact).
__device__ __forceinline__ float bf16_to_f32(uint32_t bits16) {
    return __uint_as_float(bits16 << 16);
}

// fp32 -> bf16 bit pattern, round to nearest even (finite inputs; NaN stays NaN).
__device__ __forceinline__ uint32_t f32_to_bf16_rne(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return 0x7fc0u;
    u += 0x7fffu + ((u >> 16) & 1u);
    return u >> 16;
}

// The SiLU gate of the FFN (shared by the SiLU-gated quantize and the GEMM
// epilogue that fuses it, so both give the same h for the same g, u):
// h = bf16(silu(g) * u) with silu(g) = g / (1 + e^-g) = g * rcp(1 + 2^(-g log2 e)),
// in fp32 on the hardware exp2 and reciprocal (about 1 ulp each): the bf16
// rounding of h only differs from an exact evaluation at near-ties.  Large
// |g| saturate correctly: 2^(+big) = inf gives rcp = 0 (silu -> -0), and
// 2^(-big) = 0 gives silu = g.
__device__ __forceinline__ float silu_mul_bf16(float g, float u) {
    const float e = __builtin_amdgcn_exp2f(g * -1.44269504088896341f);
    const float sg = g * __builtin_amdgcn_rcpf(1.0f + e);
    return bf16_to_f32(f32_to_bf16_rne(sg * u));
}

// Unpack 8 bf16 values held in a 16-byte vector.
__device__ __forceinline__ void unpack8(const uint4& v, float out[8]) {
    out[0] = __uint_as_float(v.x << 16);
    out[1] = __uint_as_float(v.x & 0xffff0000u);
    out[2] = __uint_as_float(v.y << 16);
    out[3] = __uint_as_float(v.y & 0xffff0000u);
    out[4] = __uint_as_float(v.z << 16);
    out[5] = __uint_as_float(v.z & 0xffff0000u);
    out[6] = __uint_as_float(v.w << 16);
    out[7] = __uint_as_float(v.w & 0xffff0000u);
}

// Four fp32 values -> four E4M3 codes packed little-endian into one dword.
// Inputs are first clamped to [-448, 448] so the hardware conversion (round
// to nearest even on the OCP E4M3 grid) only ever sees in-range values: the
// clamp is the saturation of the format's satfinite conversion.
__device__ __forceinline__ uint32_t e4m3x4(float a, float b, float c, float d) {
    a = __builtin_amdgcn_fmed3f(a, -448.0f, 448.0f);
    b = __builtin_amdgcn_fmed3f(b, -448.0f, 448.0f);
    c = __builtin_amdgcn_fmed3f(c, -448.0f, 448.0f);
    d = __builtin_amdgcn_fmed3f(d, -448.0f, 448.0f);
    int r = __builtin_amdgcn_cvt_pk_fp8_f32(a, b, 0, false);
    r = __builtin_amdgcn_cvt_pk_fp8_f32(c, d, r, true);
    return (uint32_t)r;
}

// Wave-wide reductions on DPP lane permutations (VALU operand modifiers, no
// LDS round trip): xor 1 and xor 2 inside quads, then the half-row and row
// mirrors leave every lane of a 16-lane row with the row's total; the four
// row totals are read as scalars and combined in a fixed order.  The result
// is wave-uniform and deterministic.  All 64 lanes must be active.
template <int CTRL>
__device__ __forceinline__ int dpp_mov(int v) {
    return __builtin_amdgcn_mov_dpp(v, CTRL, 0xF, 0xF, false);
}

template <class Op>
__device__ __forceinline__ int wave_reduce_i(int v, Op op) {
    v = op(v, dpp_mov<0xB1>(v));    // quad_perm [1,0,3,2]
    v = op(v, dpp_mov<0x4E>(v));    // quad_perm [2,3,0,1]
    v = op(v, dpp_mov<0x141>(v));   // row_half_mirror
    v = op(v, dpp_mov<0x140>(v));   // row_mirror
    const int r0 = __builtin_amdgcn_readlane(v, 0), r1 = __builtin_amdgcn_readlane(v, 16);
    const int r2 = __builtin_amdgcn_readlane(v, 32), r3 = __builtin_amdgcn_readlane(v, 48);
    return op(op(r0, r1), op(r2, r3));
}

__device__ __forceinline__ float wave_max(float v) {
    return __builtin_bit_cast(float, wave_reduce_i(__builtin_bit_cast(int, v), [](int a, int b) {
        return __builtin_bit_cast(int, fmaxf(__builtin_bit_cast(float, a), __builtin_bit_cast(float, b)));
    }));
}

__device__ __forceinline__ float wave_sum(float v) {
    return __builtin_bit_cast(float, wave_reduce_i(__builtin_bit_cast(int, v), [](int a, int b) {
        return __builtin_bit_cast(int, __builtin_bit_cast(float, a) + __builtin_bit_cast(float, b));
    }));
}

__device__ __forceinline__ int wave_min_i32(int v) {
    return wave_reduce_i(v, [](int a, int b) { return a < b ? a : b; });
}

__device__ __forceinline__ double wave_sum_d(double v) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, kWave);
    return v;
}

// Block-wide max / sum for blocks of up to 1024 threads; `red` holds >= 16 floats.
// The reduction order is fixed, so results are deterministic.
__device__ __forceinline__ float block_max(float v, float* red) {
    const int lane = threadIdx.x & (kWave - 1), w = threadIdx.x / kWave;
    const int nw = (blockDim.x + kWave - 1) / kWave;
    v = wave_max(v);
    __syncthreads();
    if (lane == 0) red[w] = v;
    __syncthreads();
    float r = red[0];
    for (int i = 1; i < nw; ++i) r = fmaxf(r, red[i]);
    return r;
}

__device__ __forceinline__ float block_sum(float v, float* red) {
    const int lane = threadIdx.x & (kWave - 1), w = threadIdx.x / kWave;
    const int nw = (blockDim.x + kWave - 1) / kWave;
    v = wave_sum(v);
    __syncthreads();
    if (lane == 0) red[w] = v;
    __syncthreads();
    float r = red[0];
    for (int i = 1; i < nw; ++i) r += red[i];
    return r;
}

}  // namespace specfp8
