// Row quantization of bf16 activations/weights to E4M3 with fp32 scales, and
// the SiLU-gated variant that feeds the down projection.
//
// One workgroup owns one row.  The row is read from HBM once with 16-byte
// loads (8 bf16 per load, consecutive threads on consecutive 16-byte chunks,
// so every wave reads 1 KiB contiguous per instruction) and kept in
// registers; the block reduces max|v| (wave shuffles, then LDS across waves),
// derives the scale, and encodes the registers it already holds.  HBM traffic
// is therefore the algorithmic 2 bytes in + 1 byte out per element (4 + 1 for
// the SiLU-gated input) plus 4 bytes of scale per row.  Rows wider than
// 65536 elements take a second pass that re-reads the row.
#include "device_common.hpp"
#include "kernels.hpp"

namespace specfp8 {

namespace {

constexpr int kQThreads = 256;       // threads of the element-wise kernel
constexpr int kQMaxThreads = 1024;   // threads per row of the row kernel, at most

template <int IN_KIND>
__device__ __forceinline__ void load_chunk(const uint16_t* __restrict__ xrow, int64_t cols,
                                           int64_t c, float v[8]) {
    if (IN_KIND == 0) {
        const uint4 a = *reinterpret_cast<const uint4*>(xrow + c * 8);
        unpack8(a, v);
    } else {
        const uint4 a = *reinterpret_cast<const uint4*>(xrow + c * 8);
        const uint4 b = *reinterpret_cast<const uint4*>(xrow + cols + c * 8);
        float g[8], u[8];
        unpack8(a, g);
        unpack8(b, u);
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] = silu_mul_bf16(g[e], u[e]);
    }
}

__device__ __forceinline__ void store_codes(uint8_t* __restrict__ qrow, int64_t c, const float v[8],
                                            float inv) {
    uint2 o;
    o.x = e4m3x4(v[0] * inv, v[1] * inv, v[2] * inv, v[3] * inv);
    o.y = e4m3x4(v[4] * inv, v[5] * inv, v[6] * inv, v[7] * inv);
    *reinterpret_cast<uint2*>(qrow + c * 8) = o;
}

__device__ __forceinline__ void row_scale(float amax, float* s_out, float* inv_out) {
    float s = (float)((double)amax / 448.0);
    s = fmaxf(s, 0x1p-100f);
    *s_out = s;
    *inv_out = (float)(1.0 / (double)s);
}

// Static calibration: running[0] = max(running[0], s).  Scales are finite and
// non-negative, and the bit patterns of non-negative floats order like
// unsigned integers, so an integer atomic max is exact and order-independent.
__device__ __forceinline__ void calibrate_max(float* running, float s) {
    atomicMax(reinterpret_cast<unsigned int*>(running), __float_as_uint(s));
}

// MODE 0: per-row scales (written); 1: one given scale; 2: calibration only.
// NCH > 0: the row lives in registers (NCH chunks of 8 per thread).
// NCH == 0: rows too wide for registers; amax pass and encode pass each read the row.
template <int IN_KIND, int MODE, int NCH>
__global__ __launch_bounds__(kQMaxThreads) void quantize_rows_kernel(
    const uint16_t* __restrict__ x, int64_t cols, int64_t ld_x, float* __restrict__ scales,
    uint8_t* __restrict__ q, int64_t ld_q) {
    __shared__ float red[16];
    const int64_t row = blockIdx.x;
    const int64_t nchunks = cols / 8;
    const uint16_t* xrow = x + row * ld_x;
    uint8_t* qrow = q + row * ld_q;
    const int t = threadIdx.x;
    const int nt = blockDim.x;

    if constexpr (NCH > 0) {
        float v[NCH][8];
        float amax = 0.0f;
#pragma unroll
        for (int j = 0; j < NCH; ++j) {
            const int64_t c = t + (int64_t)j * nt;
            if (c < nchunks) {
                load_chunk<IN_KIND>(xrow, cols, c, v[j]);
#pragma unroll
                for (int e = 0; e < 8; ++e) amax = fmaxf(amax, fabsf(v[j][e]));
            }
        }
        float s, inv;
        if (MODE == 2) {
            amax = block_max(amax, red);
            row_scale(amax, &s, &inv);
            if (t == 0) calibrate_max(scales, s);
            return;
        }
        if (MODE == 0) {
            amax = block_max(amax, red);
            row_scale(amax, &s, &inv);
            if (t == 0) scales[row] = s;
        } else {
            s = scales[0];
            inv = (float)(1.0 / (double)s);
        }
#pragma unroll
        for (int j = 0; j < NCH; ++j) {
            const int64_t c = t + (int64_t)j * nt;
            if (c < nchunks) store_codes(qrow, c, v[j], inv);
        }
    } else {
        float s, inv;
        if (MODE != 1) {
            float amax = 0.0f;
            for (int64_t c = t; c < nchunks; c += nt) {
                float v[8];
                load_chunk<IN_KIND>(xrow, cols, c, v);
#pragma unroll
                for (int e = 0; e < 8; ++e) amax = fmaxf(amax, fabsf(v[e]));
            }
            amax = block_max(amax, red);
            row_scale(amax, &s, &inv);
            if (MODE == 2) {
                if (t == 0) calibrate_max(scales, s);
                return;
            }
            if (t == 0) scales[row] = s;
        } else {
            s = scales[0];
            inv = (float)(1.0 / (double)s);
        }
        for (int64_t c = t; c < nchunks; c += nt) {
            float v[8];
            load_chunk<IN_KIND>(xrow, cols, c, v);
            store_codes(qrow, c, v, inv);
        }
    }
}

__global__ __launch_bounds__(kQThreads) void silu_mul_bf16_kernel(
    const uint16_t* __restrict__ x, int64_t rows, int64_t cols, int64_t ld_x,
    uint16_t* __restrict__ h, int64_t ld_h) {
    const int64_t c = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (c >= cols / 8) return;
    for (int64_t row = blockIdx.y; row < rows; row += gridDim.y) {
        float v[8];
        load_chunk<1>(x + row * ld_x, cols, c, v);
        uint4 o;
        o.x = f32_to_bf16_rne(v[0]) | (f32_to_bf16_rne(v[1]) << 16);
        o.y = f32_to_bf16_rne(v[2]) | (f32_to_bf16_rne(v[3]) << 16);
        o.z = f32_to_bf16_rne(v[4]) | (f32_to_bf16_rne(v[5]) << 16);
        o.w = f32_to_bf16_rne(v[6]) | (f32_to_bf16_rne(v[7]) << 16);
        *reinterpret_cast<uint4*>(h + row * ld_h + c * 8) = o;
    }
}

// Values the static per-tensor quantizer saturates, |fl32(x * fl32(1/s))| >
// 448 (the calibration clip rate of a test batch): grid-stride over 8-value
// chunks read with 16-byte loads, a wave then block sum, one 64-bit atomic
// add per block into the caller's counter.
__global__ __launch_bounds__(kQThreads) void clip_count_kernel(const uint16_t* __restrict__ x, int64_t rows,
                                                               int64_t cols, int64_t ld_x,
                                                               const float* __restrict__ scale,
                                                               unsigned long long* __restrict__ count) {
    __shared__ unsigned int red[kQThreads / 64];
    const float inv = (float)(1.0 / (double)scale[0]);
    const int64_t nch = cols / 8;
    const int64_t total = rows * nch;
    unsigned int c = 0;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
         i += (int64_t)gridDim.x * blockDim.x) {
        const int64_t r = i / nch;
        const int64_t ch = i - r * nch;
        const uint4 p = *reinterpret_cast<const uint4*>(x + r * ld_x + ch * 8);
        float v[8];
        unpack8(p, v);
#pragma unroll
        for (int e = 0; e < 8; ++e) c += fabsf(v[e] * inv) > 448.0f ? 1u : 0u;
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) c += __shfl_xor(c, o);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = c;
    __syncthreads();
    if (threadIdx.x == 0) {
        unsigned long long sum = 0;
        for (int w = 0; w < kQThreads / 64; ++w) sum += red[w];
        if (sum) atomicAdd(count, sum);
    }
}

template <int IN_KIND, int MODE>
hipError_t launch_quantize_t(const uint16_t* x, int64_t rows, int64_t cols, int64_t ld_x,
                             float* scales, uint8_t* q, int64_t ld_q, hipStream_t stream) {
    // One workgroup per row, wide enough that a thread holds at most 4
    // chunks of 8 (up to 1024 threads; wider rows hold up to 8 per thread or
    // take the two-pass path).  With a given scale (no row maximum, so no
    // workgroup barrier) at most 2 chunks per thread: more waves per row keep
    // more loads in flight (measured on [4096, 14336] rows: 31.5 -> 29.9 us);
    // where the row maximum is reduced across the workgroup, the extra waves
    // cost more at the barrier than they gain (32.8 -> 34.1 us).
    const int64_t nchunks = cols / 8;
    const int64_t per_thread_max = MODE == 1 ? 2 : 4;
    int threads = 256;
    while (threads < kQMaxThreads && nchunks > per_thread_max * (int64_t)threads) threads *= 2;
    if (nchunks < threads) threads = (int)(((nchunks + 63) / 64) * 64);
    const int64_t per = (nchunks + threads - 1) / threads;
    dim3 grid((unsigned)rows), block(threads);
#define SPEC_Q_CASE(N)                                                                        \
    case N:                                                                                   \
        hipLaunchKernelGGL((quantize_rows_kernel<IN_KIND, MODE, N>), grid, block, 0, stream, x, \
                           cols, ld_x, scales, q, ld_q);                                      \
        break;
    switch (per) {
        SPEC_Q_CASE(1)
        SPEC_Q_CASE(2)
        SPEC_Q_CASE(3)
        SPEC_Q_CASE(4)
        SPEC_Q_CASE(5)
        SPEC_Q_CASE(6)
        SPEC_Q_CASE(7)
        SPEC_Q_CASE(8)
        default:
            hipLaunchKernelGGL((quantize_rows_kernel<IN_KIND, MODE, 0>), grid, block, 0, stream, x,
                               cols, ld_x, scales, q, ld_q);
    }
#undef SPEC_Q_CASE
    return hipGetLastError();
}

}  // namespace

hipError_t launch_quantize(const uint16_t* x, int64_t rows, int64_t cols, int64_t ld_x, int in_kind,
                           int mode, float* scales, uint8_t* q, int64_t ld_q, hipStream_t stream) {
    if (in_kind == 0 && mode == 0)
        return launch_quantize_t<0, 0>(x, rows, cols, ld_x, scales, q, ld_q, stream);
    if (in_kind == 0 && mode == 1)
        return launch_quantize_t<0, 1>(x, rows, cols, ld_x, scales, q, ld_q, stream);
    if (in_kind == 0 && mode == 2)
        return launch_quantize_t<0, 2>(x, rows, cols, ld_x, scales, q, ld_q, stream);
    if (in_kind == 1 && mode == 0)
        return launch_quantize_t<1, 0>(x, rows, cols, ld_x, scales, q, ld_q, stream);
    if (in_kind == 1 && mode == 2)
        return launch_quantize_t<1, 2>(x, rows, cols, ld_x, scales, q, ld_q, stream);
    return launch_quantize_t<1, 1>(x, rows, cols, ld_x, scales, q, ld_q, stream);
}

hipError_t launch_clip_count(const uint16_t* x, int64_t rows, int64_t cols, int64_t ld_x, const float* scale,
                             unsigned long long* count, hipStream_t stream) {
    const int64_t total = rows * (cols / 8);
    int64_t blocks = (total + kQThreads - 1) / kQThreads;
    if (blocks > 2048) blocks = 2048;           // 8 workgroups per compute unit, grid-stride beyond
    hipLaunchKernelGGL(clip_count_kernel, dim3((unsigned)blocks), dim3(kQThreads), 0, stream, x, rows, cols, ld_x,
                       scale, count);
    return hipGetLastError();
}

hipError_t launch_silu_mul(const uint16_t* x, int64_t rows, int64_t cols, int64_t ld_x,
                           uint16_t* h, int64_t ld_h, hipStream_t stream) {
    const int64_t nchunks = cols / 8;
    const int64_t gy = rows < 65535 ? rows : 65535;
    dim3 block(kQThreads), grid((unsigned)((nchunks + kQThreads - 1) / kQThreads), (unsigned)gy);
    hipLaunchKernelGGL(silu_mul_bf16_kernel, grid, block, 0, stream, x, rows, cols, ld_x, h, ld_h);
    return hipGetLastError();
}

}  // namespace specfp8
