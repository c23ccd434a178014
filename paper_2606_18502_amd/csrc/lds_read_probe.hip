// Control measurement for the LDS bank-conflict counters of the FP8 GEMM's
// operand reads (not part of libspecfp8; a standalone program).
//
// Three kernels issue the same number of ds_read_b128 instructions from one
// LDS buffer and differ only in the addresses the 64 lanes read:
//   lds_contiguous  lane l reads bytes 16l .. 16l+15 (one 1 KiB stretch);
//   lds_gemm_swz    the GEMM's operand read: lane l reads logical 16-byte
//                   chunk 2(l/16) of 128-byte row l%16, stored in slot
//                   chunk ^ ((row >> 1) & 7)  (gemm.hip, swz);
//   lds_gemm_plain  the same rows and chunks without the swizzle;
//   lds_gemm_pair   the same with slot = chunk ^ {0,1,4,5}[(row >> 1) & 3], a
//                   swizzle that gives distinct banks to lanes l and l+16
//                   (l % 16 < 8) -- the lanes gfx950 serves together in one
//                   LDS cycle of a 128-bit read, by the first three kernels.
// Under a profiler, SQ_LDS_BANK_CONFLICT / SQ_LDS_IDX_ACTIVE of the first
// kernel is the share of LDS cycles the counters report for 128-bit reads
// that touch every bank exactly once.
//
// Build and run (one MI355X):
//   hipcc --offload-arch=gfx950 -O3 -o lds_read_probe paper_2606_18502_amd/csrc/lds_read_probe.hip
//   rocprofv3 --pmc SQ_LDS_BANK_CONFLICT SQ_LDS_IDX_ACTIVE SQ_INSTS_LDS SQ_LDS_ADDR_CONFLICT \
//       --output-format csv -d <out> -o run -- ./lds_read_probe
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

namespace {

constexpr int kThreads = 256;
constexpr int kIters = 4096;
constexpr int kBlocks = 256;

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

enum Pattern { kContiguous = 0, kGemmSwizzled = 1, kGemmPlain = 2, kGemmPair = 3 };

template <int P>
__device__ __forceinline__ uint32_t lane_offset(int lane, int it) {
    const int wave_base = (it & 7) * 2048;   // 8 regions of 2 KiB so the reads are not all one address set
    if (P == kContiguous) return wave_base + lane * 16;
    const int row = lane & 15, chunk = 2 * (lane >> 4) + (it & 1);
    const int pair_swz = (0x5410 >> (4 * ((row >> 1) & 3))) & 0xf;   // {0, 1, 4, 5}[(row >> 1) & 3]
    const int slot = P == kGemmSwizzled ? (chunk ^ ((row >> 1) & 7)) : P == kGemmPair ? (chunk ^ pair_swz) : chunk;
    return wave_base + row * 128 + slot * 16;
}

template <int P>
__global__ __launch_bounds__(kThreads) void lds_read_kernel(uint32_t* out) {
    __shared__ __attribute__((aligned(1024))) uint32_t lds[16384];   // 64 KiB
    for (int i = threadIdx.x; i < 16384; i += kThreads) lds[i] = i * 2654435761u;
    __syncthreads();
    const int lane = threadIdx.x & 63;
    const uint32_t base = (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)lds;
    u32x4 acc = {0u, 0u, 0u, 0u};
    for (int it = 0; it < kIters; it += 8) {
        u32x4 v[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const uint32_t a = base + lane_offset<P>(lane, it + j);
            asm volatile("ds_read_b128 %0, %1" : "=v"(v[j]) : "v"(a));
        }
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
#pragma unroll
        for (int j = 0; j < 8; ++j) acc ^= v[j];
    }
    if ((acc.x ^ acc.y ^ acc.z ^ acc.w) == 0x9e3779b9u) out[threadIdx.x] = 1u;
}

#define CHECK(x)                                                                     \
    do {                                                                             \
        hipError_t e_ = (x);                                                         \
        if (e_ != hipSuccess) {                                                      \
            fprintf(stderr, "HIP error %s at line %d\n", hipGetErrorString(e_), __LINE__); \
            exit(1);                                                                 \
        }                                                                            \
    } while (0)

template <int P>
void run(const char* name, uint32_t* out) {
    hipEvent_t e0, e1;
    CHECK(hipEventCreate(&e0));
    CHECK(hipEventCreate(&e1));
    CHECK(hipEventRecord(e0));
    hipLaunchKernelGGL(lds_read_kernel<P>, dim3(kBlocks), dim3(kThreads), 0, 0, out);
    CHECK(hipGetLastError());
    CHECK(hipEventRecord(e1));
    CHECK(hipEventSynchronize(e1));
    float ms = 0.0f;
    CHECK(hipEventElapsedTime(&ms, e0, e1));
    const double reads = (double)kBlocks * (kThreads / 64) * kIters;
    printf("%-16s %8.2f us  %.0f ds_read_b128 per wave\n", name, ms * 1e3, reads / (kBlocks * (kThreads / 64)));
    CHECK(hipEventDestroy(e0));
    CHECK(hipEventDestroy(e1));
}

}  // namespace

int main() {
    uint32_t* out = nullptr;
    CHECK(hipMalloc(&out, kThreads * sizeof(uint32_t)));
    for (int rep = 0; rep < 2; ++rep) {   // the first round includes the code-object load
        run<kContiguous>("lds_contiguous", out);
        run<kGemmSwizzled>("lds_gemm_swz", out);
        run<kGemmPlain>("lds_gemm_plain", out);
        run<kGemmPair>("lds_gemm_pair", out);
    }
    CHECK(hipDeviceSynchronize());
    CHECK(hipFree(out));
    return 0;
}
