// Tree attention masks for token-tree verification: for every node of a
// drafted tree, the set of tree nodes its row may attend to (the nodes on the
// path from the root to it, itself included) as a 64-bit mask, and its depth.
//
// One wave per sequence, lane n owning node n (N <= 64).  The masks come from
// pointer jumping over the parent links: after step s every lane holds the
// nodes within 2^s - 1 steps above it and a pointer to its 2^s-th ancestor,
// so six steps of lane exchanges (no memory traffic) cover any depth up to
// 64.  A node whose parent is not one of the earlier nodes (or -1) poisons
// itself and, through the same exchanges, every node below it.
#include "device_common.hpp"
#include "kernels.hpp"

namespace specfp8 {

namespace {

constexpr int kTmThreads = 256;
constexpr int kTmSeqPerBlock = kTmThreads / 64;

__global__ __launch_bounds__(kTmThreads) void tree_mask_kernel(const int32_t* __restrict__ parents, int64_t B,
                                                               int N, uint64_t* __restrict__ mask,
                                                               int32_t* __restrict__ depth) {
    const int lane = threadIdx.x & 63;
    const int64_t b = (int64_t)blockIdx.x * kTmSeqPerBlock + threadIdx.x / 64;   // wave-uniform
    if (b >= B) return;
    const bool node = lane < N;
    const int p = node ? parents[b * N + lane] : -1;
    int bad = (node && (p < -1 || p >= lane)) ? 1 : 0;
    uint32_t lo = 0, hi = 0;                  // the mask, as two halves for the lane exchanges
    if (node) {
        if (lane < 32) lo = 1u << lane;
        else hi = 1u << (lane - 32);
    }
    int anc = bad ? -1 : p;
#pragma unroll
    for (int s = 0; s < 6; ++s) {
        const int src = anc >= 0 ? anc : lane;
        const uint32_t lo_up = __shfl(lo, src);
        const uint32_t hi_up = __shfl(hi, src);
        const int bad_up = __shfl(bad, src);
        const int anc_up = __shfl(anc, src);
        if (anc >= 0) {
            lo |= lo_up;
            hi |= hi_up;
            bad |= bad_up;
            anc = anc_up;
        }
    }
    if (!node) return;
    const uint64_t m = bad ? 0ull : (((uint64_t)hi << 32) | lo);
    mask[b * N + lane] = m;
    depth[b * N + lane] = bad ? 0 : __popcll(m);
}

}  // namespace

hipError_t launch_tree_mask(const int32_t* parents, int64_t B, int64_t N, uint64_t* mask, int32_t* depth,
                            hipStream_t stream) {
    const int64_t blocks = (B + kTmSeqPerBlock - 1) / kTmSeqPerBlock;
    hipLaunchKernelGGL(tree_mask_kernel, dim3((unsigned)blocks), dim3(kTmThreads), 0, stream, parents, B, (int)N,
                       mask, depth);
    return hipGetLastError();
}

}  // namespace specfp8
