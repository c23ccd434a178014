// Acceptance test of the speculative-decoding verify step.
//
// Greedy (T == 0):
//   greedy_partial_kernel  (chunk, row) -> max logit and its lowest index
//   greedy_final_kernel    b -> argmax per position, longest matching prefix
// Speculative sampling (T > 0):
//   stoch_stats_kernel     (chunk, row) -> chunk max m and sum 2^(t - m) of
//                          t = z * log2(e)/T (the tempered logit in base 2),
//                          for target rows 0..k and draft rows 0..k-1
//   stoch_sample_kernel    (chunk, b)   -> every block merges the chunk
//                          statistics of its sequence in chunk order, takes the
//                          (identical) accept/reject decisions, and sums the
//                          residual distribution over its chunk; the last block
//                          of the sequence to finish (an atomic ticket) locates
//                          the chunk holding u*R, scans that chunk in vocabulary
//                          order and writes the tokens.
// The vocabulary is split into chunks of 8192 so that B*(2k+1)*ceil(V/8192)
// workgroups stream the logits once (2 bytes per element, 16-byte loads,
// each wave reading 1 KiB contiguous per instruction).  All reductions use a
// fixed order, so results are deterministic.  The sample kernel re-reads only
// the row(s) of the position where sampling happens (<= 2 rows per sequence).
#include "device_common.hpp"
#include "kernels.hpp"

namespace specfp8 {

namespace {

constexpr int kAThreads = 256;
constexpr int kPerThread = 128;                       // elements per thread per chunk
constexpr int64_t kChunk = kAThreads * kPerThread;    // 32768
constexpr int kMaxChunks = 1024;                      // V <= 32M

struct AcceptArgs {
    const uint16_t* zt;
    const uint16_t* zd;
    const int32_t* x;
    const float* u;
    int32_t* out;
    int32_t* num;
    float2* stats;         // [B][R][nchunk]
    float* mass;           // [B][nchunk]
    unsigned int* ctr;     // [B]
    int64_t V, chunk, nchunk;
    int B, k, R;           // R = rows per sequence in `stats`
    float c2;              // log2(e) / T
};

template <bool VEC>
__device__ __forceinline__ void load8(const uint16_t* __restrict__ row, int64_t e, int64_t V, float out[8],
                                      float fill) {
    if (VEC) {
        const uint4 v = *reinterpret_cast<const uint4*>(row + e);
        unpack8(v, out);
    } else {
#pragma unroll
        for (int i = 0; i < 8; ++i) out[i] = (e + i < V) ? bf16_to_f32(row[e + i]) : fill;
    }
}

// ------------------------------------------------------------------ greedy

struct ValIdx {
    float v;
    int i;
};

__device__ __forceinline__ bool better(float v, int i, float bv, int bi) {
    return v > bv || (v == bv && i < bi);
}

template <bool VEC>
__global__ __launch_bounds__(kAThreads) void greedy_partial_kernel(AcceptArgs a) {
    __shared__ float sv[kAThreads / 64];
    __shared__ int si[kAThreads / 64];
    const int64_t c = blockIdx.x;
    const int64_t row = blockIdx.y;                  // b*(k+1) + i
    const uint16_t* z = a.zt + row * a.V;
    const int64_t e0 = c * a.chunk;
    const int64_t e1 = min(e0 + a.chunk, a.V);
    float bv = -INFINITY;
    int bi = 0x7fffffff;
    uint4 raw[kPerThread / 8];
#pragma unroll
    for (int j = 0; j < kPerThread / 8; ++j) {           // all loads in flight first
        const int64_t e = e0 + ((int64_t)j * kAThreads + threadIdx.x) * 8;
        if (VEC && e < e1) raw[j] = *reinterpret_cast<const uint4*>(z + e);
    }
#pragma unroll
    for (int j = 0; j < kPerThread / 8; ++j) {
        const int64_t e = e0 + ((int64_t)j * kAThreads + threadIdx.x) * 8;
        if (e < e1) {
            float v[8];
            if (VEC) unpack8(raw[j], v);
            else load8<false>(z, e, a.V, v, -INFINITY);
#pragma unroll
            for (int q = 0; q < 8; ++q)
                if (e + q < e1 && better(v[q], (int)(e + q), bv, bi)) { bv = v[q]; bi = (int)(e + q); }
        }
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
        const float ov = __shfl_xor(bv, o, 64);
        const int oi = __shfl_xor(bi, o, 64);
        if (better(ov, oi, bv, bi)) { bv = ov; bi = oi; }
    }
    const int w = threadIdx.x >> 6;
    if ((threadIdx.x & 63) == 0) { sv[w] = bv; si[w] = bi; }
    __syncthreads();
    if (threadIdx.x == 0) {
        for (int q = 1; q < kAThreads / 64; ++q)
            if (better(sv[q], si[q], bv, bi)) { bv = sv[q]; bi = si[q]; }
        a.stats[row * a.nchunk + c] = make_float2(bv, __int_as_float(bi));
    }
}

__global__ __launch_bounds__(256) void greedy_final_kernel(AcceptArgs a) {
    __shared__ int g[17];
    const int b = blockIdx.x;
    const int t = threadIdx.x, lane = t & 63, wv = t >> 6;
    // wave wv merges positions wv, wv+4, ...; lanes stride over the chunks
    for (int pos = wv; pos <= a.k; pos += 4) {
        const float2* st = a.stats + ((int64_t)b * (a.k + 1) + pos) * a.nchunk;
        float bv = -INFINITY;
        int bi = 0x7fffffff;
        for (int64_t c = lane; c < a.nchunk; c += 64) {
            const float2 p = st[c];
            const int pi = __float_as_int(p.y);
            if (better(p.x, pi, bv, bi)) { bv = p.x; bi = pi; }
        }
#pragma unroll
        for (int o = 32; o >= 1; o >>= 1) {
            const float ov = __shfl_xor(bv, o, 64);
            const int oi = __shfl_xor(bi, o, 64);
            if (better(ov, oi, bv, bi)) { bv = ov; bi = oi; }
        }
        if (lane == 0) g[pos] = bi;
    }
    __syncthreads();
    if (t <= a.k) {
        // a_b = number of leading drafts equal to the target argmax
        int acc = a.k;
        for (int i = 0; i < a.k; ++i)
            if (a.x[(int64_t)b * a.k + i] != g[i]) { acc = i; break; }
        int32_t* out = a.out + (int64_t)b * (a.k + 1);
        out[t] = t < acc ? g[t] : (t == acc ? g[acc] : -1);
        if (t == 0) a.num[b] = acc;
    }
}

// ------------------------------------------------------------- stochastic

template <bool VEC>
__global__ __launch_bounds__(kAThreads) void stoch_stats_kernel(AcceptArgs a) {
    __shared__ float red[16];
    const int64_t c = blockIdx.x;
    const int b = blockIdx.y / a.R;
    const int r = blockIdx.y % a.R;
    const uint16_t* z = (r <= a.k) ? a.zt + ((int64_t)b * (a.k + 1) + r) * a.V
                                   : a.zd + ((int64_t)b * a.k + (r - a.k - 1)) * a.V;
    if (c == 0 && r == 0 && threadIdx.x == 0) a.ctr[b] = 0u;   // ticket for stoch_sample_kernel
    const int64_t e0 = c * a.chunk;
    const int64_t e1 = min(e0 + a.chunk, a.V);
    // Every thread streams its 8-element vectors and keeps an online
    // (max m, sum 2^(t - m)) pair; the loads of all vectors are issued first.
    uint4 raw[kPerThread / 8];
#pragma unroll
    for (int j = 0; j < kPerThread / 8; ++j) {
        const int64_t e = e0 + ((int64_t)j * kAThreads + threadIdx.x) * 8;
        if (VEC && e < e1) raw[j] = *reinterpret_cast<const uint4*>(z + e);
    }
    float m = -INFINITY, sum = 0.0f;
#pragma unroll
    for (int j = 0; j < kPerThread / 8; ++j) {
        const int64_t e = e0 + ((int64_t)j * kAThreads + threadIdx.x) * 8;
        if (e < e1) {
            float v[8];
            if (VEC) unpack8(raw[j], v);
            else load8<false>(z, e, a.V, v, 0.0f);
            float vm = -INFINITY;
#pragma unroll
            for (int q = 0; q < 8; ++q) {
                v[q] = (e + q < e1) ? v[q] * a.c2 : -INFINITY;
                vm = fmaxf(vm, v[q]);
            }
            if (vm > m) {
                sum = (m == -INFINITY) ? 0.0f : sum * exp2f(m - vm);
                m = vm;
            }
#pragma unroll
            for (int q = 0; q < 8; ++q) sum += exp2f(v[q] - m);
        }
    }
    const float M = block_max(m, red);
    float s = (m == -INFINITY) ? 0.0f : sum * exp2f(m - M);
    s = block_sum(s, red);
    if (threadIdx.x == 0) a.stats[((int64_t)b * a.R + r) * a.nchunk + c] = make_float2(M, s);
}

// Residual (or bonus) probability of element e given the sampled position.
struct Dist {
    const uint16_t* zt_row;   // target row j
    const uint16_t* zd_row;   // draft row j, or null (one-hot drafts / bonus)
    float mt, inv_zt;         // merged max and 1/sum of the target row
    float md, inv_zd;
    int64_t skip;             // element forced to zero (one-hot draft), -1 if none
};

template <bool VEC>
__device__ __forceinline__ void dist8(const Dist& d, float c2, int64_t e, int64_t e1, int64_t V, float r[8]) {
    float zt[8];
    load8<VEC>(d.zt_row, e, V, zt, 0.0f);
    if (d.zd_row) {
        float zd[8];
        load8<VEC>(d.zd_row, e, V, zd, 0.0f);
#pragma unroll
        for (int q = 0; q < 8; ++q) {
            const float p = exp2f(zt[q] * c2 - d.mt) * d.inv_zt;
            const float qq = exp2f(zd[q] * c2 - d.md) * d.inv_zd;
            r[q] = (e + q < e1) ? fmaxf(p - qq, 0.0f) : 0.0f;
        }
    } else {
#pragma unroll
        for (int q = 0; q < 8; ++q) {
            const float p = exp2f(zt[q] * c2 - d.mt) * d.inv_zt;
            r[q] = (e + q < e1 && e + q != d.skip) ? p : 0.0f;
        }
    }
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

template <bool VEC>
__global__ __launch_bounds__(kAThreads) void stoch_sample_kernel(AcceptArgs a) {
    __shared__ float sM[33], sZ[33];
    __shared__ int s_acc[16];
    __shared__ int s_j, s_last, s_fallback, s_cstar;
    __shared__ float red[16];
    __shared__ double dsum[kAThreads / 64];
    __shared__ double s_base, s_target;
    __shared__ float s_mass[kMaxChunks];
    __shared__ int s_found, s_lastnz;
    const int64_t c = blockIdx.x;
    const int b = blockIdx.y;
    const int t = threadIdx.x;
    const int lane = t & 63, wv = t >> 6;
    const int k = a.k;

    // 1. merge the chunk statistics of every row of sequence b: wave wv takes
    //    rows wv, wv+4, ...; lanes stride over chunks; fixed shuffle tree.
    for (int r = wv; r < a.R; r += kAThreads / 64) {
        const float2* st = a.stats + ((int64_t)b * a.R + r) * a.nchunk;
        float m = -INFINITY, z = 0.0f;
        for (int64_t q = lane; q < a.nchunk; q += 64) {
            const float2 v = st[q];
            merge_ms(m, z, v.x, v.y);
        }
        const float M = wave_max(m);
        const float Z = wave_sum(m == -INFINITY ? 0.0f : z * exp2f(m - M));
        if (lane == 0) { sM[r] = M; sZ[r] = Z; }
    }
    __syncthreads();

    // 2. accept tests of the k drafts, evaluated in parallel (identical in
    //    every block of sequence b); the first rejection j is then a scan.
    if (t < k) {
        const int32_t xi = a.x[(int64_t)b * k + t];
        double p = 0.0, q = 0.0;
        if (xi >= 0 && xi < a.V) {
            const float zt = bf16_to_f32(a.zt[((int64_t)b * (k + 1) + t) * a.V + xi]);
            p = exp2((double)(zt * a.c2) - (double)sM[t]) / (double)sZ[t];
            if (a.zd) {
                const float zd = bf16_to_f32(a.zd[((int64_t)b * k + t) * a.V + xi]);
                q = exp2((double)(zd * a.c2) - (double)sM[k + 1 + t]) / (double)sZ[k + 1 + t];
            } else {
                q = 1.0;
            }
        }
        const double ui = (double)a.u[(int64_t)b * (k + 1) + t];
        s_acc[t] = (ui * q < p) ? 1 : 0;
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
    if (j < k) {
        if (a.zd) {
            d.zd_row = a.zd + ((int64_t)b * k + j) * a.V;
            d.md = sM[k + 1 + j];
            d.inv_zd = 1.0f / sZ[k + 1 + j];
        } else {
            d.skip = a.x[(int64_t)b * k + j];
        }
    }

    // 3. residual mass of this chunk
    const int64_t e0 = c * a.chunk;
    const int64_t e1 = min(e0 + a.chunk, a.V);
    float part = 0.0f;
#pragma unroll
    for (int jj = 0; jj < kPerThread / 8; ++jj) {
        const int64_t e = e0 + ((int64_t)jj * kAThreads + t) * 8;
        if (e < e1) {
            float r[8];
            dist8<VEC>(d, a.c2, e, e1, a.V, r);
#pragma unroll
            for (int q = 0; q < 8; ++q) part += r[q];
        }
    }
    part = block_sum(part, red);
    if (t == 0) {
        a.mass[(int64_t)b * a.nchunk + c] = part;
        __threadfence();
        const unsigned int ticket = atomicAdd(a.ctr + b, 1u);
        s_last = (ticket == (unsigned int)(a.nchunk - 1));
    }
    __syncthreads();
    if (!s_last) return;
    __threadfence();

    // 4. last block of sequence b: gather the chunk masses (if the residual
    //    vanished through rounding, the chunk masses of p_j instead), find the
    //    chunk holding u*R, then scan that chunk in vocabulary order.
    {
        const float* ms = a.mass + (int64_t)b * a.nchunk;
        float mine = 0.0f;
        for (int64_t q = t; q < a.nchunk; q += kAThreads) {
            const float v = __hip_atomic_load(ms + q, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            s_mass[q] = v;
            mine += v;
        }
        const float R = block_sum(mine, red);
        if (t == 0) s_fallback = !(R > 0.0f);
    }
    __syncthreads();
    if (s_fallback) {
        const float2* st = a.stats + ((int64_t)b * a.R + j) * a.nchunk;
        for (int64_t q = t; q < a.nchunk; q += kAThreads) {
            const float2 v = st[q];
            s_mass[q] = v.x == -INFINITY ? 0.0f : v.y * exp2f(v.x - d.mt) * d.inv_zt;
        }
        d.zd_row = nullptr;
        d.skip = -1;
        __syncthreads();
    }
    if (wv == 0) {
        // wave 0: prefix over chunk masses in double (lane l owns a contiguous run)
        const int64_t per = (a.nchunk + 63) / 64;
        const int64_t q0 = lane * per, q1 = min(q0 + per, a.nchunk);
        double loc = 0.0;
        int64_t lastpos = -1;
        for (int64_t q = q0; q < q1; ++q) {
            loc += (double)s_mass[q];
            if (s_mass[q] > 0.0f) lastpos = q;
        }
        double incl = loc;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
            const double y = __shfl_up(incl, o, 64);
            if (lane >= o) incl += y;
        }
        const double R = __shfl(incl, 63, 64);
        const double target = (double)a.u[(int64_t)b * (k + 1) + k] * R;
        double cum = incl - loc;
        int64_t cstar = -1;
        double base = 0.0;
        for (int64_t q = q0; q < q1; ++q) {
            const double mq = (double)s_mass[q];
            if (cstar < 0 && cum + mq > target) { cstar = q; base = cum; }
            cum += mq;
        }
        // the first lane (in vocabulary order) that found the crossing wins
        unsigned long long hit = __ballot(cstar >= 0);
        int64_t lastall = lastpos;
#pragma unroll
        for (int o = 32; o >= 1; o >>= 1) {
            const int64_t y = __shfl_xor(lastall, o, 64);
            lastall = y > lastall ? y : lastall;
        }
        if (hit) {
            const int src = __ffsll((long long)hit) - 1;
            const int64_t cs = __shfl(cstar, src, 64);
            const double bs = __shfl(base, src, 64);
            if (lane == 0) { s_cstar = (int)cs; s_base = bs; }
        } else if (lane == 0) {
            s_cstar = (int)(lastall >= 0 ? lastall : 0);   // u*R beyond the total (rounding)
            s_base = R;
        }
        if (lane == 0) s_target = target;
    }
    if (t == 0) { s_found = 0x7fffffff; s_lastnz = -1; }
    __syncthreads();
    const int64_t cs = s_cstar;
    const double tgt = s_target - s_base;
    const int64_t f0 = cs * a.chunk;
    const int64_t f1 = min(f0 + a.chunk, a.V);
    // contiguous ownership: thread t scans elements [f0 + 128t, f0 + 128t + 128).
    // Pass 1: per-thread sums; exclusive scan across the block; pass 2: the
    // thread whose range holds the crossing walks its elements again.
    double mine = 0.0;
    int lastnz = -1;
#pragma unroll 4
    for (int jj = 0; jj < kPerThread / 8; ++jj) {
        const int64_t e = f0 + (int64_t)t * kPerThread + jj * 8;
        if (e < f1) {
            float r[8];
            dist8<VEC>(d, a.c2, e, f1, a.V, r);
#pragma unroll
            for (int q = 0; q < 8; ++q) {
                mine += (double)r[q];
                if (r[q] > 0.0f) lastnz = (int)(e + q);
            }
        }
    }
    double incl = mine;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const double y = __shfl_up(incl, o, 64);
        if (lane >= o) incl += y;
    }
    if (lane == 63) dsum[wv] = incl;
    __syncthreads();
    double before = 0.0;
    for (int q = 0; q < wv; ++q) before += dsum[q];
    double cum = before + incl - mine;
    int found = -1;
    if (cum <= tgt && cum + mine > tgt) {
        for (int jj = 0; jj < kPerThread / 8 && found < 0; ++jj) {
            const int64_t e = f0 + (int64_t)t * kPerThread + jj * 8;
            if (e < f1) {
                float r[8];
                dist8<VEC>(d, a.c2, e, f1, a.V, r);
                for (int q = 0; q < 8; ++q) {
                    cum += (double)r[q];
                    if (found < 0 && e + q < f1 && cum > tgt) found = (int)(e + q);
                }
            }
        }
    }
    if (found >= 0) atomicMin(&s_found, found);
    if (lastnz >= 0) atomicMax(&s_lastnz, lastnz);
    __syncthreads();
    if (t <= k) {
        int tok = s_found;
        if (tok == 0x7fffffff) tok = s_lastnz >= 0 ? s_lastnz : (int)f0;
        int32_t* out = a.out + (int64_t)b * (k + 1);
        out[t] = t < j ? a.x[(int64_t)b * k + t] : (t == j ? tok : -1);
        if (t == 0) {
            a.num[b] = j;
            a.ctr[b] = 0u;
        }
    }
}

inline size_t align256(size_t x) { return (x + 255) / 256 * 256; }

}  // namespace

AcceptPlan plan_accept(int64_t B, int64_t k, int64_t V) {
    AcceptPlan p{};
    p.chunk = kChunk;
    if (V < p.chunk) p.chunk = (V + 7) / 8 * 8;
    p.nchunk = (V + p.chunk - 1) / p.chunk;
    const int64_t R = 2 * k + 1;
    p.stats_off = 0;
    p.mass_off = align256((size_t)B * R * p.nchunk * sizeof(float2));
    p.ctr_off = p.mass_off + align256((size_t)B * p.nchunk * sizeof(float));
    p.bytes = p.ctr_off + align256((size_t)B * sizeof(unsigned int));
    return p;
}

hipError_t launch_accept(const AcceptPlan& p, const uint16_t* zt, const uint16_t* zd, const int32_t* x,
                         const float* u, int64_t B, int64_t k, int64_t V, float temperature,
                         int32_t* out_tokens, int32_t* num_accepted, void* workspace, hipStream_t stream) {
    AcceptArgs a;
    char* ws = reinterpret_cast<char*>(workspace);
    a.zt = zt; a.zd = zd; a.x = x; a.u = u; a.out = out_tokens; a.num = num_accepted;
    a.stats = reinterpret_cast<float2*>(ws + p.stats_off);
    a.mass = reinterpret_cast<float*>(ws + p.mass_off);
    a.ctr = reinterpret_cast<unsigned int*>(ws + p.ctr_off);
    a.V = V; a.chunk = p.chunk; a.nchunk = p.nchunk; a.B = (int)B; a.k = (int)k;
    const bool vec = (V % 8 == 0) && ((uintptr_t)zt % 16 == 0) && (zd == nullptr || (uintptr_t)zd % 16 == 0);
    if (temperature == 0.0f) {
        a.R = (int)(k + 1);
        a.c2 = 0.0f;
        dim3 g1((unsigned)p.nchunk, (unsigned)(B * (k + 1)));
        if (vec) hipLaunchKernelGGL(greedy_partial_kernel<true>, g1, dim3(kAThreads), 0, stream, a);
        else hipLaunchKernelGGL(greedy_partial_kernel<false>, g1, dim3(kAThreads), 0, stream, a);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        hipLaunchKernelGGL(greedy_final_kernel, dim3((unsigned)B), dim3(256), 0, stream, a);
        return hipGetLastError();
    }
    a.R = (int)((k + 1) + (zd ? k : 0));
    a.c2 = (float)(1.4426950408889634 / (double)temperature);
    dim3 g1((unsigned)p.nchunk, (unsigned)(B * a.R));
    if (vec) hipLaunchKernelGGL(stoch_stats_kernel<true>, g1, dim3(kAThreads), 0, stream, a);
    else hipLaunchKernelGGL(stoch_stats_kernel<false>, g1, dim3(kAThreads), 0, stream, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    dim3 g2((unsigned)p.nchunk, (unsigned)B);
    if (vec) hipLaunchKernelGGL(stoch_sample_kernel<true>, g2, dim3(kAThreads), 0, stream, a);
    else hipLaunchKernelGGL(stoch_sample_kernel<false>, g2, dim3(kAThreads), 0, stream, a);
    return hipGetLastError();
}

}  // namespace specfp8
