// Block reductions: the relative-L2 mismatch of Eq. 4 and the reference
// block statistics (sum a^2, sum |a|; mu_i of Eq. 2).
//
// drift_score is bound by HBM bandwidth: 2 B of fp16 h plus 4 B of fp32 a
// per element, each read exactly once.  Layout of the work:
//   * a block (shard, canary) of n = T*H elements is cut into chunks of
//     kReduceChunkElems; one 256-thread workgroup reduces one chunk;
//   * each thread streams groups of 8 elements (one 16-byte h load, two
//     16-byte a loads), kReduceUnroll groups in flight before any use; the
//     loads are nontemporal (read once, no reuse);
//   * chunks are handed out so that each XCD streams one contiguous range;
//   * the squares are accumulated in fp64 from the exactly widened operands
//     (h - a is exact in fp64), so the partial sums carry no cancellation;
//   * wave butterfly sums, then an LDS pass over the waves, give one
//     (D, R) pair per chunk in a fixed order (no atomics);
//   * a combine kernel adds a block's chunk partials in chunk order and
//     forms m = sqrt(D / R).
#include <math.h>

#include "cdt_device.hpp"
#include "cdt_launch.hpp"

#pragma clang fp contract(off)

namespace cdt {
namespace {

constexpr uint32_t kChunkGroups = static_cast<uint32_t>(kReduceChunkElems / 8);
constexpr int kWavesPerGroup = kReduceThreads / kWave;

struct Pair {
    double a, b;
};

// Sum a per-thread pair over the workgroup; thread 0 gets the result.
__device__ __forceinline__ Pair block_sum(Pair v) {
    __shared__ double lds[2][kWavesPerGroup];
    v.a = wave_sum(v.a);
    v.b = wave_sum(v.b);
    const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
    if (lane == 0) {
        lds[0][wave] = v.a;
        lds[1][wave] = v.b;
    }
    __syncthreads();
    Pair r{0.0, 0.0};
    if (threadIdx.x == 0) {
#pragma unroll
        for (int w = 0; w < kWavesPerGroup; ++w) {
            r.a += lds[0][w];
            r.b += lds[1][w];
        }
    }
    __syncthreads();
    return r;
}

__device__ __forceinline__ void accumulate8(const u32x4& hv, const f32x4& a0, const f32x4& a1,
                                            double& D, double& R) {
    const uint32_t hw[4] = {hv.x, hv.y, hv.z, hv.w};
    const float av[8] = {a0.x, a0.y, a0.z, a0.w, a1.x, a1.y, a1.z, a1.w};
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const double h_lo = static_cast<double>(half_bits_to_float(hw[k] & 0xFFFFu));
        const double h_hi = static_cast<double>(half_bits_to_float(hw[k] >> 16));
        const double a_lo = static_cast<double>(av[2 * k]);
        const double a_hi = static_cast<double>(av[2 * k + 1]);
        const double d_lo = h_lo - a_lo;
        const double d_hi = h_hi - a_hi;
        D = fma(d_lo, d_lo, D);
        R = fma(a_lo, a_lo, R);
        D = fma(d_hi, d_hi, D);
        R = fma(a_hi, a_hi, R);
    }
}

__global__ __launch_bounds__(kReduceThreads) void drift_partial_kernel(
    const uint16_t* __restrict__ h, const float* __restrict__ ref, uint32_t n8,
    uint64_t chunks_per_block, uint64_t total_chunks, double2* __restrict__ partial) {
    const uint64_t n = static_cast<uint64_t>(n8) * 8;
    for (uint64_t it = blockIdx.x; it < total_chunks; it += gridDim.x) {
        const uint64_t chunk = xcd_contiguous(it, total_chunks);
        const uint64_t b = chunk / chunks_per_block;
        const uint32_t g0 = static_cast<uint32_t>(chunk - b * chunks_per_block) * kChunkGroups;
        const uint32_t g_end = min(g0 + kChunkGroups, n8);
        const u32x4* hb = reinterpret_cast<const u32x4*>(h + b * n);
        const f32x4* ab = reinterpret_cast<const f32x4*>(ref + b * n);
        double D = 0.0, R = 0.0;
        for (uint32_t base = g0; base < g_end; base += kReduceThreads * kReduceUnroll) {
            u32x4 hv[kReduceUnroll];
            f32x4 a0[kReduceUnroll], a1[kReduceUnroll];
#pragma unroll
            for (int u = 0; u < kReduceUnroll; ++u) {
                const uint32_t g = base + u * kReduceThreads + threadIdx.x;
                if (g < g_end) {
                    hv[u] = __builtin_nontemporal_load(hb + g);
                    a0[u] = __builtin_nontemporal_load(ab + 2 * g);
                    a1[u] = __builtin_nontemporal_load(ab + 2 * g + 1);
                } else {
                    hv[u] = u32x4{0u, 0u, 0u, 0u};
                    a0[u] = f32x4{0.f, 0.f, 0.f, 0.f};
                    a1[u] = a0[u];
                }
            }
#pragma unroll
            for (int u = 0; u < kReduceUnroll; ++u) accumulate8(hv[u], a0[u], a1[u], D, R);
        }
        const Pair s = block_sum(Pair{D, R});
        if (threadIdx.x == 0) partial[chunk] = make_double2(s.a, s.b);
    }
}

__global__ void drift_combine_kernel(const double2* __restrict__ partial, uint64_t chunks_per_block,
                                     uint64_t nblocks, uint32_t S, uint32_t C,
                                     float* __restrict__ score, double* __restrict__ num_den) {
    const uint64_t b = static_cast<uint64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (b >= nblocks) return;
    double D = 0.0, R = 0.0;
    for (uint64_t i = 0; i < chunks_per_block; ++i) {
        const double2 p = partial[b * chunks_per_block + i];
        D += p.x;
        R += p.y;
    }
    double m;
    if (R == 0.0)
        m = (D == 0.0) ? 0.0 : static_cast<double>(INFINITY);
    else
        m = sqrt(D / R);
    const uint64_t s = b / C, c = b - s * C;
    const uint64_t o = c * S + s;
    score[o] = static_cast<float>(m);
    if (num_den) {
        num_den[2 * o] = D;
        num_den[2 * o + 1] = R;
    }
}

__global__ __launch_bounds__(kReduceThreads) void ref_stats_partial_kernel(
    const float* __restrict__ ref, uint32_t n8, uint64_t chunks_per_block, uint64_t total_chunks,
    double2* __restrict__ partial) {
    const uint64_t n = static_cast<uint64_t>(n8) * 8;
    for (uint64_t chunk = blockIdx.x; chunk < total_chunks; chunk += gridDim.x) {
        const uint64_t b = chunk / chunks_per_block;
        const uint32_t g0 = static_cast<uint32_t>(chunk - b * chunks_per_block) * kChunkGroups;
        const uint32_t g_end = min(g0 + kChunkGroups, n8);
        const float4* ab = reinterpret_cast<const float4*>(ref + b * n);
        double Q = 0.0, M = 0.0;
        for (uint32_t g = g0 + threadIdx.x; g < g_end; g += kReduceThreads) {
            const float4 a0 = ab[2 * g];
            const float4 a1 = ab[2 * g + 1];
            const float av[8] = {a0.x, a0.y, a0.z, a0.w, a1.x, a1.y, a1.z, a1.w};
#pragma unroll
            for (int k = 0; k < 8; ++k) {
                const double x = static_cast<double>(av[k]);
                Q = fma(x, x, Q);
                M += fabs(x);
            }
        }
        const Pair s = block_sum(Pair{Q, M});
        if (threadIdx.x == 0) partial[chunk] = make_double2(s.a, s.b);
    }
}

__global__ void ref_stats_combine_kernel(const double2* __restrict__ partial,
                                         uint64_t chunks_per_block, uint64_t nblocks,
                                         double* __restrict__ sumsq, double* __restrict__ sumabs) {
    const uint64_t b = static_cast<uint64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (b >= nblocks) return;
    double Q = 0.0, M = 0.0;
    for (uint64_t i = 0; i < chunks_per_block; ++i) {
        const double2 p = partial[b * chunks_per_block + i];
        Q += p.x;
        M += p.y;
    }
    sumsq[b] = Q;
    sumabs[b] = M;
}

// One workgroup per chunk up to 2^20 chunks, then a grid-stride walk whose
// stride (2^20) is a multiple of the XCD count, as xcd_contiguous needs.
inline uint32_t reduce_grid(uint64_t total_chunks) {
    const uint64_t cap = 1ull << 20;
    return static_cast<uint32_t>(total_chunks < cap ? total_chunks : cap);
}

}  // namespace

hipError_t launch_drift_score(uint32_t S, uint32_t C, uint32_t T, uint32_t H, const uint16_t* h,
                              const float* ref, float* score, double* num_den, void* ws,
                              hipStream_t st) {
    const uint64_t n = static_cast<uint64_t>(T) * H;
    const uint64_t nblocks = static_cast<uint64_t>(S) * C;
    if (nblocks == 0) return hipSuccess;
    const uint64_t cpb = reduce_chunks_per_block(n);
    const uint64_t total = cpb * nblocks;
    double2* partial = static_cast<double2*>(ws);
    if (total > 0) {
        hipLaunchKernelGGL(drift_partial_kernel, dim3(reduce_grid(total)), dim3(kReduceThreads), 0,
                           st, h, ref, static_cast<uint32_t>(n / 8), cpb, total, partial);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    const uint64_t grid = (nblocks + 255) / 256;
    hipLaunchKernelGGL(drift_combine_kernel, dim3(static_cast<uint32_t>(grid)), dim3(256), 0, st,
                       partial, cpb, nblocks, S, C, score, num_den);
    return hipGetLastError();
}

hipError_t launch_ref_stats(uint32_t S, uint32_t C, uint32_t T, uint32_t H, const float* ref,
                            double* sumsq, double* sumabs, void* ws, hipStream_t st) {
    const uint64_t n = static_cast<uint64_t>(T) * H;
    const uint64_t nblocks = static_cast<uint64_t>(S) * C;
    if (nblocks == 0) return hipSuccess;
    const uint64_t cpb = reduce_chunks_per_block(n);
    const uint64_t total = cpb * nblocks;
    double2* partial = static_cast<double2*>(ws);
    if (total > 0) {
        hipLaunchKernelGGL(ref_stats_partial_kernel, dim3(reduce_grid(total)),
                           dim3(kReduceThreads), 0, st, ref, static_cast<uint32_t>(n / 8), cpb,
                           total, partial);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    const uint64_t grid = (nblocks + 255) / 256;
    hipLaunchKernelGGL(ref_stats_combine_kernel, dim3(static_cast<uint32_t>(grid)), dim3(256), 0,
                       st, partial, cpb, nblocks, sumsq, sumabs);
    return hipGetLastError();
}

}  // namespace cdt
