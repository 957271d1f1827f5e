// Eq. 4, the relative-L2 mismatch m = sqrt(sum (h - a)^2 / sum a^2) of
// every (shard, canary) block, and its ablations (an fp16 reference; the
// cosine mismatch of Section 4.4).
//
// drift_score is bound by HBM bandwidth: 2 B of fp16 h plus 4 B of fp32 a
// per element, each read exactly once.  Layout of the work:
//   * a block of n = T*H elements is cut into chunks of kReduceChunkElems;
//     one kReduceThreads-thread workgroup reduces one chunk;
//   * each thread streams groups of 8 elements (one 16-byte h load, two
//     16-byte a loads), kReduceUnroll groups in flight before any use; the
//     loads are nontemporal (read once, no reuse);
//   * an fp32 reference is read so that each load instruction covers one
//     contiguous 1 KB run per wave, then moved across lanes to the thread
//     that owns the elements (quads_to_groups);
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
#include "cdt_reduce.hpp"

#pragma clang fp contract(off)

namespace cdt {
namespace {

// Eq. 4 from the block sums: m = sqrt(D / R); R = 0 gives 0 (D = 0) or +inf.
__device__ __forceinline__ double relative_l2(double D, double R) {
    if (R == 0.0) return (D == 0.0) ? 0.0 : static_cast<double>(INFINITY);
    return sqrt(D / R);
}

// 1 - cos(h, a) from D = |h-a|^2, A = |a|^2, P = a.(h-a): with |h|^2 = A + 2P + D
// and h.a = A + P, 1 - cos = (A D - P^2) / (sqrt(A |h|^2) (sqrt(A |h|^2) + A + P)),
// which keeps full relative accuracy as the angle goes to 0.
__device__ __forceinline__ double cosine_mismatch(double D, double A, double P) {
    const double hn = A + 2.0 * P + D;
    if (A == 0.0 || hn <= 0.0) return (A == 0.0 && hn <= 0.0) ? 0.0 : 1.0;
    const double g = sqrt(A * hn);
    const double dot = A + P;
    if (dot > 0.0) return (A * D - P * P) / (g * (g + dot));
    return 1.0 - dot / g;
}

// Score and optional sums of block b = s * C + c from its total sums,
// written at [c][s] (scores) and [c][s][k] (sums).
template <DriftMetric kM>
__device__ __forceinline__ void finish_block(const double (&acc)[DriftTraits<kM>::kSums],
                                             uint64_t b, uint32_t S, uint32_t C,
                                             float* __restrict__ score, double* __restrict__ sums) {
    using Tr = DriftTraits<kM>;
    double m;
    if constexpr (Tr::kCos)
        m = cosine_mismatch(acc[0], acc[1], acc[2]);
    else
        m = relative_l2(acc[0], acc[1]);
    const uint64_t s = b / C, c = b - s * C;
    const uint64_t o = c * S + s;
    score[o] = static_cast<float>(m);
    if (sums) {
#pragma unroll
        for (int k = 0; k < Tr::kSums; ++k) sums[Tr::kSums * o + k] = acc[k];
    }
}

// XOR of every word a thread loaded; a value no load pattern is meant to
// produce selects the (practically never taken) store that keeps the loads.
constexpr uint32_t kFoldSentinel = 0x7F3A5C91u;

__device__ __forceinline__ uint32_t fold_group(const u32x4& hv, const u32x4& rv, const f32x4& a0,
                                               const f32x4& a1) {
    uint32_t x = hv.x ^ hv.y ^ hv.z ^ hv.w ^ rv.x ^ rv.y ^ rv.z ^ rv.w;
#pragma unroll
    for (int k = 0; k < 4; ++k) x ^= __float_as_uint(a0[k]) ^ __float_as_uint(a1[k]);
    return x;
}

// kReadOnly: the same chunks, loads and lane exchange with Eq. 4's
// arithmetic replaced by an XOR fold of the loaded words: the rate the memory
// system gives this access pattern, against which the drift kernel is judged.
// direct (a block is one chunk): the chunk's sums are the block's, and the
// score is written here; the combine launch is skipped (it would add the one
// partial to zero, which changes nothing).
// One chunk of one block array: its partial sums (or, direct, its block's
// score), in a fixed order.  Shared by the single-array and batched launches.
template <DriftMetric kM, bool kReadOnly>
__device__ __forceinline__ void drift_chunk(const uint16_t* __restrict__ h,
                                            const void* __restrict__ ref, uint32_t n8,
                                            uint64_t chunks_per_block, uint64_t chunk,
                                            double* __restrict__ partial, bool direct, uint32_t S,
                                            uint32_t C, float* __restrict__ score,
                                            double* __restrict__ sums) {
    using Tr = DriftTraits<kM>;
    const uint64_t n = static_cast<uint64_t>(n8) * 8;
    {
        const uint64_t b = chunk / chunks_per_block;
        const uint32_t g0 = static_cast<uint32_t>(chunk - b * chunks_per_block) * kChunkGroups;
        const uint32_t g_end = min(g0 + kChunkGroups, n8);
        const gptr<const u32x4> hb = global_ptr(reinterpret_cast<const u32x4*>(h + b * n));
        gptr<const f32x4> ab = nullptr;  // fp32 reference block
        gptr<const u32x4> rb = nullptr;  // fp16 reference block
        if constexpr (Tr::kHalfRef)
            rb = global_ptr(
                reinterpret_cast<const u32x4*>(static_cast<const uint16_t*>(ref) + b * n));
        else
            ab = global_ptr(
                reinterpret_cast<const f32x4*>(static_cast<const float*>(ref) + b * n));
        double acc[Tr::kSums];
#pragma unroll
        for (int k = 0; k < Tr::kSums; ++k) acc[k] = 0.0;
        uint32_t fold = 0;
        for (uint32_t base = g0; base < g_end; base += kReduceThreads * kReduceUnroll) {
            u32x4 hv[kReduceUnroll], rv[kReduceUnroll];
            f32x4 a0[kReduceUnroll], a1[kReduceUnroll];
            if (!Tr::kHalfRef && base + kReduceThreads * kReduceUnroll <= g_end) {
                // every group of the step is in range (workgroup-uniform)
                const uint32_t lane = threadIdx.x % kWave, wave0 = threadIdx.x - lane;
#pragma unroll
                for (int u = 0; u < kReduceUnroll; ++u) {
                    const uint32_t g = base + u * kReduceThreads + threadIdx.x;
                    const gptr<const f32x4> aw = ab + 2 * (base + u * kReduceThreads + wave0);
                    hv[u] = __builtin_nontemporal_load(hb + g);
                    rv[u] = u32x4{0u, 0u, 0u, 0u};
                    quads_to_groups(__builtin_nontemporal_load(aw + lane),
                                    __builtin_nontemporal_load(aw + kWave + lane), a0[u], a1[u]);
                }
#pragma unroll
                for (int u = 0; u < kReduceUnroll; ++u) {
                    if constexpr (kReadOnly)
                        fold ^= fold_group(hv[u], rv[u], a0[u], a1[u]);
                    else
                        accumulate8<kM>(hv[u], rv[u], a0[u], a1[u], acc);
                }
                continue;
            }
#pragma unroll
            for (int u = 0; u < kReduceUnroll; ++u) {
                const uint32_t g = base + u * kReduceThreads + threadIdx.x;
                hv[u] = u32x4{0u, 0u, 0u, 0u};
                rv[u] = hv[u];
                a0[u] = f32x4{0.f, 0.f, 0.f, 0.f};
                a1[u] = a0[u];
                if (g < g_end) {
                    hv[u] = __builtin_nontemporal_load(hb + g);
                    if constexpr (Tr::kHalfRef) {
                        rv[u] = __builtin_nontemporal_load(rb + g);
                    } else {
                        a0[u] = __builtin_nontemporal_load(ab + 2 * g);
                        a1[u] = __builtin_nontemporal_load(ab + 2 * g + 1);
                    }
                }
            }
#pragma unroll
            for (int u = 0; u < kReduceUnroll; ++u) {
                if constexpr (kReadOnly)
                    fold ^= fold_group(hv[u], rv[u], a0[u], a1[u]);
                else
                    accumulate8<kM>(hv[u], rv[u], a0[u], a1[u], acc);
            }
        }
        if constexpr (kReadOnly) {
            if (fold == kFoldSentinel) {
                if (direct) score[0] = __uint_as_float(fold);
                else partial[chunk * Tr::kSums] = static_cast<double>(fold);
            }
        } else {
            block_sum<Tr::kSums>(acc);
            if (threadIdx.x == 0) {
                if (direct) {
                    finish_block<kM>(acc, chunk, S, C, score, sums);
                } else {
#pragma unroll
                    for (int k = 0; k < Tr::kSums; ++k) partial[chunk * Tr::kSums + k] = acc[k];
                }
            }
        }
    }
}

template <DriftMetric kM, bool kReadOnly = false>
__global__ __launch_bounds__(kReduceThreads) void drift_partial_kernel(
    const uint16_t* __restrict__ h, const void* __restrict__ ref, uint32_t n8,
    uint64_t chunks_per_block, uint64_t total_chunks, double* __restrict__ partial, bool direct,
    uint32_t S, uint32_t C, float* __restrict__ score, double* __restrict__ sums) {
    for (uint64_t it = blockIdx.x; it < total_chunks; it += gridDim.x)
        drift_chunk<kM, kReadOnly>(h, ref, n8, chunks_per_block, xcd_contiguous(it, total_chunks),
                                   partial, direct, S, C, score, sums);
}

// Eq. 4's element step for kJ arrays against one reference: the reference
// value is widened once, its square added once to the shared R (it is the
// same sum for every job), and each job's d = h - a squared into its own D.
// Each accumulator sees the same values in the same order as accumulate8's.
template <int kJ>
__device__ __forceinline__ void accumulate8_jobs(const u32x4 (&hv)[kJ], const f32x4& a0,
                                                 const f32x4& a1, double (&d_acc)[kJ],
                                                 double& r_acc) {
    const float av[8] = {a0.x, a0.y, a0.z, a0.w, a1.x, a1.y, a1.z, a1.w};
#pragma unroll
    for (int k = 0; k < 4; ++k) {
#pragma unroll
        for (int half = 0; half < 2; ++half) {
            const double a = static_cast<double>(av[2 * k + half]);
            r_acc = fma(a, a, r_acc);
#pragma unroll
            for (int j = 0; j < kJ; ++j) {
                const uint32_t w = (k == 0 ? hv[j].x : k == 1 ? hv[j].y : k == 2 ? hv[j].z : hv[j].w);
                const double h = static_cast<double>(half_bits_to_float(half ? w >> 16 : w & 0xFFFFu));
                const double d = h - a;
                d_acc[j] = fma(d, d, d_acc[j]);
            }
        }
    }
}

// One chunk of kJ arrays scored against one shared reference (Eq. 4): each
// step's reference groups are loaded once and every job's activations of
// the step are loaded at once and accumulated against them; the
// reference's own sum R is formed once for all of them.  The reference is
// read with ordinary (cached) loads, unlike drift_chunk's nontemporal ones:
// the later units of a group of more than 8 jobs re-read the chunk, and
// then find it in L2 (the 216-configuration sweep's Eq. 4: 12.9-13.2 ms
// against 13.6-13.8 ms; the 70B step's single unit is unchanged).  The step is kMultiUnroll groups per thread
// (not drift_chunk's kReduceUnroll, so that every job's loads fit in
// registers together); a thread still visits its groups g0 + tid + 256 m in
// the order m = 0, 1, 2, ... and adds the same values in the same order as
// drift_chunk, so each job's sums are bitwise those of one launch per job.
// With 8 jobs that is 256 VGPRs (no spills), the same two waves per SIMD as
// 3 or 4 jobs take; 2 groups per step for 5-8 jobs measured no faster.
constexpr int kMultiUnroll = 4;

template <int kJ, bool kReadOnly = false>
__device__ __forceinline__ void drift_chunk_jobs(const DriftJobDev* __restrict__ jobs,
                                                 uint64_t chunk) {
    constexpr int kU = kMultiUnroll;
    const DriftJobDev& J0 = jobs[0];
    const uint64_t n = static_cast<uint64_t>(J0.n8) * 8;
    const uint64_t b = chunk / J0.cpb;
    const uint32_t g0 = static_cast<uint32_t>(chunk - b * J0.cpb) * kChunkGroups;
    const uint32_t g_end = min(g0 + kChunkGroups, J0.n8);
    const gptr<const f32x4> ab = global_ptr(reinterpret_cast<const f32x4*>(J0.ref + b * n));
    gptr<const u32x4> hb[kJ];
#pragma unroll
    for (int j = 0; j < kJ; ++j) hb[j] = global_ptr(reinterpret_cast<const u32x4*>(jobs[j].h + b * n));
    const u32x4 zero = u32x4{0u, 0u, 0u, 0u};
    double d_acc[kJ], r_acc = 0.0;
#pragma unroll
    for (int j = 0; j < kJ; ++j) d_acc[j] = 0.0;
    uint32_t fold = 0;
    for (uint32_t base = g0; base < g_end; base += kReduceThreads * kU) {
        f32x4 a0[kU], a1[kU];
        u32x4 hv[kJ][kU];
        if (base + kReduceThreads * kU <= g_end) {
            // every group of the step is in range (workgroup-uniform)
            const uint32_t lane = threadIdx.x % kWave, wave0 = threadIdx.x - lane;
#pragma unroll
            for (int u = 0; u < kU; ++u) {
                const gptr<const f32x4> aw = ab + 2 * (base + u * kReduceThreads + wave0);
                const f32x4 r0 = aw[lane], r1 = aw[kWave + lane];
                quads_to_groups(r0, r1, a0[u], a1[u]);
            }
#pragma unroll
            for (int j = 0; j < kJ; ++j)
#pragma unroll
                for (int u = 0; u < kU; ++u)
                    hv[j][u] =
                        __builtin_nontemporal_load(hb[j] + base + u * kReduceThreads + threadIdx.x);
        } else {
            // the last, partial step of a ragged block: every lane loads an
            // element in range (its own, or the chunk's last) and keeps zeros
            // where its own is out of range
#pragma unroll
            for (int u = 0; u < kU; ++u) {
                const uint32_t g = base + u * kReduceThreads + threadIdx.x;
                const uint32_t gc = g < g_end ? g : g_end - 1;
                const f32x4 l0 = ab[2 * gc];
                const f32x4 l1 = ab[2 * gc + 1];
                const f32x4 z = f32x4{0.f, 0.f, 0.f, 0.f};
                a0[u] = g < g_end ? l0 : z;
                a1[u] = g < g_end ? l1 : z;
#pragma unroll
                for (int j = 0; j < kJ; ++j) {
                    const u32x4 l = __builtin_nontemporal_load(hb[j] + gc);
                    hv[j][u] = g < g_end ? l : zero;
                }
            }
        }
#pragma unroll
        for (int u = 0; u < kU; ++u) {
            u32x4 hu[kJ];
#pragma unroll
            for (int j = 0; j < kJ; ++j) hu[j] = hv[j][u];
            if constexpr (kReadOnly) {
                fold ^= fold_group(hu[0], zero, a0[u], a1[u]);
#pragma unroll
                for (int j = 1; j < kJ; ++j) fold ^= hu[j].x ^ hu[j].y ^ hu[j].z ^ hu[j].w;
            } else {
                accumulate8_jobs<kJ>(hu, a0[u], a1[u], d_acc, r_acc);
            }
        }
    }
    if constexpr (kReadOnly) {  // keeps the loads; the sentinel never occurs in practice
        if (fold == kFoldSentinel) jobs[0].score[0] = __uint_as_float(fold);
        return;
    }
    double sums[kJ + 1];
#pragma unroll
    for (int j = 0; j < kJ; ++j) sums[j] = d_acc[j];
    sums[kJ] = r_acc;
    block_sum<kJ + 1>(sums);
    if (threadIdx.x == 0) {
#pragma unroll
        for (int j = 0; j < kJ; ++j) {
            const DriftJobDev& J = jobs[j];
            const double acc[2] = {sums[j], sums[kJ]};
            if (J.direct) {
                finish_block<DriftMetric::kL2>(acc, chunk, J.S, J.C, J.score, J.sums);
            } else {
                J.partial[chunk * 2] = acc[0];
                J.partial[chunk * 2 + 1] = acc[1];
            }
        }
    }
}

// Batched Eq. 4: the jobs' chunks form one iteration range walked by one
// grid, group by group (batch_iter): jobs sharing a reference are taken up
// to kDriftJobsPerIter at a time per chunk (drift_chunk_jobs reads the
// reference chunk once for them), chunk-major, each XCD on its own eighth
// of the group.  Every job's sums are bitwise those of the single launch.
// The combine kernel finds a block's job by a binary search over the jobs'
// first blocks.
__device__ __forceinline__ uint32_t find_job(const DriftJobDev* __restrict__ jobs,
                                             uint32_t n_jobs, uint64_t block) {
    uint32_t lo = 0, hi = n_jobs;  // last job whose first block <= block
    while (hi - lo > 1) {
        const uint32_t mid = (lo + hi) / 2;
        if (jobs[mid].block_begin <= block) lo = mid; else hi = mid;
    }
    return lo;
}

template <bool kReadOnly>
__global__ __launch_bounds__(kReduceThreads) void drift_batch_partial_kernel(
    const DriftJobDev* __restrict__ jobs, const BatchGroupDev* __restrict__ groups,
    uint32_t n_groups, uint64_t total_iters) {
    for (uint64_t it = blockIdx.x; it < total_iters; it += gridDim.x) {
        uint32_t j, unit_jobs, group_jobs;
        uint64_t chunk;
        if (!batch_iter(groups, n_groups, it, &j, &unit_jobs, &chunk, &group_jobs)) continue;
        static_assert(kDriftJobsPerIter == 8, "one case per unit size");
        if (unit_jobs == 8) {
            drift_chunk_jobs<8, kReadOnly>(jobs + j, chunk);
        } else if (unit_jobs == 7) {
            drift_chunk_jobs<7, kReadOnly>(jobs + j, chunk);
        } else if (unit_jobs == 6) {
            drift_chunk_jobs<6, kReadOnly>(jobs + j, chunk);
        } else if (unit_jobs == 5) {
            drift_chunk_jobs<5, kReadOnly>(jobs + j, chunk);
        } else if (unit_jobs == 4) {
            drift_chunk_jobs<4, kReadOnly>(jobs + j, chunk);
        } else if (unit_jobs == 3) {
            drift_chunk_jobs<3, kReadOnly>(jobs + j, chunk);
        } else if (unit_jobs == 2) {
            drift_chunk_jobs<2, kReadOnly>(jobs + j, chunk);
        } else {
            const DriftJobDev& J = jobs[j];
            drift_chunk<DriftMetric::kL2, kReadOnly>(J.h, J.ref, J.n8, J.cpb, chunk, J.partial,
                                                     J.direct, J.S, J.C, J.score, J.sums);
        }
    }
}

__global__ void drift_batch_combine_kernel(const DriftJobDev* __restrict__ jobs, uint32_t n_jobs,
                                           uint64_t total_blocks) {
    const uint64_t g = static_cast<uint64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (g >= total_blocks) return;
    const DriftJobDev& J = jobs[find_job(jobs, n_jobs, g)];
    if (J.direct) return;  // scored by the partial kernel itself
    const uint64_t b = g - J.block_begin;
    double acc[2] = {0.0, 0.0};
    for (uint64_t i = 0; i < J.cpb; ++i) {
        acc[0] += J.partial[(b * J.cpb + i) * 2];
        acc[1] += J.partial[(b * J.cpb + i) * 2 + 1];
    }
    finish_block<DriftMetric::kL2>(acc, b, J.S, J.C, J.score, J.sums);
}

template <DriftMetric kM>
__global__ void drift_combine_kernel(const double* __restrict__ partial, uint64_t chunks_per_block,
                                     uint64_t nblocks, uint32_t S, uint32_t C,
                                     float* __restrict__ score, double* __restrict__ sums) {
    using Tr = DriftTraits<kM>;
    const uint64_t b = static_cast<uint64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (b >= nblocks) return;
    double acc[Tr::kSums];
#pragma unroll
    for (int k = 0; k < Tr::kSums; ++k) acc[k] = 0.0;
    for (uint64_t i = 0; i < chunks_per_block; ++i) {
#pragma unroll
        for (int k = 0; k < Tr::kSums; ++k) acc[k] += partial[(b * chunks_per_block + i) * Tr::kSums + k];
    }
    finish_block<kM>(acc, b, S, C, score, sums);
}

}  // namespace

template <DriftMetric kM>
hipError_t launch_combine_t(const double* partial, uint64_t cpb, uint64_t nblocks, uint32_t S,
                            uint32_t C, float* score, double* sums, hipStream_t st) {
    const uint64_t grid = (nblocks + 255) / 256;
    hipLaunchKernelGGL(drift_combine_kernel<kM>, dim3(static_cast<uint32_t>(grid)), dim3(256), 0,
                       st, partial, cpb, nblocks, S, C, score, sums);
    return hipGetLastError();
}

template <DriftMetric kM>
hipError_t launch_drift_t(uint32_t S, uint32_t C, uint32_t T, uint32_t H, const uint16_t* h,
                          const void* ref, float* score, double* sums, void* ws, hipStream_t st) {
    const uint64_t n = static_cast<uint64_t>(T) * H;
    const uint64_t nblocks = static_cast<uint64_t>(S) * C;
    if (nblocks == 0) return hipSuccess;
    const uint64_t cpb = reduce_chunks_per_block(n);
    const uint64_t total = cpb * nblocks;
    double* partial = static_cast<double*>(ws);
    const bool direct = cpb == 1;
    if (total > 0) {
        hipLaunchKernelGGL(drift_partial_kernel<kM>, dim3(reduce_grid(total)),
                           dim3(kReduceThreads), 0, st, h, ref, static_cast<uint32_t>(n / 8), cpb,
                           total, partial, direct, S, C, score, sums);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    if (direct) return hipSuccess;
    return launch_combine_t<kM>(partial, cpb, nblocks, S, C, score, sums, st);
}

hipError_t launch_drift_batch(const DriftJobDev* jobs_dev, uint32_t n_jobs,
                              const BatchGroupDev* groups_dev, uint32_t n_groups,
                              uint64_t total_iters, uint64_t total_blocks, hipStream_t st) {
    if (n_jobs == 0) return hipSuccess;
    if (total_iters > 0) {
        hipLaunchKernelGGL(drift_batch_partial_kernel<false>, dim3(reduce_grid(total_iters)),
                           dim3(kReduceThreads), 0, st, jobs_dev, groups_dev, n_groups,
                           total_iters);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    if (total_blocks == 0) return hipSuccess;
    const uint64_t grid = (total_blocks + 255) / 256;
    hipLaunchKernelGGL(drift_batch_combine_kernel, dim3(static_cast<uint32_t>(grid)), dim3(256), 0,
                       st, jobs_dev, n_jobs, total_blocks);
    return hipGetLastError();
}

hipError_t launch_drift_batch_read_stream(const DriftJobDev* jobs_dev,
                                          const BatchGroupDev* groups_dev, uint32_t n_groups,
                                          uint64_t total_iters, hipStream_t st) {
    if (total_iters == 0) return hipSuccess;
    hipLaunchKernelGGL(drift_batch_partial_kernel<true>, dim3(reduce_grid(total_iters)),
                       dim3(kReduceThreads), 0, st, jobs_dev, groups_dev, n_groups, total_iters);
    return hipGetLastError();
}

hipError_t launch_drift_read_stream(uint32_t S, uint32_t C, uint32_t T, uint32_t H,
                                   const uint16_t* h, const float* ref, void* ws, hipStream_t st) {
    const uint64_t n = static_cast<uint64_t>(T) * H;
    const uint64_t total = reduce_chunks_per_block(n) * S * C;
    if (total == 0) return hipSuccess;
    hipLaunchKernelGGL((drift_partial_kernel<DriftMetric::kL2, true>), dim3(reduce_grid(total)),
                       dim3(kReduceThreads), 0, st, h, ref, static_cast<uint32_t>(n / 8),
                       reduce_chunks_per_block(n), total, static_cast<double*>(ws), false, S, C,
                       nullptr, nullptr);
    return hipGetLastError();
}

hipError_t launch_drift(DriftMetric metric, uint32_t S, uint32_t C, uint32_t T, uint32_t H,
                        const uint16_t* h, const void* ref, float* score, double* sums, void* ws,
                        hipStream_t st) {
    switch (metric) {
        case DriftMetric::kL2:
            return launch_drift_t<DriftMetric::kL2>(S, C, T, H, h, ref, score, sums, ws, st);
        case DriftMetric::kL2HalfRef:
            return launch_drift_t<DriftMetric::kL2HalfRef>(S, C, T, H, h, ref, score, sums, ws,
                                                           st);
        case DriftMetric::kCosine:
            return launch_drift_t<DriftMetric::kCosine>(S, C, T, H, h, ref, score, sums, ws, st);
        case DriftMetric::kCosineHalfRef:
            return launch_drift_t<DriftMetric::kCosineHalfRef>(S, C, T, H, h, ref, score, sums,
                                                               ws, st);
    }
    return hipErrorInvalidValue;
}

hipError_t launch_drift_combine(DriftMetric metric, const double* partial, uint64_t cpb,
                                uint64_t nblocks, uint32_t S, uint32_t C, float* score,
                                double* sums, hipStream_t st) {
    switch (metric) {
        case DriftMetric::kL2:
            return launch_combine_t<DriftMetric::kL2>(partial, cpb, nblocks, S, C, score, sums, st);
        case DriftMetric::kL2HalfRef:
            return launch_combine_t<DriftMetric::kL2HalfRef>(partial, cpb, nblocks, S, C, score,
                                                             sums, st);
        case DriftMetric::kCosine:
            return launch_combine_t<DriftMetric::kCosine>(partial, cpb, nblocks, S, C, score, sums,
                                                          st);
        case DriftMetric::kCosineHalfRef:
            return launch_combine_t<DriftMetric::kCosineHalfRef>(partial, cpb, nblocks, S, C,
                                                                 score, sums, st);
    }
    return hipErrorInvalidValue;
}

}  // namespace cdt
