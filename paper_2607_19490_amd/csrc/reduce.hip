// Block reductions over generated data and the reference statistics: the
// live pass fused with Eq. 4 (activations scored in registers), the norms of
// the exact-norm Gaussian tamper of Section 3.2, and the per-block sums
// sum a^2 and sum |a| (mu_i of Eq. 2).  Chunking, workgroup sums and the
// per-element accumulation are those of drift_score.
#include <math.h>

#include "cdt_device.hpp"
#include "cdt_launch.hpp"
#include "cdt_reduce.hpp"
#include "cdt_sim.hpp"

#pragma clang fp contract(off)

namespace cdt {
namespace {

// One chunk of a workgroup's grid-stride walk: its index in the XCD-aware
// order, its block, its groups [g0, g_end) and the rounds of kReduceThreads
// groups (one per thread) that cover them.  Uniform over the workgroup.
struct ReduceChunk {
    uint64_t chunk, block;
    uint32_t g0, g_end, rounds;
};

__device__ __forceinline__ ReduceChunk reduce_chunk(uint64_t it, uint64_t total_chunks,
                                                    uint64_t chunks_per_block, uint32_t n8) {
    ReduceChunk p;
    p.chunk = xcd_contiguous(it, total_chunks);
    p.block = p.chunk / chunks_per_block;
    p.g0 = static_cast<uint32_t>(p.chunk - p.block * chunks_per_block) * kChunkGroups;
    p.g_end = min(p.g0 + kChunkGroups, n8);
    p.rounds = (p.g_end - p.g0 + kReduceThreads - 1) / kReduceThreads;
    return p;
}

// The walk of one workgroup over (chunk, round) in order: thread t handles
// group g0 + round * kReduceThreads + t of each chunk, so a thread meets its
// groups in the order drift_partial_kernel accumulates them.  next() moves
// to the following round, crossing into the workgroup's next chunk, and
// returns false past the last one.
struct ReduceWalk {
    uint64_t it, total_chunks, chunks_per_block;
    uint32_t n8, round;
    ReduceChunk cur;

    __device__ __forceinline__ ReduceWalk(uint64_t first, uint64_t total, uint64_t cpb,
                                          uint32_t n8_)
        : it(first), total_chunks(total), chunks_per_block(cpb), n8(n8_), round(0) {
        if (first < total) cur = reduce_chunk(first, total, cpb, n8_);
    }
    __device__ __forceinline__ bool valid() const { return it < total_chunks; }
    __device__ __forceinline__ bool last_round() const { return round + 1 == cur.rounds; }
    __device__ __forceinline__ uint32_t group() const {
        return cur.g0 + round * kReduceThreads + threadIdx.x;
    }
    __device__ __forceinline__ bool next() {
        if (++round < cur.rounds) return true;
        round = 0;
        it += gridDim.x;
        if (it >= total_chunks) return false;
        cur = reduce_chunk(it, total_chunks, chunks_per_block, n8);
        return true;
    }
};

// Fused live pass and Eq. 4: each group of 8 references is read once, turned
// into fp16 live activations in registers (exactly as canary_sim does), and
// scored at once.  Same chunking, thread-to-group mapping and accumulation
// order as drift_partial_kernel<kL2>, so the block sums are bitwise those of
// canary_sim followed by drift_score.  kStoreH also writes the activations.
// The next group's references are loaded while the current one is
// generated and scored (also across chunks), and the register budget is
// held to 64 (a few spills) so that eight waves share each SIMD.  Per
// 16 x 256 x 256 x 8192 run: 13.1 ms without the prefetch, 12.4 ms with it,
// 12.0 ms with the cap (1024-thread groups), 11.4 ms with 512-thread groups,
// 10.6-11.2 ms with the current 256-thread groups.
template <bool kT3, bool kBlock, bool kStoreH>
__global__ __launch_bounds__(kReduceThreads) __attribute__((amdgpu_waves_per_eu(8, 8)))
void sim_score_partial_kernel(
    SimArgs A, const float* __restrict__ ref, uint16_t* __restrict__ h,
    double* __restrict__ partial) {
    constexpr DriftMetric kM = DriftMetric::kL2;
    const uint64_t n = static_cast<uint64_t>(A.n8) * 8;
    ReduceWalk w(blockIdx.x, A.total_chunks, A.chunks_per_block, A.n8);
    if (!w.valid()) return;
    auto load = [&](const ReduceWalk& at, f32x4& lo, f32x4& hi) {
        lo = f32x4{0.f, 0.f, 0.f, 0.f};
        hi = lo;
        const uint32_t g = at.group();
        if (g < at.cur.g_end) {
            const f32x4* ab = reinterpret_cast<const f32x4*>(ref + at.cur.block * n);
            lo = __builtin_nontemporal_load(ab + 2 * g);
            hi = __builtin_nontemporal_load(ab + 2 * g + 1);
        }
    };
    f32x4 nxt_lo, nxt_hi;
    load(w, nxt_lo, nxt_hi);
    SimBlock B = sim_block<kBlock>(A, w.cur.block);
    double acc[2] = {0.0, 0.0};
    for (;;) {
        const f32x4 a_lo = nxt_lo, a_hi = nxt_hi;
        const uint32_t g = w.group(), g_end = w.cur.g_end;
        const uint64_t chunk = w.cur.chunk, block = w.cur.block;
        const bool chunk_done = w.last_round();
        const bool more = w.next();
        if (more) load(w, nxt_lo, nxt_hi);
        u32x4 hv = u32x4{0u, 0u, 0u, 0u};
        if (g < g_end) {
            hv = sim_group8<kT3, kBlock>(A, B, g * 8, a_lo, a_hi);
            if constexpr (kStoreH)
                __builtin_nontemporal_store(hv, reinterpret_cast<u32x4*>(h + block * n) + g);
        }
        accumulate8<kM>(hv, hv, a_lo, a_hi, acc);
        if (chunk_done) {
            block_sum<2>(acc);
            if (threadIdx.x == 0) {
                partial[chunk * 2] = acc[0];
                partial[chunk * 2 + 1] = acc[1];
            }
            acc[0] = 0.0;
            acc[1] = 0.0;
            if (more) B = sim_block<kBlock>(A, w.cur.block);
        }
        if (!more) break;
    }
}

// Norms for the exact-norm Gaussian tamper of Section 3.2, tau(v) = v +
// eps ||v|| N / ||N||: per block vv = sum v^2 over the untampered output (the
// benign a + delta, or a itself for the clean base) and zz = sum z^2 over
// the TAMPER_ADD normals, both in fp64.  A scale c = eps sqrt(vv / zz) on
// those normals adds a perturbation of norm eps ||v||.
template <bool kT3, bool kBlock>
__global__ __launch_bounds__(kReduceThreads) void tamper_norms_partial_kernel(
    SimArgs A, const float* __restrict__ ref, double* __restrict__ partial) {
    const uint64_t n = static_cast<uint64_t>(A.n8) * 8;
    for (uint64_t it = blockIdx.x; it < A.total_chunks; it += gridDim.x) {
        const uint64_t chunk = xcd_contiguous(it, A.total_chunks);
        const uint64_t b = chunk / A.chunks_per_block;
        const uint32_t g0 = static_cast<uint32_t>(chunk - b * A.chunks_per_block) * kChunkGroups;
        const uint32_t g_end = min(g0 + kChunkGroups, A.n8);
        const SimBlock B = sim_block<kBlock>(A, b);
        const f32x4* ab = reinterpret_cast<const f32x4*>(ref + b * n);
        double acc[2] = {0.0, 0.0};
        for (uint32_t g = g0 + threadIdx.x; g < g_end; g += kReduceThreads) {
            const f32x4 lo = ab[2 * g], hi = ab[2 * g + 1];
            const float a[8] = {lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
            float v[8], z[8];
            if (A.clean) {
#pragma unroll
                for (int k = 0; k < 8; ++k) v[k] = a[k];
            } else {
                benign8<kT3, kBlock>(A, B, g * 8, a, a, v);
            }
            normals8(A.key, g * 8, B.c, B.s, A.tag_add, z);
#pragma unroll
            for (int k = 0; k < 8; ++k) {
                const double vd = static_cast<double>(v[k]), zd = static_cast<double>(z[k]);
                acc[0] = fma(vd, vd, acc[0]);
                acc[1] = fma(zd, zd, acc[1]);
            }
        }
        block_sum<2>(acc);
        if (threadIdx.x == 0) {
            partial[chunk * 2] = acc[0];
            partial[chunk * 2 + 1] = acc[1];
        }
    }
}

// The same norms under the propagation model, for one malicious stage m:
// every element is walked through stages 0 .. m-1 exactly as
// canary_chain_kernel walks it (earlier malicious stages tampered with the
// scales already written to A.tscale), and at stage m the untampered output
// v (or the clean base u) and the TAMPER_ADD normals are summed in fp64.
// Chunks are reduction chunks of one canary's stage-m block: chunk index =
// canary * chunks_per_block + chunk within the block.
template <bool kT3, bool kBlock>
__global__ __launch_bounds__(kReduceThreads) void chain_norms_partial_kernel(
    SimArgs A, uint32_t m, float gain, const float* __restrict__ ref,
    double* __restrict__ partial) {
    const uint64_t n = static_cast<uint64_t>(A.n8) * 8;
    for (uint64_t it = blockIdx.x; it < A.total_chunks; it += gridDim.x) {
        const uint64_t chunk = xcd_contiguous(it, A.total_chunks);
        const uint32_t c = static_cast<uint32_t>(chunk / A.chunks_per_block);
        const uint32_t g0 =
            static_cast<uint32_t>(chunk - static_cast<uint64_t>(c) * A.chunks_per_block) *
            kChunkGroups;
        const uint32_t g_end = min(g0 + kChunkGroups, A.n8);
        double acc[2] = {0.0, 0.0};
        for (uint32_t g = g0 + threadIdx.x; g < g_end; g += kReduceThreads) {
            float d[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll 1
            for (uint32_t s = 0; s < m; ++s) {
                const uint64_t block = static_cast<uint64_t>(s) * A.C + c;
                const SimBlock B = sim_block<kBlock>(A, block);
                const f32x4* in = reinterpret_cast<const f32x4*>(ref + block * n);
                chain_group8<kT3, kBlock>(A, B, g * 8, s == 0, gain, in[2 * g], in[2 * g + 1], d);
            }
            const uint64_t block = static_cast<uint64_t>(m) * A.C + c;
            const SimBlock B = sim_block<kBlock>(A, block);
            const f32x4* in = reinterpret_cast<const f32x4*>(ref + block * n);
            const f32x4 lo = in[2 * g], hi = in[2 * g + 1];
            const float a[8] = {lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
            float u[8], v[8], z[8];
#pragma unroll
            for (int k = 0; k < 8; ++k) u[k] = m == 0 ? a[k] : a[k] + gain * d[k];
            benign8<kT3, kBlock>(A, B, g * 8, a, u, v);
            normals8(A.key, g * 8, B.c, B.s, A.tag_add, z);
#pragma unroll
            for (int k = 0; k < 8; ++k) {
                const double vd = static_cast<double>(A.clean ? u[k] : v[k]);
                const double zd = static_cast<double>(z[k]);
                acc[0] = fma(vd, vd, acc[0]);
                acc[1] = fma(zd, zd, acc[1]);
            }
        }
        block_sum<2>(acc);
        if (threadIdx.x == 0) {
            partial[chunk * 2] = acc[0];
            partial[chunk * 2 + 1] = acc[1];
        }
    }
}

// Stage m's scales from chain_norms_partial_kernel's partials: one thread per
// canary adds its chunks in order.
__global__ void chain_scale_combine_kernel(const double* __restrict__ partial,
                                           uint64_t chunks_per_block, uint32_t C, uint32_t m,
                                           double eps, float* __restrict__ tscale,
                                           double* __restrict__ norms) {
    const uint32_t c = blockIdx.x * blockDim.x + threadIdx.x;
    if (c >= C) return;
    double vv = 0.0, zz = 0.0;
    for (uint64_t i = 0; i < chunks_per_block; ++i) {
        vv += partial[(c * chunks_per_block + i) * 2];
        zz += partial[(c * chunks_per_block + i) * 2 + 1];
    }
    const uint64_t b = static_cast<uint64_t>(m) * C + c;
    tscale[b] = zz > 0.0 ? static_cast<float>(eps * sqrt(vv / zz)) : 0.0f;
    if (norms) {
        norms[2 * b] = vv;
        norms[2 * b + 1] = zz;
    }
}

// Benign stages get no exact-norm scale under the propagation model: their
// entries are cleared first (a kernel, not a memset, so that a stream
// capture records no memset node).
__global__ void clear_scales_kernel(uint64_t nblocks, float* __restrict__ tscale,
                                    double* __restrict__ norms) {
    const uint64_t b = static_cast<uint64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (b >= nblocks) return;
    tscale[b] = 0.0f;
    if (norms) {
        norms[2 * b] = 0.0;
        norms[2 * b + 1] = 0.0;
    }
}

__global__ void tamper_scale_combine_kernel(const double* __restrict__ partial,
                                            uint64_t chunks_per_block, uint64_t nblocks,
                                            double eps, float* __restrict__ tscale,
                                            double* __restrict__ norms) {
    const uint64_t b = static_cast<uint64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (b >= nblocks) return;
    double vv = 0.0, zz = 0.0;
    for (uint64_t i = 0; i < chunks_per_block; ++i) {
        vv += partial[(b * chunks_per_block + i) * 2];
        zz += partial[(b * chunks_per_block + i) * 2 + 1];
    }
    tscale[b] = zz > 0.0 ? static_cast<float>(eps * sqrt(vv / zz)) : 0.0f;
    if (norms) {
        norms[2 * b] = vv;
        norms[2 * b + 1] = zz;
    }
}

__global__ __launch_bounds__(kReduceThreads) void ref_stats_partial_kernel(
    const float* __restrict__ ref, uint32_t n8, uint64_t chunks_per_block, uint64_t total_chunks,
    double2* __restrict__ partial) {
    // Same chunking, XCD order and reads as drift_score: kReduceUnroll groups
    // in flight per thread, the reference in contiguous runs moved to the
    // owning lanes (quads_to_groups); each thread adds its groups in
    // ascending order (groups past the block end contribute exact zeros).
    const uint64_t n = static_cast<uint64_t>(n8) * 8;
    for (uint64_t it = blockIdx.x; it < total_chunks; it += gridDim.x) {
        const uint64_t chunk = xcd_contiguous(it, total_chunks);
        const uint64_t b = chunk / chunks_per_block;
        const uint32_t g0 = static_cast<uint32_t>(chunk - b * chunks_per_block) * kChunkGroups;
        const uint32_t g_end = min(g0 + kChunkGroups, n8);
        const f32x4* ab = reinterpret_cast<const f32x4*>(ref + b * n);
        double Q = 0.0, M = 0.0;
        for (uint32_t base = g0; base < g_end; base += kReduceThreads * kReduceUnroll) {
            f32x4 a0[kReduceUnroll], a1[kReduceUnroll];
            if (base + kReduceThreads * kReduceUnroll <= g_end) {  // workgroup-uniform
                const uint32_t lane = threadIdx.x % kWave, wave0 = threadIdx.x - lane;
#pragma unroll
                for (int u = 0; u < kReduceUnroll; ++u) {
                    const f32x4* aw = ab + 2 * (base + u * kReduceThreads + wave0);
                    quads_to_groups(__builtin_nontemporal_load(aw + lane),
                                    __builtin_nontemporal_load(aw + kWave + lane), a0[u], a1[u]);
                }
            } else {
#pragma unroll
                for (int u = 0; u < kReduceUnroll; ++u) {
                    const uint32_t g = base + u * kReduceThreads + threadIdx.x;
                    a0[u] = f32x4{0.f, 0.f, 0.f, 0.f};
                    a1[u] = a0[u];
                    if (g < g_end) {
                        a0[u] = __builtin_nontemporal_load(ab + 2 * g);
                        a1[u] = __builtin_nontemporal_load(ab + 2 * g + 1);
                    }
                }
            }
#pragma unroll
            for (int u = 0; u < kReduceUnroll; ++u) {
                const float av[8] = {a0[u].x, a0[u].y, a0[u].z, a0[u].w,
                                     a1[u].x, a1[u].y, a1[u].z, a1[u].w};
#pragma unroll
                for (int k = 0; k < 8; ++k) {
                    const double x = static_cast<double>(av[k]);
                    Q = fma(x, x, Q);
                    M += fabs(x);
                }
            }
        }
        double acc[2] = {Q, M};
        block_sum<2>(acc);
        if (threadIdx.x == 0) partial[chunk] = make_double2(acc[0], acc[1]);
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

}  // namespace

template <bool kT3, bool kBlock>
void launch_sim_score_t(const SimArgs& A, dim3 grid, const float* ref, uint16_t* h,
                        double* partial, hipStream_t st) {
    if (h)
        hipLaunchKernelGGL((sim_score_partial_kernel<kT3, kBlock, true>), grid,
                           dim3(kReduceThreads), 0, st, A, ref, h, partial);
    else
        hipLaunchKernelGGL((sim_score_partial_kernel<kT3, kBlock, false>), grid,
                           dim3(kReduceThreads), 0, st, A, ref, h, partial);
}

hipError_t launch_sim_score(const SimLaunch& p, const float* ref, uint16_t* h, float* score,
                            double* num_den, void* ws, hipStream_t st) {
    const uint64_t n = static_cast<uint64_t>(p.T) * p.H;
    const uint64_t nblocks = static_cast<uint64_t>(p.S) * p.C;
    if (nblocks == 0) return hipSuccess;
    const uint64_t cpb = reduce_chunks_per_block(n);
    const uint64_t total = cpb * nblocks;
    double* partial = static_cast<double*>(ws);
    if (total > 0) {
        const SimArgs A = make_sim_args(p, cpb, total);
        const dim3 grid(reduce_grid(total));
        if (A.t3 && A.block_mode)
            launch_sim_score_t<true, true>(A, grid, ref, h, partial, st);
        else if (A.t3)
            launch_sim_score_t<true, false>(A, grid, ref, h, partial, st);
        else if (A.block_mode)
            launch_sim_score_t<false, true>(A, grid, ref, h, partial, st);
        else
            launch_sim_score_t<false, false>(A, grid, ref, h, partial, st);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return launch_drift_combine(DriftMetric::kL2, partial, cpb, nblocks, p.S, p.C, score,
                                num_den, st);
}

hipError_t launch_tamper_scale_exact(const SimLaunch& p, const float* ref, double eps,
                                     float* tscale, double* norms, void* ws, hipStream_t st) {
    const uint64_t n = static_cast<uint64_t>(p.T) * p.H;
    const uint64_t nblocks = static_cast<uint64_t>(p.S) * p.C;
    if (nblocks == 0) return hipSuccess;
    const uint64_t cpb = reduce_chunks_per_block(n);
    const uint64_t total = cpb * nblocks;
    double* partial = static_cast<double*>(ws);
    if (total > 0) {
        const SimArgs A = make_sim_args(p, cpb, total);
        const dim3 grid(reduce_grid(total)), block(kReduceThreads);
        if (A.t3 && A.block_mode)
            hipLaunchKernelGGL((tamper_norms_partial_kernel<true, true>), grid, block, 0, st, A,
                               ref, partial);
        else if (A.t3)
            hipLaunchKernelGGL((tamper_norms_partial_kernel<true, false>), grid, block, 0, st, A,
                               ref, partial);
        else if (A.block_mode)
            hipLaunchKernelGGL((tamper_norms_partial_kernel<false, true>), grid, block, 0, st, A,
                               ref, partial);
        else
            hipLaunchKernelGGL((tamper_norms_partial_kernel<false, false>), grid, block, 0, st, A,
                               ref, partial);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    const uint64_t grid = (nblocks + 255) / 256;
    hipLaunchKernelGGL(tamper_scale_combine_kernel, dim3(static_cast<uint32_t>(grid)), dim3(256),
                       0, st, partial, cpb, nblocks, eps, tscale, norms);
    return hipGetLastError();
}

template <bool kT3, bool kBlock>
void launch_chain_norms_t(const SimArgs& A, uint32_t m, float gain, const float* ref,
                          double* partial, hipStream_t st) {
    hipLaunchKernelGGL((chain_norms_partial_kernel<kT3, kBlock>), dim3(reduce_grid(A.total_chunks)),
                       dim3(kReduceThreads), 0, st, A, m, gain, ref, partial);
}

hipError_t launch_tamper_scale_exact_chain(const SimLaunch& p, const float* ref, double eps,
                                           float* tscale, double* norms, void* ws,
                                           hipStream_t st) {
    const uint64_t n = static_cast<uint64_t>(p.T) * p.H;
    const uint64_t nblocks = static_cast<uint64_t>(p.S) * p.C;
    if (nblocks == 0) return hipSuccess;
    hipLaunchKernelGGL(clear_scales_kernel, dim3(static_cast<uint32_t>((nblocks + 255) / 256)),
                       dim3(256), 0, st, nblocks, tscale, norms);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || n == 0) return e;
    const uint64_t cpb = reduce_chunks_per_block(n);
    // The scales of earlier malicious stages are read from tscale itself.
    SimLaunch q = p;
    q.tscale = tscale;
    const SimArgs A = make_sim_args(q, cpb, cpb * p.C);  // one stage's blocks
    double* partial = static_cast<double*>(ws);
    for (uint32_t m = 0; m < p.S; ++m) {  // malicious stages in pipeline order
        if (!((p.mal_mask >> m) & 1u)) continue;
        if (A.t3 && A.block_mode)
            launch_chain_norms_t<true, true>(A, m, p.carry, ref, partial, st);
        else if (A.t3)
            launch_chain_norms_t<true, false>(A, m, p.carry, ref, partial, st);
        else if (A.block_mode)
            launch_chain_norms_t<false, true>(A, m, p.carry, ref, partial, st);
        else
            launch_chain_norms_t<false, false>(A, m, p.carry, ref, partial, st);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
        hipLaunchKernelGGL(chain_scale_combine_kernel, dim3((p.C + 255) / 256), dim3(256), 0, st,
                           partial, cpb, p.C, m, eps, tscale, norms);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
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
