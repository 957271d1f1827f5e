// Generator kernels: synthetic fp32 references (stand-in for the verifier's
// offline pass of Eq. 1), per-block scales, and the simulated live pass of
// Eqs. 2-3 (benign hardware noise, tampering, fp16 hand-off).
//
// Every random number comes from Philox4x32-10 evaluated in registers from
// its counter, so noise and tamper directions never touch HBM: a thread
// reads 8 fp32 references (two 16-byte loads) and writes 8 fp16 activations
// (one 16-byte store).  All fp32 arithmetic is written one operation per
// step with FMA contraction off, so results are reproducible bit for bit.
#include <math.h>
#include <string.h>

#include <vector>

#include "cdt_device.hpp"
#include "cdt_launch.hpp"
#include "cdt_sim.hpp"

#pragma clang fp contract(off)

namespace cdt {
namespace {

constexpr uint32_t kMaxOutlierH = 32768;

// ---------------------------------------------------------------------------
// Outlier channels: every workgroup draws all H channel words into LDS, then
// each thread ranks one channel against all of them.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void outlier_gain_kernel(uint32_t H, uint32_t n_out, float big,
                                                           Key key, uint32_t tag,
                                                           float* __restrict__ gain) {
    __shared__ uint32_t words[kMaxOutlierH];
    for (uint32_t j = threadIdx.x; j < H; j += blockDim.x) words[j] = draw(key, j, 0, 0, tag).x;
    __syncthreads();
    const uint32_t j = blockIdx.x * blockDim.x + threadIdx.x;
    if (j >= H) return;
    const uint32_t wj = words[j];
    uint32_t rank = 0;
    for (uint32_t i = 0; i < H; ++i) {
        const uint32_t wi = words[i];
        rank += (wi < wj) || (wi == wj && i < j);
    }
    gain[j] = rank < n_out ? big : 1.0f;
}

// ---------------------------------------------------------------------------
// Streamed loads and stores of the elementwise kernels (each byte is touched
// once per launch).  The fp16 output is stored nontemporally: it leaves no
// dirty lines behind in L2 / the Infinity Cache for the next kernel to evict.
// ---------------------------------------------------------------------------
template <typename P>
__device__ __forceinline__ f32x4 load_stream(P p) { return *p; }
template <typename P>
__device__ __forceinline__ void store_stream(P p, u32x4 v) {
    __builtin_nontemporal_store(v, p);
}

// ---------------------------------------------------------------------------
// Chunk walk shared by the elementwise kernels: chunk -> (block, first group).
// ---------------------------------------------------------------------------
struct ChunkPos {
    uint64_t block;
    uint32_t s, c;
    uint32_t g0;  // first 8-element group of this chunk inside the block
};

__device__ __forceinline__ ChunkPos chunk_pos(uint64_t chunk, uint64_t chunks_per_block,
                                              uint32_t C, uint32_t chunk_groups = kGenChunkGroups) {
    ChunkPos p;
    p.block = chunk / chunks_per_block;
    p.g0 = static_cast<uint32_t>(chunk - p.block * chunks_per_block) * chunk_groups;
    p.s = static_cast<uint32_t>(p.block / C);
    p.c = static_cast<uint32_t>(p.block - static_cast<uint64_t>(p.s) * C);
    return p;
}

// ---------------------------------------------------------------------------
// Synthetic references: ref = fp32(z_REF * gain[j]).
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kGenThreads) void ref_synth_kernel(
    uint32_t C, uint32_t canary_base, uint32_t H, uint32_t n8, uint64_t chunks_per_block,
    uint64_t total_chunks, Key key, uint32_t tag, const float* __restrict__ gain,
    float* __restrict__ ref) {
    const uint64_t n = static_cast<uint64_t>(n8) * 8;
    for (uint64_t it = blockIdx.x; it < total_chunks; it += gridDim.x) {
        const ChunkPos p = chunk_pos(xcd_contiguous(it, total_chunks), chunks_per_block, C);
        float4* out = reinterpret_cast<float4*>(ref + p.block * n);
#pragma unroll
        for (int item = 0; item < kGenItems; ++item) {
            const uint32_t g = p.g0 + item * kGenThreads + threadIdx.x;
            if (g >= n8) break;
            const uint32_t e0 = g * 8;
            const uint32_t j0 = e0 % H;
            const float4 g_lo = *reinterpret_cast<const float4*>(gain + j0);
            const float4 g_hi = *reinterpret_cast<const float4*>(gain + j0 + 4);
            float z[8];
            normals8(key, e0, canary_base + p.c, p.s, tag, z);
            out[2 * g] = make_float4(z[0] * g_lo.x, z[1] * g_lo.y, z[2] * g_lo.z, z[3] * g_lo.w);
            out[2 * g + 1] =
                make_float4(z[4] * g_hi.x, z[5] * g_hi.y, z[6] * g_hi.z, z[7] * g_hi.w);
        }
    }
}

// ---------------------------------------------------------------------------
// Per-block scales (fp64, rounded once to fp32).
// ---------------------------------------------------------------------------
__global__ void block_scales_kernel(uint64_t nblocks, double n, const double* __restrict__ sumsq,
                                    const double* __restrict__ sumabs, double eps, double sigma_b,
                                    float* __restrict__ tscale, float* __restrict__ bscale) {
    const uint64_t b = static_cast<uint64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
    if (b >= nblocks) return;
    if (tscale) {
        const double rms = n > 0 ? sqrt(sumsq[b] / n) : 0.0;
        tscale[b] = static_cast<float>(eps * rms);
    }
    if (bscale) {
        const double mu = n > 0 ? sumabs[b] / n : 0.0;
        bscale[b] = static_cast<float>(sigma_b * mu);
    }
}

// ---------------------------------------------------------------------------
// Live pass (Eqs. 2-3) -> fp16.
// ---------------------------------------------------------------------------
// Specialised on the two launch-uniform noise modes so that the common
// (Gaussian, elementwise) path carries no Student-t or block-scale code.
template <bool kT3>
constexpr int sim_threads() { return kGenThreads; }

template <bool kT3>
constexpr uint32_t sim_chunk_groups() { return sim_threads<kT3>() * kGenItems; }

// kStream: the same chunks, loads, prefetch and stores with the live pass
// replaced by h = fp16(a) (no random numbers): the memory bound of the live
// pass's access pattern, against which the live pass is judged.
// One chunk of one run's live pass; shared by the single-run and batched
// launches.
template <bool kT3, bool kBlock, bool kStream>
__device__ __forceinline__ void sim_chunk(const SimArgs& A, uint64_t chunk,
                                          const float* __restrict__ ref,
                                          uint16_t* __restrict__ h) {
    constexpr int kThreads = sim_threads<kT3>();
    const uint64_t n = static_cast<uint64_t>(A.n8) * 8;
    {
        const ChunkPos p = chunk_pos(chunk, A.chunks_per_block, A.C, sim_chunk_groups<kT3>());
        const SimBlock B = sim_block<kBlock>(A, p.block);
        const gptr<const f32x4> in = global_ptr(reinterpret_cast<const f32x4*>(ref + p.block * n));
        const gptr<u32x4> out = global_ptr(reinterpret_cast<u32x4*>(h + p.block * n));
        // Double buffer: the next group's reference loads are issued before
        // the Philox work on the current group, so loads overlap the ALU work.
        uint32_t g = p.g0 + threadIdx.x;
        f32x4 nxt_lo = f32x4{0.f, 0.f, 0.f, 0.f}, nxt_hi = nxt_lo;
        if (g < A.n8) {
            nxt_lo = load_stream(in + 2 * g);
            nxt_hi = load_stream(in + 2 * g + 1);
        }
#pragma unroll 1
        for (int item = 0; item < kGenItems; ++item, g += kThreads) {
            if (g >= A.n8) break;
            const f32x4 a_lo = nxt_lo, a_hi = nxt_hi;
            const uint32_t g_next = g + kThreads;
            if (item + 1 < kGenItems && g_next < A.n8) {
                nxt_lo = load_stream(in + 2 * g_next);
                nxt_hi = load_stream(in + 2 * g_next + 1);
            }
            if constexpr (kStream) {
                const float a[8] = {a_lo.x, a_lo.y, a_lo.z, a_lo.w, a_hi.x, a_hi.y, a_hi.z, a_hi.w};
                store_stream(out + g, pack_half8(a));
            } else {
                store_stream(out + g, sim_group8<kT3, kBlock>(A, B, g * 8, a_lo, a_hi));
            }
        }
    }
}

template <bool kT3, bool kBlock, bool kStream = false>
__global__ __launch_bounds__(sim_threads<kT3>()) void canary_sim_kernel(
    SimArgs A, const float* __restrict__ ref, uint16_t* __restrict__ h) {
    for (uint64_t it = blockIdx.x; it < A.total_chunks; it += gridDim.x)
        sim_chunk<kT3, kBlock, kStream>(A, xcd_contiguous(it, A.total_chunks), ref, h);
}

// Batched live pass: the jobs' chunks form one iteration range walked by
// one grid, group by group (batch_iter): the runs of a group share their
// references and are walked chunk-major, so a reference chunk is read from
// HBM once and served from L2 to the group's other runs, and each XCD
// generates its own eighth of the group.  Each chunk is generated exactly as
// the single-run launch generates it.
template <bool kT3, bool kBlock>
__global__ __launch_bounds__(sim_threads<kT3>()) void canary_sim_batch_kernel(
    const SimJobDev* __restrict__ jobs, const BatchGroupDev* __restrict__ groups,
    uint32_t n_groups, uint64_t total_iters) {
    for (uint64_t it = blockIdx.x; it < total_iters; it += gridDim.x) {
        uint32_t j, unit_jobs, group_jobs;
        uint64_t chunk;
        if (!batch_iter(groups, n_groups, it, &j, &unit_jobs, &chunk, &group_jobs)) continue;
        const SimJobDev& J = jobs[j];
        sim_chunk<kT3, kBlock, false>(J.A, chunk, J.ref, J.h);
    }
}

// Propagation model: a thread walks one group of 8 elements of one canary
// through all S stages in order, carrying the live error in registers; a
// workgroup chunk covers kChainChunkGroups groups of one canary, so the
// per-stage block state is workgroup-uniform.  Same bytes as the live pass
// (4 B read, 2 B written per element); nothing is re-read.  With Student-t
// noise the carried error and the extra draws need more than the 128
// registers a 1024-thread workgroup allows, so that variant runs 256-thread
// workgroups (no spills: 26.5 ms against 27.9 ms on the 16 x 256 x 256 x 8192
// shape); the Gaussian variant keeps 1024 threads (10.5 ms against 11.5 ms).
template <bool kT3>
constexpr int chain_threads() { return kT3 ? 256 : kGenThreads; }

template <bool kT3>
constexpr uint32_t chain_chunk_groups() { return chain_threads<kT3>() * kGenItems; }

template <bool kT3, bool kBlock>
__global__ __launch_bounds__(chain_threads<kT3>()) void canary_chain_kernel(SimArgs A, uint32_t S,
                                                                   float gain,
                                                                   const float* __restrict__ ref,
                                                                   uint16_t* __restrict__ h) {
    const uint64_t n = static_cast<uint64_t>(A.n8) * 8;
    for (uint64_t it = blockIdx.x; it < A.total_chunks; it += gridDim.x) {
        const uint64_t chunk = xcd_contiguous(it, A.total_chunks);
        const uint32_t c = static_cast<uint32_t>(chunk / A.chunks_per_block);
        const uint32_t g0 =
            static_cast<uint32_t>(chunk - static_cast<uint64_t>(c) * A.chunks_per_block) *
            chain_chunk_groups<kT3>();
#pragma unroll 1
        for (int item = 0; item < kGenItems; ++item) {
            const uint32_t g = g0 + item * chain_threads<kT3>() + threadIdx.x;
            if (g >= A.n8) break;
            float d[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll 1
            for (uint32_t s = 0; s < S; ++s) {
                const uint64_t block = static_cast<uint64_t>(s) * A.C + c;
                const SimBlock B = sim_block<kBlock>(A, block);
                const f32x4* in = reinterpret_cast<const f32x4*>(ref + block * n);
                u32x4* out = reinterpret_cast<u32x4*>(h + block * n);
                const f32x4 a_lo = load_stream(in + 2 * g), a_hi = load_stream(in + 2 * g + 1);
                store_stream(out + g,
                             chain_group8<kT3, kBlock>(A, B, g * 8, s == 0, gain, a_lo, a_hi, d));
            }
        }
    }
}

// Grid for a chunked elementwise walk: 64 workgroups per CU; larger jobs
// loop with a stride (16384) that is a multiple of the XCD count, as
// xcd_contiguous needs.
inline uint32_t gen_grid(uint64_t total_chunks) {
    const uint64_t cap = 256ull * 64;
    return static_cast<uint32_t>(total_chunks < cap ? total_chunks : cap);
}

}  // namespace

hipError_t launch_outlier_gain(uint32_t H, uint32_t n_out, float big, uint64_t seed,
                               uint32_t ref_set_id, float* gain, hipStream_t st) {
    if (H == 0) return hipSuccess;
    const uint32_t grid = (H + 255) / 256;
    hipLaunchKernelGGL(outlier_gain_kernel, dim3(grid), dim3(256), 0, st, H, n_out, big,
                       Key{static_cast<uint32_t>(seed), static_cast<uint32_t>(seed >> 32)},
                       stream_tag(kStreamOutlier, ref_set_id), gain);
    return hipGetLastError();
}

hipError_t launch_ref_synth(uint32_t S, uint32_t C, uint32_t T, uint32_t H, uint64_t seed,
                            uint32_t ref_set_id, uint32_t canary_base, const float* gain,
                            float* ref, hipStream_t st) {
    const uint64_t n = static_cast<uint64_t>(T) * H;
    const uint64_t nblocks = static_cast<uint64_t>(S) * C;
    if (n == 0 || nblocks == 0) return hipSuccess;
    const uint32_t n8 = static_cast<uint32_t>(n / 8);
    const uint64_t cpb = (n8 + kGenChunkGroups - 1) / kGenChunkGroups;
    const uint64_t total = cpb * nblocks;
    hipLaunchKernelGGL(ref_synth_kernel, dim3(gen_grid(total)), dim3(kGenThreads), 0, st, C,
                       canary_base, H, n8, cpb, total,
                       Key{static_cast<uint32_t>(seed), static_cast<uint32_t>(seed >> 32)},
                       stream_tag(kStreamRef, ref_set_id), gain, ref);
    return hipGetLastError();
}

hipError_t launch_block_scales(uint64_t nblocks, uint32_t T, uint32_t H, const double* sumsq,
                               const double* sumabs, double eps, double sigma_b, float* tscale,
                               float* bscale, hipStream_t st) {
    if (nblocks == 0) return hipSuccess;
    const uint64_t grid = (nblocks + 255) / 256;
    hipLaunchKernelGGL(block_scales_kernel, dim3(static_cast<uint32_t>(grid)), dim3(256), 0, st,
                       nblocks, static_cast<double>(T) * static_cast<double>(H), sumsq, sumabs,
                       eps, sigma_b, tscale, bscale);
    return hipGetLastError();
}

template <bool kT3, bool kBlock>
hipError_t launch_chain_t(const SimLaunch& p, const float* ref, uint16_t* h, hipStream_t st) {
    const uint64_t n8 = static_cast<uint64_t>(p.T) * p.H / 8;
    const uint64_t cpc = (n8 + chain_chunk_groups<kT3>() - 1) / chain_chunk_groups<kT3>();
    const SimArgs A = make_sim_args(p, cpc, cpc * p.C);  // cpc chunks per canary
    hipLaunchKernelGGL((canary_chain_kernel<kT3, kBlock>), dim3(gen_grid(A.total_chunks)),
                       dim3(chain_threads<kT3>()), 0, st, A, p.S, p.carry, ref, h);
    return hipGetLastError();
}

hipError_t launch_canary_chain(const SimLaunch& p, const float* ref, uint16_t* h,
                               hipStream_t st) {
    const bool t3 = p.benign_dist == 1, block_mode = p.benign_mode == 1;
    if (t3 && block_mode) return launch_chain_t<true, true>(p, ref, h, st);
    if (t3) return launch_chain_t<true, false>(p, ref, h, st);
    if (block_mode) return launch_chain_t<false, true>(p, ref, h, st);
    return launch_chain_t<false, false>(p, ref, h, st);
}

template <bool kT3>
hipError_t launch_sim_t(const SimLaunch& p, const float* ref, uint16_t* h, hipStream_t st) {
    const uint64_t n8 = static_cast<uint64_t>(p.T) * p.H / 8;
    const uint64_t nblocks = static_cast<uint64_t>(p.S) * p.C;
    const uint64_t cpb = (n8 + sim_chunk_groups<kT3>() - 1) / sim_chunk_groups<kT3>();
    const SimArgs A = make_sim_args(p, cpb, cpb * nblocks);
    const dim3 grid(gen_grid(A.total_chunks)), block(sim_threads<kT3>());
    if (A.block_mode)
        hipLaunchKernelGGL((canary_sim_kernel<kT3, true>), grid, block, 0, st, A, ref, h);
    else
        hipLaunchKernelGGL((canary_sim_kernel<kT3, false>), grid, block, 0, st, A, ref, h);
    return hipGetLastError();
}

hipError_t launch_canary_sim(const SimLaunch& p, const float* ref, uint16_t* h, hipStream_t st) {
    const uint64_t n = static_cast<uint64_t>(p.T) * p.H;
    const uint64_t nblocks = static_cast<uint64_t>(p.S) * p.C;
    if (n == 0 || nblocks == 0) return hipSuccess;
    if (p.carry != 0.0f) return launch_canary_chain(p, ref, h, st);
    return p.benign_dist == 1 ? launch_sim_t<true>(p, ref, h, st)
                              : launch_sim_t<false>(p, ref, h, st);
}

// Table layout: n_jobs SimJobDev, then (256-byte aligned) up to n_jobs
// BatchGroupDev.
size_t sim_batch_groups_offset(uint32_t n_jobs) {
    return (static_cast<size_t>(n_jobs) * sizeof(SimJobDev) + 255) & ~static_cast<size_t>(255);
}

size_t sim_batch_table_bytes(uint32_t n_jobs) {
    return sim_batch_groups_offset(n_jobs) + static_cast<size_t>(n_jobs) * sizeof(BatchGroupDev);
}

template <bool kT3, bool kBlock>
void launch_sim_batch_t(const SimJobDev* jobs, const BatchGroupDev* groups, uint32_t n_groups,
                        uint64_t total, hipStream_t st) {
    hipLaunchKernelGGL((canary_sim_batch_kernel<kT3, kBlock>), dim3(gen_grid(total)),
                       dim3(sim_threads<kT3>()), 0, st, jobs, groups, n_groups, total);
}

hipError_t launch_canary_sim_batch(uint32_t n_jobs, const SimLaunch* runs,
                                   const float* const* refs, uint16_t* const* hs, void* table,
                                   hipStream_t st) {
    std::vector<SimJobDev> jobs;
    std::vector<BatchKey> keys;
    jobs.reserve(n_jobs);
    bool t3 = false, block_mode = false;
    for (uint32_t j = 0; j < n_jobs; ++j) {
        const SimLaunch& p = runs[j];
        const uint64_t n8 = static_cast<uint64_t>(p.T) * p.H / 8;
        const uint64_t nblocks = static_cast<uint64_t>(p.S) * p.C;
        if (n8 == 0 || nblocks == 0) continue;
        t3 = p.benign_dist == 1;
        block_mode = p.benign_mode == 1;
        const uint64_t cpb = t3 ? (n8 + sim_chunk_groups<true>() - 1) / sim_chunk_groups<true>()
                                : (n8 + sim_chunk_groups<false>() - 1) / sim_chunk_groups<false>();
        SimJobDev d;
        d.A = make_sim_args(p, cpb, cpb * nblocks);
        d.ref = refs[j];
        d.h = hs[j];
        jobs.push_back(d);
        keys.push_back(BatchKey{refs[j], cpb * nblocks, p.S, p.C, static_cast<uint32_t>(n8)});
    }
    if (jobs.empty()) return hipSuccess;
    const uint32_t n = static_cast<uint32_t>(jobs.size());
    const size_t goff = sim_batch_groups_offset(n);
    std::vector<char> staged(goff + n * sizeof(BatchGroupDev), 0);
    BatchGroupDev* groups = reinterpret_cast<BatchGroupDev*>(staged.data() + goff);
    uint32_t n_groups = 0;
    const uint64_t total = plan_batch_groups(n, keys.data(), kSimJobsPerIter, kSimJobMajorFrom,
                                             groups, &n_groups);
    memcpy(staged.data(), jobs.data(), n * sizeof(SimJobDev));
    const size_t bytes = goff + n_groups * sizeof(BatchGroupDev);
    hipError_t e = hipMemcpyAsync(table, staged.data(), bytes, hipMemcpyHostToDevice, st);
    if (e != hipSuccess) return e;
    const SimJobDev* dev = static_cast<const SimJobDev*>(table);
    const BatchGroupDev* gdev =
        reinterpret_cast<const BatchGroupDev*>(static_cast<const char*>(table) + goff);
    if (t3 && block_mode)
        launch_sim_batch_t<true, true>(dev, gdev, n_groups, total, st);
    else if (t3)
        launch_sim_batch_t<true, false>(dev, gdev, n_groups, total, st);
    else if (block_mode)
        launch_sim_batch_t<false, true>(dev, gdev, n_groups, total, st);
    else
        launch_sim_batch_t<false, false>(dev, gdev, n_groups, total, st);
    return hipGetLastError();
}

hipError_t launch_canary_sim_stream(uint32_t S, uint32_t C, uint32_t T, uint32_t H,
                                    const float* ref, uint16_t* h, hipStream_t st) {
    const uint64_t n8 = static_cast<uint64_t>(T) * H / 8;
    const uint64_t nblocks = static_cast<uint64_t>(S) * C;
    if (n8 == 0 || nblocks == 0) return hipSuccess;
    SimLaunch p{};
    p.S = S;
    p.C = C;
    p.T = T;
    p.H = H;
    const uint64_t cpb = (n8 + sim_chunk_groups<false>() - 1) / sim_chunk_groups<false>();
    const SimArgs A = make_sim_args(p, cpb, cpb * nblocks);
    hipLaunchKernelGGL((canary_sim_kernel<false, false, true>), dim3(gen_grid(A.total_chunks)),
                       dim3(sim_threads<false>()), 0, st, A, ref, h);
    return hipGetLastError();
}

}  // namespace cdt
