// Internal launch interface between the C ABI layer and the kernel files.
// Arguments reaching these functions have been validated by the ABI layer.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "cdt_device.hpp"
#include "cdt_reduce.hpp"

namespace cdt {

// Elementwise kernels: a thread owns groups of 8 consecutive elements (one
// 16-byte fp16 vector, two 16-byte fp32 vectors); a 1024-thread workgroup
// covers kGenItems groups per thread of one block per chunk.  On the
// 16 x 256 x 256 x 8192 live pass, with the XCD-contiguous chunk order,
// 1024 x 8 runs 9.8 ms against 10.1 ms for 1024 x 2, 9.9 ms for 1024 x 16,
// 10.1 ms for 1024 x 32 and 10.2-10.3 ms for 256 x 2..8 (the next group's
// reference is always loaded before the current one is generated, so only
// the first load of a chunk is exposed).
constexpr int kGenThreads = 1024;
// Batch groups (BatchGroupDev): jobs per iteration, and the unit count
// from which a group is walked job-major, for the live pass and Eq. 4.
constexpr uint32_t kSimJobsPerIter = 1;
constexpr uint32_t kSimJobMajorFrom = 8;
constexpr uint32_t kDriftJobsPerIter = 8;
constexpr uint32_t kDriftJobMajorFrom = 0xFFFFFFFFu;
constexpr int kGenItems = 8;
constexpr uint32_t kGenChunkGroups = kGenThreads * kGenItems;

struct SimLaunch {
    uint32_t S, C, T, H;
    uint64_t seed;
    uint32_t cfg_id;
    uint32_t benign_mode, benign_dist, tamper, tamper_base, redraw;
    uint64_t mal_mask;
    float sigma_b;       // fp32(sigma_b)
    uint32_t flip_thr;   // floor(p 2^32) (p < 1)
    uint32_t flip_all;   // p >= 1
    float scale;         // fp32(scale)
    float carry;         // fp32(carry): propagation gain (0: independent stages)
    uint32_t canary_base;  // global index of canary 0 (RNG counters)
    const float* bscale;
    const float* tscale;
};

struct AurocCfgDev {
    uint32_t S, C;
    uint64_t score_off;
    uint64_t pos_mask;
    uint32_t cfg_id;
    uint32_t canary_base;
};
static_assert(sizeof(AurocCfgDev) == 32, "cfg layout must match cdt_auroc_cfg");

hipError_t launch_outlier_gain(uint32_t H, uint32_t n_out, float big, uint64_t seed,
                               uint32_t ref_set_id, float* gain, hipStream_t st);
hipError_t launch_ref_synth(uint32_t S, uint32_t C, uint32_t T, uint32_t H, uint64_t seed,
                            uint32_t ref_set_id, uint32_t canary_base, const float* gain,
                            float* ref, hipStream_t st);
hipError_t launch_block_scales(uint64_t nblocks, uint32_t T, uint32_t H, const double* sumsq,
                               const double* sumabs, double eps, double sigma_b, float* tscale,
                               float* bscale, hipStream_t st);
hipError_t launch_canary_sim(const SimLaunch& p, const float* ref, uint16_t* h, hipStream_t st);

// A run of consecutive jobs of a batched launch that read one reference
// array in one layout, and the order its iterations take.  An iteration is one chunk of
// up to `jobs_per_iter` of the group's jobs (a unit); each XCD takes one
// contiguous eighth of the group's iterations, and
//   * chunk-major: on each chunk, the group's units one after another, so
//     neighbouring workgroups of one XCD read the same reference chunk at
//     nearly the same time and all but the first read of it are served by
//     the XCD's L2;
//   * job-major: each unit from its first chunk on, so with at least 8
//     units the 8 XCDs generate 8 different jobs over the same reference
//     offsets at the same time and the last-level cache serves most of the
//     re-reads.
// Eq. 4 scores up to 8 jobs per iteration, chunk-major, reading each
// reference chunk once for them (the sweep's 24-run groups: 13.3-13.8 ms of
// Eq. 4 per sweep in units of up to 8, 13.8-14.3 ms in units of up to 4,
// whose later units re-read each chunk, some of it from HBM).  The live pass generates one job per
// iteration (its work is the random numbers, not the reads), job-major from
// 8 jobs on: for the sweep's 24-run groups that beats chunk-major (33.5 ms
// against 39.4-45.8 ms over the sweep), whose reuse in L2 does not make up
// for the traffic it adds there; with fewer jobs chunk-major wins (3 runs of
// the 16 x 256 x 256 x 8192 shape: 25.9 ms against 29 ms).
struct BatchGroupDev {
    uint64_t iter_begin;  // first iteration of the group (a multiple of 8)
    uint64_t chunks;      // chunks of one of its jobs
    uint32_t first_job, n_jobs;
    uint32_t chunk_major, jobs_per_iter;
};

// Iteration `it` of a grouped batch -> (first job of its unit, jobs in the
// unit, chunk, jobs in the group); false for the padding that rounds each
// group up to a multiple of 8 iterations.  The group is found by a binary
// search (workgroup-uniform).  Iteration it runs on XCD it % 8 (a grid
// stride that is a multiple of 8), and so does the group-local index, since
// every group starts on a multiple of 8.
__device__ __forceinline__ bool batch_iter(const BatchGroupDev* __restrict__ groups,
                                           uint32_t n_groups, uint64_t it, uint32_t* job,
                                           uint32_t* unit_jobs, uint64_t* chunk,
                                           uint32_t* group_jobs) {
    uint32_t lo = 0, hi = n_groups;  // last group whose first iteration <= it
    while (hi - lo > 1) {
        const uint32_t mid = (lo + hi) / 2;
        if (groups[mid].iter_begin <= it) lo = mid; else hi = mid;
    }
    const BatchGroupDev& G = groups[lo];
    const uint64_t units = (G.n_jobs + G.jobs_per_iter - 1) / G.jobs_per_iter;
    const uint64_t local = it - G.iter_begin, span = G.chunks * units;
    if (local >= span) return false;
    const uint64_t x = xcd_contiguous(local, span);
    uint64_t u;
    if (G.chunk_major) {
        *chunk = x / units;
        u = x - *chunk * units;
    } else {
        u = x / G.chunks;
        *chunk = x - u * G.chunks;
    }
    const uint32_t first = static_cast<uint32_t>(u) * G.jobs_per_iter;
    *job = G.first_job + first;
    *unit_jobs = G.n_jobs - first < G.jobs_per_iter ? G.n_jobs - first : G.jobs_per_iter;
    *group_jobs = G.n_jobs;
    return true;
}

// What decides whether two jobs of a batch can share their reference reads:
// the same reference array in the same layout (blocks, elements per block,
// chunks), so that a chunk index means the same elements for both.
struct BatchKey {
    const void* ref;
    uint64_t chunks;
    uint32_t S, C, n8;
    bool operator==(const BatchKey& o) const {
        return ref == o.ref && chunks == o.chunks && S == o.S && C == o.C && n8 == o.n8;
    }
};

// Host side: the groups of a batch whose job j (jobs without chunks left
// out by the caller) has key keys[j]; consecutive jobs with equal keys form
// a group (the kernels may then read one job's reference layout for all of
// them).  A group is walked chunk-major when it has fewer than
// `job_major_from` units.  Fills groups[0 .. *n_groups) and returns the
// padded iteration count.
inline uint64_t plan_batch_groups(uint32_t n_jobs, const BatchKey* keys, uint32_t jobs_per_iter,
                                  uint32_t job_major_from, BatchGroupDev* groups,
                                  uint32_t* n_groups) {
    *n_groups = 0;
    for (uint32_t j = 0; j < n_jobs; ++j) {
        if (*n_groups) {
            BatchGroupDev& last = groups[*n_groups - 1];
            if (keys[last.first_job] == keys[j]) {
                ++last.n_jobs;
                continue;
            }
        }
        BatchGroupDev g;
        g.iter_begin = 0;
        g.chunks = keys[j].chunks;
        g.first_job = j;
        g.n_jobs = 1;
        g.chunk_major = 1;
        g.jobs_per_iter = jobs_per_iter;
        groups[(*n_groups)++] = g;
    }
    uint64_t total = 0;
    for (uint32_t k = 0; k < *n_groups; ++k) {
        BatchGroupDev& g = groups[k];
        const uint64_t units = (g.n_jobs + jobs_per_iter - 1) / jobs_per_iter;
        g.chunk_major = units < job_major_from;
        g.iter_begin = total;
        total += (g.chunks * units + 7) / 8 * 8;
    }
    return total;
}

// Batched live pass over runs of one noise distribution and mode, carry 0:
// the device table (sim_batch_table_bytes(n_jobs) bytes: jobs, then groups)
// is filled from `runs` on the stream, then one grid generates every run's
// chunks.
size_t sim_batch_table_bytes(uint32_t n_jobs);
hipError_t launch_canary_sim_batch(uint32_t n_jobs, const SimLaunch* runs,
                                   const float* const* refs, uint16_t* const* hs, void* table,
                                   hipStream_t st);

// The live pass's loads and stores with h = fp16(a): its memory bound.
hipError_t launch_canary_sim_stream(uint32_t S, uint32_t C, uint32_t T, uint32_t H,
                                    const float* ref, uint16_t* h, hipStream_t st);

hipError_t launch_ref_stats(uint32_t S, uint32_t C, uint32_t T, uint32_t H, const float* ref,
                            double* sumsq, double* sumabs, void* ws, hipStream_t st);
// Eq. 4 (or its cosine variant) per block: partial sums per chunk into ws,
// then the combine.
hipError_t launch_drift(DriftMetric metric, uint32_t S, uint32_t C, uint32_t T, uint32_t H,
                        const uint16_t* h, const void* ref, float* score, double* sums, void* ws,
                        hipStream_t st);

// One array of a batched Eq. 4 launch, as the kernels read it from the
// device table: its arrays, shape, chunking and place in the batch's block
// index range.
struct DriftJobDev {
    const uint16_t* h;
    const float* ref;
    float* score;
    double* sums;     // [C][S][2] or null
    double* partial;  // its per-chunk partial sums (unused when direct)
    uint64_t cpb;     // chunks per block
    uint64_t block_begin;
    uint32_t n8, S, C, direct;
};

hipError_t launch_drift_batch(const DriftJobDev* jobs_dev, uint32_t n_jobs,
                              const BatchGroupDev* groups_dev, uint32_t n_groups,
                              uint64_t total_iters, uint64_t total_blocks, hipStream_t st);

// The batched Eq. 4's reads (same iterations, chunks, loads, lane exchange
// and order) with no arithmetic; nothing is written in practice.
hipError_t launch_drift_batch_read_stream(const DriftJobDev* jobs_dev,
                                          const BatchGroupDev* groups_dev, uint32_t n_groups,
                                          uint64_t total_iters, hipStream_t st);

// drift_score's reads (same chunks, loads and order) with no arithmetic; ws
// is drift_score's workspace and may be overwritten.
hipError_t launch_drift_read_stream(uint32_t S, uint32_t C, uint32_t T, uint32_t H,
                                   const uint16_t* h, const float* ref, void* ws, hipStream_t st);

// The combine step alone, over partial sums laid out as drift_score's.
hipError_t launch_drift_combine(DriftMetric metric, const double* partial, uint64_t cpb,
                                uint64_t nblocks, uint32_t S, uint32_t C, float* score,
                                double* sums, hipStream_t st);

// Live pass and Eq. 4 in one kernel (h may be NULL: not stored).
hipError_t launch_sim_score(const SimLaunch& p, const float* ref, uint16_t* h, float* score,
                            double* num_den, void* ws, hipStream_t st);

// Per-block scale of the exact-norm Gaussian tamper (and its two norms).
hipError_t launch_tamper_scale_exact(const SimLaunch& p, const float* ref, double eps,
                                     float* tscale, double* norms, void* ws, hipStream_t st);

// The same under the propagation model (p.carry > 0): the malicious stages'
// scales in pipeline order, benign entries cleared to 0.
hipError_t launch_tamper_scale_exact_chain(const SimLaunch& p, const float* ref, double eps,
                                           float* tscale, double* norms, void* ws,
                                           hipStream_t st);

// Eqs. 5-6 over a device table of configurations; a configuration whose
// table lies outside [0, n_scores) (or, pooled, exceeds the LDS sort) gets
// counts of all ones instead of being read.
hipError_t launch_auroc(uint32_t n_cfg, const AurocCfgDev* cfgs_dev, const float* scores,
                        uint64_t n_scores, uint64_t seed, uint32_t flags, uint64_t* counts,
                        uint64_t* pooled, uint64_t* baseline, hipStream_t st);

// Eq. 6 (strict and Mann-Whitney) from the counts of launch_auroc.
hipError_t launch_auroc_values(uint32_t n_cfg, const uint64_t* counts, const uint64_t* pooled,
                               const uint64_t* baseline, double* values, hipStream_t st);

}  // namespace cdt
