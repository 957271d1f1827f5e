// Internal launch interface between the C ABI layer and the kernel files.
// Arguments reaching these functions have been validated by the ABI layer.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

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

// Batched live pass over runs of one noise distribution and mode, carry 0:
// the device table (sim_batch_table_bytes(n_jobs) bytes) is filled from
// `runs` on the stream, then one grid generates every run's chunks.
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
// device table: its arrays, shape, chunking and place in the batch's chunk
// and block index ranges.
struct DriftJobDev {
    const uint16_t* h;
    const float* ref;
    float* score;
    double* sums;     // [C][S][2] or null
    double* partial;  // its per-chunk partial sums (unused when direct)
    uint64_t cpb;     // chunks per block
    uint64_t chunk_begin, block_begin;
    uint32_t n8, S, C, direct;
};

hipError_t launch_drift_batch(const DriftJobDev* jobs_dev, uint32_t n_jobs, uint64_t total_chunks,
                              uint64_t total_blocks, hipStream_t st);

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
