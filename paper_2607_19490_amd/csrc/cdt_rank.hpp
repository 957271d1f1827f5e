// Launch interface of the per-canary ranking (Eq. 5 per canary), between
// the C ABI layer and rank.hip; arguments have been validated by the ABI.
#pragma once

#include "cdt_launch.hpp"

namespace cdt {

// Each configuration g's canaries t: six uint32 counts (detector, control,
// random baseline: wins and ties) at per_canary[(offsets_dev[g] + t) * 6].
hipError_t launch_auroc_canaries(uint32_t n_cfg, const AurocCfgDev* cfgs_dev,
                                 const uint64_t* offsets_dev, const float* scores,
                                 uint64_t n_scores, uint64_t seed, uint32_t flags,
                                 uint32_t* per_canary, hipStream_t st);

}  // namespace cdt
