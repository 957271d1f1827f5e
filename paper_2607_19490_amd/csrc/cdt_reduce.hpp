// Shared pieces of the block reductions (Eq. 4, its fused form with the
// live pass, the exact-norm tamper and the reference statistics): the
// chunking constants, the workgroup sum and the per-element accumulation
// of Eq. 4 and its cosine variant.  A block (shard, canary) of n = T*H
// elements is cut into chunks of kReduceChunkElems; one workgroup reduces
// one chunk to fp64 partial sums in a fixed order (no atomics); a combine
// kernel adds a block's partials in chunk order.
#pragma once

#include <stdint.h>

#include "cdt_device.hpp"

#pragma clang fp contract(off)

namespace cdt {

// Threads per workgroup and 8-element groups in flight per thread.  On the
// 16 x 256 x 256 x 8192 stream, with the fp32 reference read in contiguous
// runs, 256 x 8 reaches 89.4-89.6% of the HBM peak against 87.3-88.1% for
// 512 x 4, 89.1-89.3% for 256 x 4 and 89.8-90.2% for 256 x 16 and 128 x 16;
// over the 216-configuration sweep's smaller blocks 256 x 8 is the fastest
// of these, and the fused live-pass-and-score kernel, which shares this
// thread-to-group mapping, runs 3-4% faster than at 512 x 4.
constexpr int kReduceThreads = 256;
constexpr int kReduceUnroll = 8;
constexpr uint64_t kReduceChunkElems = 32768;

inline uint64_t reduce_chunks_per_block(uint64_t n) {
    return (n + kReduceChunkElems - 1) / kReduceChunkElems;
}

// Reduction variants of Eq. 4: the relative-L2 mismatch (the detector) and
// the cosine mismatch (the metric ablation), each against an fp32 reference
// or an fp16 reference (a second live pass).
enum class DriftMetric { kL2, kL2HalfRef, kCosine, kCosineHalfRef };

// Partial sums per chunk: (D, R) for the L2 metrics, (D, A, P) for cosine.
constexpr int kReduceMaxSums = 3;

namespace {

constexpr uint32_t kChunkGroups = static_cast<uint32_t>(kReduceChunkElems / 8);
constexpr int kWavesPerGroup = kReduceThreads / kWave;

// Sum kN per-thread values over the workgroup; thread 0 gets the result.
template <int kN>
__device__ __forceinline__ void block_sum(double (&v)[kN]) {
    __shared__ double lds[kN][kWavesPerGroup];
#pragma unroll
    for (int k = 0; k < kN; ++k) v[k] = wave_sum(v[k]);
    const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
    if (lane == 0) {
#pragma unroll
        for (int k = 0; k < kN; ++k) lds[k][wave] = v[k];
    }
    __syncthreads();
    if (threadIdx.x == 0) {
#pragma unroll
        for (int k = 0; k < kN; ++k) {
            double t = 0.0;
            for (int w = 0; w < kWavesPerGroup; ++w) t += lds[k][w];
            v[k] = t;
        }
    }
    __syncthreads();
}

// Per-metric element step.  h and the reference are widened exactly to
// fp64, so d = h - a is exact and the sums carry no cancellation.
template <DriftMetric kM>
struct DriftTraits {
    static constexpr bool kHalfRef =
        kM == DriftMetric::kL2HalfRef || kM == DriftMetric::kCosineHalfRef;
    static constexpr bool kCos = kM == DriftMetric::kCosine || kM == DriftMetric::kCosineHalfRef;
    static constexpr int kSums = kCos ? 3 : 2;

    __device__ static __forceinline__ void add(double hv, double av, double (&acc)[kSums]) {
        const double d = hv - av;
        acc[0] = fma(d, d, acc[0]);      // D = sum d^2
        acc[1] = fma(av, av, acc[1]);    // R = A = sum a^2
        if constexpr (kSums == 3) acc[2] = fma(av, d, acc[2]);  // P = sum a d
    }
};

template <DriftMetric kM>
__device__ __forceinline__ void accumulate8(const u32x4& hv, const u32x4& r_half,
                                            const f32x4& a0, const f32x4& a1,
                                            double (&acc)[DriftTraits<kM>::kSums]) {
    const uint32_t hw[4] = {hv.x, hv.y, hv.z, hv.w};
    const uint32_t rw[4] = {r_half.x, r_half.y, r_half.z, r_half.w};
    const float av[8] = {a0.x, a0.y, a0.z, a0.w, a1.x, a1.y, a1.z, a1.w};
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const double h_lo = static_cast<double>(half_bits_to_float(hw[k] & 0xFFFFu));
        const double h_hi = static_cast<double>(half_bits_to_float(hw[k] >> 16));
        double a_lo, a_hi;
        if constexpr (DriftTraits<kM>::kHalfRef) {
            a_lo = static_cast<double>(half_bits_to_float(rw[k] & 0xFFFFu));
            a_hi = static_cast<double>(half_bits_to_float(rw[k] >> 16));
        } else {
            a_lo = static_cast<double>(av[2 * k]);
            a_hi = static_cast<double>(av[2 * k + 1]);
        }
        DriftTraits<kM>::add(h_lo, a_lo, acc);
        DriftTraits<kM>::add(h_hi, a_hi, acc);
    }
}

// One workgroup per chunk up to 2^20 chunks, then a grid-stride walk whose
// stride (2^20) is a multiple of the XCD count, as xcd_contiguous needs.
inline uint32_t reduce_grid(uint64_t total_chunks) {
    const uint64_t cap = 1ull << 20;
    return static_cast<uint32_t>(total_chunks < cap ? total_chunks : cap);
}

}  // namespace

}  // namespace cdt
