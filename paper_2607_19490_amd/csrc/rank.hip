// Detection AUROC (Eqs. 5-6), its Mann-Whitney form and the scrambled-label
// control of Section 4.5, batched over configurations.
//
// Per-canary counts: one workgroup per configuration; each wave takes one
// canary at a time with lane s holding shard s's score as an order key
// (S <= 64 = one wave), and loads its next canary's scores before ranking
// the current one.  Every positive lane compares itself with every negative
// shard through wave shuffles; integer counts are summed over waves in a
// fixed order.
//
// Pooled Mann-Whitney: one 1024-thread workgroup per configuration sorts the
// C*S (key, label) pairs with a bitonic network, scans the negatives in
// sorted order, and for each positive binary-searches its tie group: it beats
// the negatives before the group and ties those inside it.  Each thread holds
// E = max(1, P2 / 1024) consecutive elements of the padded length P2 in
// registers: compare-exchange stages between elements of one thread run in
// registers, stages between threads of one wave through lane shuffles, and
// only the stages that span waves go through LDS, with one barrier each.
#include "cdt_device.hpp"
#include "cdt_launch.hpp"
#include "cdt_rank.hpp"

namespace cdt {
namespace {

// 16 waves per configuration: on 256 canaries (one 70B-shaped run) each wave
// walks 16 of them instead of 64 at 256 threads.
constexpr int kCountThreads = 1024;
constexpr int kCountWaves = kCountThreads / kWave;
constexpr int kPoolThreads = 1024;
constexpr uint32_t kPoolMax = 16384;

__device__ __forceinline__ uint64_t shard_mask(uint32_t S) {
    return S >= 64 ? ~0ull : ((1ull << S) - 1ull);
}

// r-th set bit (0-based) of m; m has more than r bits set.
__device__ __forceinline__ uint32_t nth_set_bit(uint64_t m, uint32_t r) {
    for (uint32_t i = 0; i < r; ++i) m &= m - 1;
    return static_cast<uint32_t>(__builtin_ctzll(m));
}

// Random-baseline score of (canary t, shard s): 24 random bits scaled into
// [0, 1), exact in fp32.
__device__ __forceinline__ float random_score(Key key, uint32_t t, uint32_t s, uint32_t tag) {
    return static_cast<float>(draw(key, t, s, 0, tag).x >> 8) * 0x1p-24f;
}

// A configuration the kernels can score without reading outside the score
// array or the pooled sort's LDS.  The host validates every table before it
// reaches the device; this check keeps a table reused against a different
// score array from reading out of bounds.
__device__ __forceinline__ bool cfg_in_bounds(const AurocCfgDev& cfg, uint64_t n_scores) {
    const uint64_t len = static_cast<uint64_t>(cfg.S) * cfg.C;
    return cfg.S <= 64 && cfg.score_off <= n_scores && len <= n_scores - cfg.score_off;
}

constexpr unsigned long long kBadCfg = ~0ull;  // counts of a configuration out of bounds

// What one wave needs to rank a configuration's canaries (lane = shard).
struct RankCtx {
    uint64_t pos, neg;
    uint32_t n_benign, tag, tag_random;
    bool lane_in, lane_pos, control, include_true, random;
};

__device__ __forceinline__ RankCtx rank_ctx(const AurocCfgDev& cfg, uint32_t flags) {
    const uint32_t lane = threadIdx.x % kWave;
    const uint64_t all = shard_mask(cfg.S);
    RankCtx r;
    r.pos = cfg.pos_mask & all;
    r.neg = all & ~r.pos;
    r.lane_in = lane < cfg.S;
    r.lane_pos = r.lane_in && ((r.pos >> lane) & 1u);
    r.control = flags & 1u;
    r.include_true = flags & 4u;
    r.random = flags & 8u;
    r.n_benign = __builtin_popcountll(r.neg);
    r.tag = stream_tag(kStreamScramble, cfg.cfg_id);
    r.tag_random = stream_tag(kStreamRandom, cfg.cfg_id);
    return r;
}

// One canary's Eq. 5 counts as this lane sees them: a positive lane's wins
// and ties over the negative shards (q = 0, 1), the scrambled-label
// control's chosen stage against this lane's (q = 2, 3) and the random
// baseline's (q = 4, 5).  cur is this lane's score, t the canary's local
// index.  Every lane of the wave must call it.
__device__ __forceinline__ void rank_canary(const RankCtx& r, const AurocCfgDev& cfg, Key key,
                                            uint32_t t, float cur, uint32_t (&c)[6]) {
    const uint32_t lane = threadIdx.x % kWave;
    for (int q = 0; q < 6; ++q) c[q] = 0;
    const uint32_t k = r.lane_in ? order_key(cur) : 0u;
    for (uint32_t j = 0; j < cfg.S; ++j) {
        const uint32_t kj = __shfl(k, j, kWave);
        if (r.lane_pos && ((r.neg >> j) & 1u)) {
            c[0] += k > kj;
            c[1] += k == kj;
        }
    }
    if (r.random) {
        const uint32_t kr =
            r.lane_in ? order_key(random_score(key, cfg.canary_base + t, lane, r.tag_random)) : 0u;
        for (uint32_t j = 0; j < cfg.S; ++j) {
            const uint32_t kj = __shfl(kr, j, kWave);
            if (r.lane_pos && ((r.neg >> j) & 1u)) {
                c[4] += kr > kj;
                c[5] += kr == kj;
            }
        }
    }
    if (r.control && r.n_benign > 0) {
        const uint32_t u = draw(key, cfg.canary_base + t, 0, 0, r.tag).x;
        const uint32_t js = nth_set_bit(r.neg, u % r.n_benign);
        const uint32_t kjs = __shfl(k, js, kWave);
        const bool counted =
            r.lane_in && lane != js && (r.include_true || !((r.pos >> lane) & 1u));
        if (counted) {
            c[2] += kjs > k;
            c[3] += kjs == k;
        }
    }
}

// Eqs. 5-6 counts of configuration blockIdx.x (every thread of the
// workgroup calls it).
__device__ __forceinline__ void counts_body(
    const AurocCfgDev* __restrict__ cfgs, const float* __restrict__ scores, uint64_t n_scores,
    Key key, uint32_t flags, unsigned long long* __restrict__ counts,
    unsigned long long* __restrict__ baseline) {
    const AurocCfgDev cfg = cfgs[blockIdx.x];
    if (!cfg_in_bounds(cfg, n_scores)) {  // uniform over the workgroup
        if (threadIdx.x == 0) {
            for (int q = 0; q < 6; ++q) counts[6ull * blockIdx.x + q] = kBadCfg;
            if (flags & 8u)
                for (int q = 0; q < 3; ++q) baseline[3ull * blockIdx.x + q] = kBadCfg;
        }
        return;
    }
    const uint32_t lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
    const RankCtx r = rank_ctx(cfg, flags);
    const uint64_t pos = r.pos;
    const bool control = r.control, include_true = r.include_true, random = r.random;
    const uint32_t n_benign = r.n_benign;

    unsigned long long g = 0, e = 0, gc = 0, ec = 0, gr = 0, er = 0;
    const float* base = scores + cfg.score_off;
    const bool lane_in = r.lane_in;
    float next = (wave < cfg.C && lane_in) ? base[static_cast<uint64_t>(wave) * cfg.S + lane] : 0.f;
    for (uint32_t t = wave; t < cfg.C; t += kCountWaves) {
        const float cur = next;
        const uint32_t tn = t + kCountWaves;
        if (tn < cfg.C && lane_in) next = base[static_cast<uint64_t>(tn) * cfg.S + lane];
        uint32_t c[6];
        rank_canary(r, cfg, key, t, cur, c);
        g += c[0];
        e += c[1];
        gc += c[2];
        ec += c[3];
        gr += c[4];
        er += c[5];
    }

    __shared__ unsigned long long lds[6][kCountWaves];
    unsigned long long part[6] = {g, e, gc, ec, gr, er};
#pragma unroll
    for (int q = 0; q < 6; ++q) part[q] = wave_sum(part[q]);
    if (lane == 0) {
#pragma unroll
        for (int q = 0; q < 6; ++q) lds[q][wave] = part[q];
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        unsigned long long tot[6] = {0, 0, 0, 0, 0, 0};
        for (int q = 0; q < 6; ++q)
            for (int w = 0; w < kCountWaves; ++w) tot[q] += lds[q][w];
        const unsigned long long n_pos = __builtin_popcountll(pos);
        unsigned long long* out = counts + 6ull * blockIdx.x;
        out[0] = tot[0];
        out[1] = tot[1];
        out[2] = static_cast<unsigned long long>(cfg.C) * n_pos * n_benign;
        unsigned long long n_ctrl = 0;
        if (control && n_benign > 0) n_ctrl = include_true ? cfg.S - 1 : n_benign - 1;
        out[3] = control ? tot[2] : 0;
        out[4] = control ? tot[3] : 0;
        out[5] = static_cast<unsigned long long>(cfg.C) * n_ctrl;
        if (random) {
            unsigned long long* rb = baseline + 3ull * blockIdx.x;
            rb[0] = tot[4];
            rb[1] = tot[5];
            rb[2] = out[2];
        }
    }
}

// Eq. 5 per canary: the same ranking as auroc_counts_kernel, each canary's
// six counts summed over its wave and written by lane 0 to
// out[(offset[g] + t) * 6 + q].  A configuration out of bounds gets
// 0xFFFFFFFF in its entries instead of being read.
__global__ __launch_bounds__(kCountThreads) void auroc_canaries_kernel(
    const AurocCfgDev* __restrict__ cfgs, const uint64_t* __restrict__ offsets,
    const float* __restrict__ scores, uint64_t n_scores, Key key, uint32_t flags,
    uint32_t* __restrict__ out) {
    const AurocCfgDev cfg = cfgs[blockIdx.x];
    uint32_t* o = out + 6ull * offsets[blockIdx.x];
    const uint32_t lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
    if (!cfg_in_bounds(cfg, n_scores)) {  // uniform over the workgroup
        for (uint64_t i = threadIdx.x; i < 6ull * cfg.C; i += kCountThreads) o[i] = ~0u;
        return;
    }
    const RankCtx r = rank_ctx(cfg, flags);
    const float* base = scores + cfg.score_off;
    float next =
        (wave < cfg.C && r.lane_in) ? base[static_cast<uint64_t>(wave) * cfg.S + lane] : 0.f;
    for (uint32_t t = wave; t < cfg.C; t += kCountWaves) {
        const float cur = next;
        const uint32_t tn = t + kCountWaves;
        if (tn < cfg.C && r.lane_in) next = base[static_cast<uint64_t>(tn) * cfg.S + lane];
        uint32_t c[6];
        rank_canary(r, cfg, key, t, cur, c);
        unsigned long long w[6];
#pragma unroll
        for (int q = 0; q < 6; ++q) w[q] = wave_sum(static_cast<unsigned long long>(c[q]));
        if (lane == 0) {
#pragma unroll
            for (int q = 0; q < 6; ++q) o[6ull * t + q] = static_cast<uint32_t>(w[q]);
        }
    }
}

__device__ __forceinline__ uint64_t shfl_xor_u64(uint64_t x, int m) {
    const int lo = __shfl_xor(static_cast<int>(static_cast<uint32_t>(x)), m, kWave);
    const int hi = __shfl_xor(static_cast<int>(static_cast<uint32_t>(x >> 32)), m, kWave);
    return (static_cast<uint64_t>(static_cast<uint32_t>(hi)) << 32) | static_cast<uint32_t>(lo);
}

// Ascending bitonic sort of P2 (a power of two, <= kE * kPoolThreads)
// elements, thread t holding elements t*kE .. t*kE + kE - 1 in x; v is LDS
// scratch of P2 elements.  Every thread of the workgroup must call it.
template <int kE>
__device__ __forceinline__ void bitonic_sort_regs(uint64_t (&x)[kE], uint32_t P2, uint64_t* v) {
    const uint32_t t = threadIdx.x, base = t * kE;
    for (uint32_t k = 2; k <= P2; k <<= 1) {
        uint32_t j = k >> 1;
        if (j >= kWave * kE) {  // partners in other waves: in place in LDS
#pragma unroll
            for (int r = 0; r < kE; ++r)
                if (base + r < P2) v[base + r] = x[r];
            __syncthreads();
            for (; j >= kWave * kE; j >>= 1) {
                for (uint32_t p = t; p < P2 / 2; p += kPoolThreads) {
                    const uint32_t i = 2 * p - (p & (j - 1));
                    const uint32_t l = i + j;
                    const uint64_t a = v[i], b = v[l];
                    if ((a > b) == ((i & k) == 0)) {
                        v[i] = b;
                        v[l] = a;
                    }
                }
                __syncthreads();
            }
#pragma unroll
            for (int r = 0; r < kE; ++r)
                if (base + r < P2) x[r] = v[base + r];
        }
        for (; j >= static_cast<uint32_t>(kE); j >>= 1) {  // partner lane t ^ (j / kE)
            const int m = static_cast<int>(j / kE);
            const bool keep_min = ((t & m) == 0) == ((base & k) == 0);
#pragma unroll
            for (int r = 0; r < kE; ++r) {
                const uint64_t y = shfl_xor_u64(x[r], m);
                x[r] = keep_min ? (x[r] < y ? x[r] : y) : (x[r] < y ? y : x[r]);
            }
        }
#pragma unroll
        for (int jj = kE / 2; jj >= 1; jj >>= 1) {  // partner in this thread
            if (static_cast<uint32_t>(jj) < k) {
#pragma unroll
                for (int r = 0; r < kE; ++r) {
                    const int rp = r ^ jj;
                    if (rp > r) {
                        const uint64_t a = x[r], b = x[rp];
                        if ((a > b) == (((base + r) & k) == 0)) {
                            x[r] = b;
                            x[rp] = a;
                        }
                    }
                }
            }
        }
    }
}

// Loads the configuration's n (key, label) pairs padded to P2, sorts them,
// and leaves the sorted array in v[0 .. P2).
template <int kE>
__device__ void pooled_sort(const float* tab, uint32_t n, uint32_t P2, uint32_t S, uint64_t pos,
                            uint64_t* v) {
    uint64_t x[kE];
    const uint32_t base = threadIdx.x * kE;
#pragma unroll
    for (int r = 0; r < kE; ++r) {
        const uint32_t i = base + r;
        x[r] = i < n ? (static_cast<uint64_t>(order_key(tab[i])) << 32) | ((pos >> (i % S)) & 1u)
                     : ~0ull;  // padding sorts last
    }
    bitonic_sort_regs<kE>(x, P2, v);
#pragma unroll
    for (int r = 0; r < kE; ++r)
        if (base + r < P2) v[base + r] = x[r];
    __syncthreads();
}

// Element layout in the pooled sort: key << 32 | label (label 1 = positive);
// after the negative scan: key << 32 | negatives_before << 1 | label.
// Pooled Mann-Whitney counts of configuration blockIdx.x (every thread of
// the workgroup calls it).
__device__ __forceinline__ void pooled_body(
    const AurocCfgDev* __restrict__ cfgs, const float* __restrict__ scores, uint64_t n_scores,
    unsigned long long* __restrict__ pooled) {
    __shared__ uint64_t v[kPoolMax];
    __shared__ uint32_t scan[kPoolThreads];
    __shared__ unsigned long long red[2][kPoolThreads / kWave];
    const AurocCfgDev cfg = cfgs[blockIdx.x];
    if (!cfg_in_bounds(cfg, n_scores) ||
        static_cast<uint64_t>(cfg.S) * cfg.C > kPoolMax) {  // uniform over the workgroup
        if (threadIdx.x == 0)
            for (int q = 0; q < 3; ++q) pooled[3ull * blockIdx.x + q] = kBadCfg;
        return;
    }
    const uint32_t n = cfg.S * cfg.C;
    uint32_t P2 = 1;
    while (P2 < n) P2 <<= 1;
    const uint64_t pos = cfg.pos_mask & shard_mask(cfg.S);
    const float* tab = scores + cfg.score_off;

    static_assert(kPoolMax == 16 * kPoolThreads, "at most 16 elements per thread");
    switch (P2 <= kPoolThreads ? 1u : P2 / kPoolThreads) {  // uniform over the workgroup
        case 1: pooled_sort<1>(tab, n, P2, cfg.S, pos, v); break;
        case 2: pooled_sort<2>(tab, n, P2, cfg.S, pos, v); break;
        case 4: pooled_sort<4>(tab, n, P2, cfg.S, pos, v); break;
        case 8: pooled_sort<8>(tab, n, P2, cfg.S, pos, v); break;
        default: pooled_sort<16>(tab, n, P2, cfg.S, pos, v); break;
    }

    // Exclusive scan of negatives over the sorted order: each thread owns a
    // contiguous run of `per` elements.
    const uint32_t per = (n + kPoolThreads - 1) / kPoolThreads;
    const uint32_t lo = threadIdx.x * per;
    const uint32_t hi = min(lo + per, n);
    uint32_t cnt = 0;
    for (uint32_t i = lo; i < hi; ++i) cnt += !(v[i] & 1u);
    scan[threadIdx.x] = cnt;
    __syncthreads();
    for (uint32_t off = 1; off < kPoolThreads; off <<= 1) {
        const uint32_t add = threadIdx.x >= off ? scan[threadIdx.x - off] : 0u;
        __syncthreads();
        scan[threadIdx.x] += add;
        __syncthreads();
    }
    const uint32_t n_neg = scan[kPoolThreads - 1];
    uint32_t before = scan[threadIdx.x] - cnt;
    for (uint32_t i = lo; i < hi; ++i) {
        const uint64_t x = v[i];
        v[i] = (x & ~0xFFFFFFFFull) | (static_cast<uint64_t>(before) << 1) | (x & 1u);
        before += !(x & 1u);
    }
    __syncthreads();

    // Positives: negatives strictly below the key, and inside its tie group.
    unsigned long long gp = 0, ep = 0;
    for (uint32_t i = threadIdx.x; i < n; i += kPoolThreads) {
        const uint64_t x = v[i];
        if (!(x & 1u)) continue;
        const uint32_t key = static_cast<uint32_t>(x >> 32);
        uint32_t a = 0, b = n;  // first index with key >= this key
        while (a < b) {
            const uint32_t m = (a + b) >> 1;
            if (static_cast<uint32_t>(v[m] >> 32) < key) a = m + 1; else b = m;
        }
        const uint32_t first = a;
        a = first;
        b = n;  // first index with key > this key
        while (a < b) {
            const uint32_t m = (a + b) >> 1;
            if (static_cast<uint32_t>(v[m] >> 32) <= key) a = m + 1; else b = m;
        }
        const uint32_t last = a;
        const uint32_t neg_lt = first < n ? static_cast<uint32_t>((v[first] >> 1) & 0x7FFFFFFFu) : n_neg;
        const uint32_t neg_le = last < n ? static_cast<uint32_t>((v[last] >> 1) & 0x7FFFFFFFu) : n_neg;
        gp += neg_lt;
        ep += neg_le - neg_lt;
    }
    gp = wave_sum(gp);
    ep = wave_sum(ep);
    const uint32_t lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
    if (lane == 0) {
        red[0][wave] = gp;
        red[1][wave] = ep;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        unsigned long long G = 0, E = 0;
        for (int w = 0; w < kPoolThreads / kWave; ++w) {
            G += red[0][w];
            E += red[1][w];
        }
        const unsigned long long n_pos = static_cast<unsigned long long>(n) - n_neg;
        unsigned long long* out = pooled + 3ull * blockIdx.x;
        out[0] = G;
        out[1] = E;
        out[2] = n_pos * n_neg;
    }
}


__global__ __launch_bounds__(kCountThreads) void auroc_counts_kernel(
    const AurocCfgDev* __restrict__ cfgs, const float* __restrict__ scores, uint64_t n_scores,
    Key key, uint32_t flags, unsigned long long* __restrict__ counts,
    unsigned long long* __restrict__ baseline) {
    counts_body(cfgs, scores, n_scores, key, flags, counts, baseline);
}

// The counts and the pooled ranking of a configuration in one workgroup:
// one launch instead of two when the pooled form is asked for (the two
// parts share nothing but the configuration; the counts use a few hundred
// bytes of LDS, the sort up to 128 KiB).
static_assert(kCountThreads == kPoolThreads, "one workgroup shape for both parts");
__global__ __launch_bounds__(kCountThreads) void auroc_counts_pooled_kernel(
    const AurocCfgDev* __restrict__ cfgs, const float* __restrict__ scores, uint64_t n_scores,
    Key key, uint32_t flags, unsigned long long* __restrict__ counts,
    unsigned long long* __restrict__ baseline, unsigned long long* __restrict__ pooled) {
    counts_body(cfgs, scores, n_scores, key, flags, counts, baseline);
    pooled_body(cfgs, scores, n_scores, pooled);
}
// Eq. 6 from integer counts: G / pairs (ties count 0, the equation as
// printed) and (G + E / 2) / pairs (ties count one half, the Mann-Whitney
// form), in fp64.  A triple with no pairs, or one holding the out-of-bounds
// marker, gives NaN.
__device__ __forceinline__ void ratios(const unsigned long long* c, double* out) {
    const unsigned long long G = c[0], E = c[1], N = c[2];
    if (N == 0 || G == kBadCfg || E == kBadCfg || N == kBadCfg) {
        out[0] = out[1] = __builtin_nan("");
        return;
    }
    const double n = static_cast<double>(N);
    out[0] = static_cast<double>(G) / n;
    out[1] = (static_cast<double>(G) + 0.5 * static_cast<double>(E)) / n;
}

__global__ void auroc_values_kernel(uint32_t n_cfg, const unsigned long long* __restrict__ counts,
                                    const unsigned long long* __restrict__ pooled,
                                    const unsigned long long* __restrict__ baseline,
                                    double* __restrict__ values) {
    const uint32_t g = blockIdx.x * blockDim.x + threadIdx.x;
    if (g >= n_cfg) return;
    double* v = values + 8ull * g;
    ratios(counts + 6ull * g, v);
    ratios(counts + 6ull * g + 3, v + 2);
    if (pooled) {
        ratios(pooled + 3ull * g, v + 4);
    } else {
        v[4] = v[5] = __builtin_nan("");
    }
    if (baseline) {
        ratios(baseline + 3ull * g, v + 6);
    } else {
        v[6] = v[7] = __builtin_nan("");
    }
}

}  // namespace

hipError_t launch_auroc_values(uint32_t n_cfg, const uint64_t* counts, const uint64_t* pooled,
                               const uint64_t* baseline, double* values, hipStream_t st) {
    if (n_cfg == 0) return hipSuccess;
    hipLaunchKernelGGL(auroc_values_kernel, dim3((n_cfg + 255) / 256), dim3(256), 0, st, n_cfg,
                       reinterpret_cast<const unsigned long long*>(counts),
                       reinterpret_cast<const unsigned long long*>(pooled),
                       reinterpret_cast<const unsigned long long*>(baseline), values);
    return hipGetLastError();
}

hipError_t launch_auroc_canaries(uint32_t n_cfg, const AurocCfgDev* cfgs_dev,
                                 const uint64_t* offsets_dev, const float* scores,
                                 uint64_t n_scores, uint64_t seed, uint32_t flags,
                                 uint32_t* per_canary, hipStream_t st) {
    if (n_cfg == 0) return hipSuccess;
    const Key key{static_cast<uint32_t>(seed), static_cast<uint32_t>(seed >> 32)};
    hipLaunchKernelGGL(auroc_canaries_kernel, dim3(n_cfg), dim3(kCountThreads), 0, st, cfgs_dev,
                       offsets_dev, scores, n_scores, key, flags, per_canary);
    return hipGetLastError();
}

hipError_t launch_auroc(uint32_t n_cfg, const AurocCfgDev* cfgs_dev, const float* scores,
                        uint64_t n_scores, uint64_t seed, uint32_t flags, uint64_t* counts,
                        uint64_t* pooled, uint64_t* baseline, hipStream_t st) {
    if (n_cfg == 0) return hipSuccess;
    const Key key{static_cast<uint32_t>(seed), static_cast<uint32_t>(seed >> 32)};
    if (flags & 2u) {
        hipLaunchKernelGGL(auroc_counts_pooled_kernel, dim3(n_cfg), dim3(kCountThreads), 0, st,
                           cfgs_dev, scores, n_scores, key, flags,
                           reinterpret_cast<unsigned long long*>(counts),
                           reinterpret_cast<unsigned long long*>(baseline),
                           reinterpret_cast<unsigned long long*>(pooled));
    } else {
        hipLaunchKernelGGL(auroc_counts_kernel, dim3(n_cfg), dim3(kCountThreads), 0, st,
                           cfgs_dev, scores, n_scores, key, flags,
                           reinterpret_cast<unsigned long long*>(counts),
                           reinterpret_cast<unsigned long long*>(baseline));
    }
    return hipGetLastError();
}

}  // namespace cdt
