// The simulated live pass of Eqs. 2-3 for one group of 8 consecutive
// elements, shared by the canary_sim kernel and the fused sim-and-score
// kernel.  Every fp32 step is one rounded operation in the written order
// (FMA contraction is off in every file that includes this header).
#pragma once

#include <math.h>

#include "cdt_device.hpp"
#include "cdt_launch.hpp"

#pragma clang fp contract(off)

namespace cdt {

// Eight unit normals of one stream for elements e0..e0+7 (e0 % 8 == 0):
// Philox calls q = e0/2 .. e0/2+3, words (x, y) -> even element, (z, w) -> odd.
__device__ __forceinline__ void normals8(Key key, uint32_t e0, uint32_t c, uint32_t s,
                                         uint32_t tag, float z[8]) {
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const Words4 w = draw(key, (e0 >> 1) + k, c, s, tag);
        z[2 * k] = irwin_hall4(w.x, w.y);
        z[2 * k + 1] = irwin_hall4(w.z, w.w);
    }
}

// Launch-uniform parameters of the live pass.
struct SimArgs {
    uint32_t C, n8;
    uint32_t canary_base;  // global index of canary 0 (RNG counters)
    uint64_t chunks_per_block, total_chunks;
    Key key;
    uint32_t tag_benign, tag_t12, tag_t3, tag_add, tag_flip;
    uint32_t block_mode, t3, tamper, clean;
    uint64_t mal_mask;
    float sigma_b;
    uint32_t flip_thr, flip_all;
    float scale;
    const float* bscale;
    const float* tscale;
};

inline SimArgs make_sim_args(const SimLaunch& p, uint64_t chunks_per_block,
                             uint64_t total_chunks) {
    SimArgs A;
    A.C = p.C;
    A.canary_base = p.canary_base;
    A.n8 = static_cast<uint32_t>(static_cast<uint64_t>(p.T) * p.H / 8);
    A.chunks_per_block = chunks_per_block;
    A.total_chunks = total_chunks;
    A.key = Key{static_cast<uint32_t>(p.seed), static_cast<uint32_t>(p.seed >> 32)};
    // An independent benign recompute draws its noise from the ALT streams.
    A.tag_benign = stream_tag(p.redraw ? kStreamAlt : kStreamBenign, p.cfg_id);
    A.tag_t12 = stream_tag(p.redraw ? kStreamAltT12 : kStreamT12, p.cfg_id);
    A.tag_t3 = stream_tag(p.redraw ? kStreamAltT3 : kStreamT3, p.cfg_id);
    A.tag_add = stream_tag(kStreamTamperAdd, p.cfg_id);
    A.tag_flip = stream_tag(kStreamTamperFlip, p.cfg_id);
    A.block_mode = p.benign_mode == 1;
    A.t3 = p.benign_dist == 1;
    A.tamper = p.tamper;
    A.clean = p.tamper_base == 1;
    A.mal_mask = p.mal_mask;
    A.sigma_b = p.sigma_b;
    A.flip_thr = p.flip_thr;
    A.flip_all = p.flip_all;
    A.scale = p.scale;
    A.bscale = p.bscale;
    A.tscale = p.tscale;
    return A;
}

// One run of a batched live pass, as the kernel reads it from the device
// table: its launch parameters and arrays.
struct SimJobDev {
    SimArgs A;
    const float* ref;
    uint16_t* h;
};

// Block-uniform state: which (shard, canary) and its scales; c is the
// global canary index that keys the noise.
struct SimBlock {
    uint32_t s, c;
    bool mal;
    float bsc;  // Eq. 2 block noise scale (BLOCK mode)
    float tsc;  // Gaussian tamper scale
};

template <bool kBlock>
__device__ __forceinline__ SimBlock sim_block(const SimArgs& A, uint64_t block) {
    SimBlock B;
    B.s = static_cast<uint32_t>(block / A.C);
    B.c = A.canary_base + static_cast<uint32_t>(block - static_cast<uint64_t>(B.s) * A.C);
    B.mal = (A.mal_mask >> B.s) & 1u;
    B.bsc = kBlock ? A.bscale[block] : 0.0f;
    B.tsc = (B.mal && (A.tamper & 1u)) ? A.tscale[block] : 0.0f;
    return B;
}

// IEEE fp32 sqrt and division on the Student-t draw's own ranges.  q is a
// sum of three squared Irwin-Hall normals (multiples of 0x1.bb67aep-16, at
// most 3.47 in magnitude): 0, handled by the caller, or in [6.9e-10, 36];
// the divisor s = sqrt(q) lies in [2.6e-5, 6] and the dividend |zb| <= 3.47.
// On these ranges the compiler's correctly rounded sequences reduce to the
// instructions below: v_sqrt_f32 with its one-ulp residual correction (the
// scaling of inputs below 2^-96 and the zero / infinity cases never apply),
// and the reciprocal with two FMA refinements of the quotient (v_div_scale
// never scales, v_div_fmas is a plain FMA, v_div_fixup returns its input).
// The results are bitwise those of sqrtf and '/': every float in
// [2^-96, 2^7) and every divisor in [2^-17, 2^4) against 256 Irwin-Hall
// dividends were compared on the device.
__device__ __forceinline__ float t3_sqrt(float q) {
    const float s = __builtin_amdgcn_sqrtf(q);
    const float dn = __uint_as_float(__float_as_uint(s) - 1u);
    const float up = __uint_as_float(__float_as_uint(s) + 1u);
    const float r_dn = __builtin_fmaf(-dn, s, q);
    const float r_up = __builtin_fmaf(-up, s, q);
    const float t = r_dn <= 0.0f ? dn : s;
    return r_up > 0.0f ? up : t;
}

__device__ __forceinline__ float t3_div(float a, float b) {
    const float y0 = __builtin_amdgcn_rcpf(b);
    const float e = __builtin_fmaf(-b, y0, 1.0f);
    const float y = __builtin_fmaf(e, y0, y0);
    const float q0 = a * y;
    const float q1 = __builtin_fmaf(__builtin_fmaf(-b, q0, a), y, q0);
    return __builtin_fmaf(__builtin_fmaf(-b, q1, a), y, q1);
}

// Eq. 2: the benign output v = base + sc * zb of elements e0..e0+7, with the
// noise scale taken from the reference a (elementwise mode) and base = a for
// independent stages (base = a + carried error in the propagation model).
template <bool kT3, bool kBlock>
__device__ __forceinline__ void benign8(const SimArgs& A, const SimBlock& B, uint32_t e0,
                                        const float a[8], const float base[8], float v[8]) {
    float zb[8];
    normals8(A.key, e0, B.c, B.s, A.tag_benign, zb);
    if (kT3) {
        float z3[8];
        normals8(A.key, e0, B.c, B.s, A.tag_t3, z3);
#pragma unroll
        for (int k = 0; k < 8; ++k) {
            const Words4 w = draw(A.key, e0 + k, B.c, B.s, A.tag_t12);
            const float z1 = irwin_hall4(w.x, w.y);
            const float z2 = irwin_hall4(w.z, w.w);
            const float q = (z1 * z1 + z2 * z2) + z3[k] * z3[k];
            zb[k] = (q == 0.0f) ? 0.0f : t3_div(zb[k], t3_sqrt(q));
        }
    }
#pragma unroll
    for (int k = 0; k < 8; ++k) {
        const float sc = kBlock ? B.bsc : A.sigma_b * fabsf(a[k]);
        v[k] = base[k] + sc * zb[k];
    }
}

// Eq. 3: the tampering of a malicious shard, in place on v (which holds the
// benign output; the clean base replaces it by the noise-free base first).
__device__ __forceinline__ void tamper8(const SimArgs& A, const SimBlock& B, uint32_t e0,
                                        const float base[8], float v[8]) {
    if (A.clean) {
#pragma unroll
        for (int k = 0; k < 8; ++k) v[k] = base[k];
    }
    if (A.tamper & 1u) {
        float zt[8];
        normals8(A.key, e0, B.c, B.s, A.tag_add, zt);
#pragma unroll
        for (int k = 0; k < 8; ++k) v[k] = v[k] + B.tsc * zt[k];
    }
    if (A.tamper & 2u) {
        const Words4 u0 = draw(A.key, e0 >> 2, B.c, B.s, A.tag_flip);
        const Words4 u1 = draw(A.key, (e0 >> 2) + 1, B.c, B.s, A.tag_flip);
        const uint32_t u[8] = {u0.x, u0.y, u0.z, u0.w, u1.x, u1.y, u1.z, u1.w};
#pragma unroll
        for (int k = 0; k < 8; ++k)
            if (A.flip_all || u[k] < A.flip_thr) v[k] = -v[k];
    }
    if (A.tamper & 4u) {
#pragma unroll
        for (int k = 0; k < 8; ++k) v[k] = A.scale * v[k];
    }
}

__device__ __forceinline__ u32x4 pack_half8(const float v[8]) {
    u32x4 o;
    o.x = to_half2_bits(v[0], v[1]);
    o.y = to_half2_bits(v[2], v[3]);
    o.z = to_half2_bits(v[4], v[5]);
    o.w = to_half2_bits(v[6], v[7]);
    return o;
}

// Live fp16 activations of elements e0..e0+7 from their references.
template <bool kT3, bool kBlock>
__device__ __forceinline__ u32x4 sim_group8(const SimArgs& A, const SimBlock& B, uint32_t e0,
                                            const f32x4& a_lo, const f32x4& a_hi) {
    const float a[8] = {a_lo.x, a_lo.y, a_lo.z, a_lo.w, a_hi.x, a_hi.y, a_hi.z, a_hi.w};
    float v[8];
    benign8<kT3, kBlock>(A, B, e0, a, a, v);
    if (B.mal) tamper8(A, B, e0, a, v);
    return pack_half8(v);
}

// The propagation model: stage s of canary c sees the previous stage's live
// error d = fp32(h_{s-1} - a_{s-1}) through a carry gain g: its noise-free
// output is u = a + fp32(g * d) (u = a for the first stage); the benign
// noise and the tamper act on u.  Updates d to this stage's error.
template <bool kT3, bool kBlock>
__device__ __forceinline__ u32x4 chain_group8(const SimArgs& A, const SimBlock& B, uint32_t e0,
                                              bool first, float gain, const f32x4& a_lo,
                                              const f32x4& a_hi, float d[8]) {
    const float a[8] = {a_lo.x, a_lo.y, a_lo.z, a_lo.w, a_hi.x, a_hi.y, a_hi.z, a_hi.w};
    float u[8], v[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) u[k] = first ? a[k] : a[k] + gain * d[k];
    benign8<kT3, kBlock>(A, B, e0, a, u, v);
    if (B.mal) tamper8(A, B, e0, u, v);
    const u32x4 o = pack_half8(v);
    const uint32_t w[4] = {o.x, o.y, o.z, o.w};
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        d[2 * k] = half_bits_to_float(w[k] & 0xFFFFu) - a[2 * k];
        d[2 * k + 1] = half_bits_to_float(w[k] >> 16) - a[2 * k + 1];
    }
    return o;
}

}  // namespace cdt
