/*
 * oracle.c -- plain, slow CPU oracle for the canary-versus-reference drift
 * detector of "Integrity of peer-to-peer distributed LLM inference under
 * malicious nodes" (Cihangiroglu & Nocera).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may link, load or
 * call this file; only the test suite, the smoke check and the CPU-baseline
 * leg of the benchmark do.  It shares no code, header, constant or table with
 * the HIP library: every constant below is written out here from its
 * published definition.
 *
 * Precision rules.
 *  - Drift (Eq. 4) and its sums are computed in fp64 directly from the
 *    definition, element by element, in index order.
 *  - AUROC (Eqs. 5-6 and the Mann-Whitney form stated right after Eq. 6) is
 *    counted pair by pair (brute force) on the fp32 scores.
 *  - The synthetic generator (the stand-in for the fp32 pipeline of Eq. 1 and
 *    the live pass of Eqs. 2-3) must reproduce fp32 arithmetic bit for bit.
 *    Every fp32 operation is computed as the fp64 operation on the fp32
 *    operands and then rounded once to fp32 (r32).  For + - * / and sqrt this
 *    equals the fp32 operation itself because 53 >= 2*24 + 2 (double rounding
 *    is innocuous; S. Figueroa, "When is double rounding innocuous?", 1995).
 *  - Build with -ffp-contract=off and without fast-math.
 *
 * The paper fixes none of the random number generator, the normal sampler or
 * the fp16 rounding; the readings used (Philox4x32-10, an Irwin-Hall sum of
 * four 16-bit uniforms, IEEE round-to-nearest-even) are listed with the
 * other readings of the paper in the design notes that accompany the code.
 */
#include <math.h>
#include <stddef.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORC_VERSION 1

int orc_version(void) { return ORC_VERSION; }

/* Round an fp64 value to fp32 (IEEE round-to-nearest-even). */
static float r32(double x) { return (float)x; }

/* ------------------------------------------------------------------------ */
/* Philox4x32-10: J. Salmon, M. Moraes, R. Dror, D. Shaw, "Parallel random   */
/* numbers: as easy as 1, 2, 3", SC'11.  Ten rounds; each round multiplies   */
/* counter words 0 and 2 by the two round multipliers (32x32 -> 64 bit),      */
/* mixes the high halves with words 1 and 3 and the round key by XOR, and     */
/* permutes the words.  The key is advanced by the two Weyl increments        */
/* (golden ratio and sqrt(3) - 1, scaled to 32 bits) before rounds 2..10.     */
/* ------------------------------------------------------------------------ */
static const uint32_t PHILOX_MUL0 = 0xD2511F53u;
static const uint32_t PHILOX_MUL1 = 0xCD9E8D57u;
static const uint32_t PHILOX_WEYL0 = 0x9E3779B9u;
static const uint32_t PHILOX_WEYL1 = 0xBB67AE85u;

void orc_philox(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4])
{
    uint32_t x0 = ctr[0], x1 = ctr[1], x2 = ctr[2], x3 = ctr[3];
    uint32_t k0 = key[0], k1 = key[1];
    for (int round = 0; round < 10; ++round) {
        if (round > 0) {
            k0 += PHILOX_WEYL0;
            k1 += PHILOX_WEYL1;
        }
        uint64_t p0 = (uint64_t)PHILOX_MUL0 * (uint64_t)x0;
        uint64_t p1 = (uint64_t)PHILOX_MUL1 * (uint64_t)x2;
        uint32_t y0 = (uint32_t)(p1 >> 32) ^ x1 ^ k0;
        uint32_t y1 = (uint32_t)p1;
        uint32_t y2 = (uint32_t)(p0 >> 32) ^ x3 ^ k1;
        uint32_t y3 = (uint32_t)p0;
        x0 = y0; x1 = y1; x2 = y2; x3 = y3;
    }
    out[0] = x0; out[1] = x1; out[2] = x2; out[3] = x3;
}

/* Random streams: the fourth counter word is (stream << 24) | id. */
enum {
    ST_REF = 0,      /* reference activations (stand-in for Eq. 1)      */
    ST_BENIGN = 1,   /* benign hardware noise delta_i (Eq. 2)             */
    ST_T12 = 2,      /* chi-square normals 1, 2 of the Student-t noise    */
    ST_T3 = 3,       /* chi-square normal 3 of the Student-t noise        */
    ST_TADD = 4,     /* Gaussian tamper direction (Eq. 3, Gaussian)       */
    ST_TFLIP = 5,    /* sign-flip selection (Eq. 3, sign flip)            */
    ST_SCRAMBLE = 6, /* scrambled-label stage j* (Section 4.5)            */
    ST_RANDOM = 7,   /* random-baseline scores (Section 4.5)              */
    ST_OUTLIER = 8,  /* outlier channel choice of the synthetic reference */
    ST_ALT = 9,      /* independent benign redraw (Section 4.5 ceiling)   */
    ST_ALT_T12 = 10, /* ... its Student-t chi-square normals 1, 2          */
    ST_ALT_T3 = 11   /* ... and normal 3                                   */
};

static void philox_at(uint64_t seed, uint32_t w0, uint32_t w1, uint32_t w2,
                      uint32_t stream, uint32_t id, uint32_t out[4])
{
    uint32_t ctr[4] = {w0, w1, w2, (stream << 24) | (id & 0xFFFFFFu)};
    uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
    orc_philox(ctr, key, out);
}

/* ------------------------------------------------------------------------ */
/* Standard normal stand-in: the Irwin-Hall sum of four independent 16-bit   */
/* uniforms, centred and scaled to unit variance.  Each 16-bit uniform has    */
/* mean (2^16-1)/2 and variance (2^32-1)/12, so the centred sum n has         */
/* variance (2^32-1)/3 and z = n * sqrt(3/(2^32-1)).                          */
/* ------------------------------------------------------------------------ */
static float unit_scale_k16(void)
{
    return r32(sqrt(3.0 / 4294967295.0));
}

float orc_z16(uint32_t w0, uint32_t w1)
{
    int32_t n = (int32_t)(w0 & 0xFFFFu) + (int32_t)(w0 >> 16) + (int32_t)(w1 & 0xFFFFu) +
                (int32_t)(w1 >> 16) - 131070;
    return r32((double)(float)n * (double)unit_scale_k16());
}

float orc_k16(void) { return unit_scale_k16(); }

/* One normal per element: element e uses Philox call q = e / 2, words 0-1 for
 * even e and words 2-3 for odd e.  Counter = (q, c, s, stream|id). */
static float normal1(uint64_t seed, uint32_t stream, uint32_t id, uint32_t s, uint32_t c,
                     uint32_t e)
{
    uint32_t w[4];
    philox_at(seed, e >> 1, c, s, stream, id, w);
    return (e & 1u) ? orc_z16(w[2], w[3]) : orc_z16(w[0], w[1]);
}

/* Two normals per element from one Philox call with q = e. */
static void normal2(uint64_t seed, uint32_t stream, uint32_t id, uint32_t s, uint32_t c,
                    uint32_t e, float* z1, float* z2)
{
    uint32_t w[4];
    philox_at(seed, e, c, s, stream, id, w);
    *z1 = orc_z16(w[0], w[1]);
    *z2 = orc_z16(w[2], w[3]);
}

/* One uniform 32-bit word per element: Philox call q = e / 4, word e mod 4. */
static uint32_t word1(uint64_t seed, uint32_t stream, uint32_t id, uint32_t s, uint32_t c,
                      uint32_t e)
{
    uint32_t w[4];
    philox_at(seed, e >> 2, c, s, stream, id, w);
    return w[e & 3u];
}

/* ------------------------------------------------------------------------ */
/* IEEE 754 binary16 conversion, round to nearest, ties to even.  The live   */
/* activations travel in fp16 (Section 3.3); subnormals are kept and values  */
/* at or beyond the overflow midpoint become infinities.                     */
/* ------------------------------------------------------------------------ */
uint16_t orc_f16_rne(float xf)
{
    double x = (double)xf;
    uint16_t sign = signbit(x) ? 0x8000u : 0u;
    if (isnan(x))
        return (uint16_t)(sign | 0x7E00u);
    double ax = fabs(x);
    /* Largest finite half is 65504 = 2047 * 2^5; the next step would be 2^16,
     * so the midpoint 65520 and everything above rounds to infinity. */
    if (ax >= 65520.0)
        return (uint16_t)(sign | 0x7C00u);
    /* Spacing of representable halves around ax. */
    double quantum;
    if (ax < 0x1p-14) {
        quantum = 0x1p-24; /* subnormal spacing */
    } else {
        int e2;
        frexp(ax, &e2); /* ax = f * 2^e2, f in [0.5, 1) */
        quantum = ldexp(1.0, (e2 - 1) - 10);
    }
    double r = ax / quantum; /* exact: division by a power of two */
    double f = floor(r);
    double frac = r - f;     /* exact */
    if (frac > 0.5 || (frac == 0.5 && fmod(f, 2.0) == 1.0))
        f += 1.0;
    double v = f * quantum; /* the rounded magnitude, exact */
    if (v == 0.0)
        return sign;
    if (v < 0x1p-14)
        return (uint16_t)(sign | (uint16_t)(v / 0x1p-24));
    int e2;
    frexp(v, &e2);
    int ex = e2 - 1; /* v in [2^ex, 2^(ex+1)) */
    uint16_t mant = (uint16_t)((v / ldexp(1.0, ex) - 1.0) * 1024.0);
    return (uint16_t)(sign | (uint16_t)((ex + 15) << 10) | mant);
}

double orc_f16_value(uint16_t bits)
{
    double sign = (bits & 0x8000u) ? -1.0 : 1.0;
    int ex = (bits >> 10) & 0x1F;
    int mant = bits & 0x3FF;
    if (ex == 0x1F)
        return mant ? NAN : sign * INFINITY;
    if (ex == 0)
        return sign * ldexp((double)mant, -24);
    return sign * ldexp(1.0 + (double)mant / 1024.0, ex - 15);
}

/* Convert count consecutive fp32 bit patterns starting at `start`. */
void orc_f16_rne_range(uint64_t start, uint64_t count, uint16_t* out)
{
    for (uint64_t i = 0; i < count; ++i) {
        uint32_t bits = (uint32_t)(start + i);
        float x;
        memcpy(&x, &bits, 4);
        out[i] = orc_f16_rne(x);
    }
}

void orc_f16_rne_array(uint64_t n, const float* x, uint16_t* out)
{
    for (uint64_t i = 0; i < n; ++i)
        out[i] = orc_f16_rne(x[i]);
}

/* ------------------------------------------------------------------------ */
/* Synthetic fp32 references (stand-in for the precomputed a*_i of Eq. 1 and */
/* Section 3.3): a[s][c][t][j] = fp32(z_REF * gain[j]).  gain marks outlier  */
/* channels: the n_out channels j with the smallest (word, j) pairs, word =  */
/* Philox((j, 0, 0, OUTLIER|ref_set_id))[0], get gain `big`, the rest 1.      */
/* ------------------------------------------------------------------------ */
typedef struct {
    uint32_t word;
    uint32_t j;
} orc_keyed;

static int cmp_keyed(const void* pa, const void* pb)
{
    const orc_keyed* a = (const orc_keyed*)pa;
    const orc_keyed* b = (const orc_keyed*)pb;
    if (a->word != b->word)
        return a->word < b->word ? -1 : 1;
    if (a->j != b->j)
        return a->j < b->j ? -1 : 1;
    return 0;
}

int orc_outlier_gain(uint32_t H, uint32_t n_out, float big, uint64_t seed, uint32_t ref_set_id,
                     float* gain)
{
    if (n_out > H)
        return 1;
    orc_keyed* keys = (orc_keyed*)malloc(sizeof(orc_keyed) * (H ? H : 1));
    if (!keys)
        return 2;
    for (uint32_t j = 0; j < H; ++j) {
        uint32_t w[4];
        philox_at(seed, j, 0, 0, ST_OUTLIER, ref_set_id, w);
        keys[j].word = w[0];
        keys[j].j = j;
        gain[j] = 1.0f;
    }
    qsort(keys, H, sizeof(orc_keyed), cmp_keyed);
    for (uint32_t r = 0; r < n_out; ++r)
        gain[keys[r].j] = big;
    free(keys);
    return 0;
}

/* Elements [e0, e0 + count) of block (s, c), element e = t*H + j. */
void orc_ref_range(uint32_t s, uint32_t c, uint32_t H, uint64_t e0, uint64_t count,
                   uint64_t seed, uint32_t ref_set_id, const float* gain, float* out)
{
    for (uint64_t k = 0; k < count; ++k) {
        uint32_t e = (uint32_t)(e0 + k);
        uint32_t j = e % H;
        float z = normal1(seed, ST_REF, ref_set_id, s, c, e);
        out[k] = r32((double)z * (double)gain[j]);
    }
}

void orc_ref_block(uint32_t s, uint32_t c, uint32_t T, uint32_t H, uint64_t seed,
                   uint32_t ref_set_id, const float* gain, float* out)
{
    orc_ref_range(s, c, H, 0, (uint64_t)T * H, seed, ref_set_id, gain, out);
}

/* Whole reference array [S][C][T][H]. */
void orc_ref_synth(uint32_t S, uint32_t C, uint32_t T, uint32_t H, uint64_t seed,
                   uint32_t ref_set_id, const float* gain, float* out)
{
    uint64_t n = (uint64_t)T * H;
    for (uint32_t s = 0; s < S; ++s)
        for (uint32_t c = 0; c < C; ++c)
            orc_ref_block(s, c, T, H, seed, ref_set_id, gain, out + ((uint64_t)s * C + c) * n);
}

/* ------------------------------------------------------------------------ */
/* Block statistics of a reference block: sum of squares (gives the rms used */
/* by the per-element Gaussian tamper) and sum of magnitudes (gives mu_i of   */
/* Eq. 2, the mean absolute activation).                                      */
/* ------------------------------------------------------------------------ */
void orc_ref_stats_block(uint64_t n, const float* a, double* sumsq, double* sumabs)
{
    double q = 0.0, m = 0.0;
    for (uint64_t e = 0; e < n; ++e) {
        double x = (double)a[e];
        q += x * x;
        m += fabs(x);
    }
    *sumsq = q;
    *sumabs = m;
}

void orc_ref_stats(uint32_t S, uint32_t C, uint32_t T, uint32_t H, const float* ref, double* sumsq,
                   double* sumabs)
{
    uint64_t n = (uint64_t)T * H;
    for (uint64_t b = 0; b < (uint64_t)S * C; ++b)
        orc_ref_stats_block(n, ref + b * n, sumsq + b, sumabs + b);
}

/* Per-block scale factors, each rounded once to fp32:
 *   tscale = eps * sqrt(sumsq / (T H))     (Gaussian tamper, eps times rms)
 *   bscale = sigma_b * (sumabs / (T H))    (Eq. 2 block noise sigma_hw mu_i) */
void orc_block_scales(uint64_t nblocks, uint32_t T, uint32_t H, const double* sumsq,
                      const double* sumabs, double eps, double sigma_b, float* tscale,
                      float* bscale)
{
    double n = (double)T * (double)H;
    for (uint64_t b = 0; b < nblocks; ++b) {
        double rms = n > 0 ? sqrt(sumsq[b] / n) : 0.0;
        double mu = n > 0 ? sumabs[b] / n : 0.0;
        if (tscale)
            tscale[b] = r32(eps * rms);
        if (bscale)
            bscale[b] = r32(sigma_b * mu);
    }
}

/* ------------------------------------------------------------------------ */
/* Live activations of one (shard, canary) block.                            */
/*  benign (Eq. 2):   v = a + sc * zb, sc = sigma_b |a| (elementwise) or the  */
/*                    block scale sigma_hw mu_i; zb a unit normal or a unit-   */
/*                    variance Student-t with 3 degrees of freedom.            */
/*  tamper (Eq. 3), malicious shards only, applied to v (or to a when the     */
/*  clean base is asked for), in this order:                                   */
/*     Gaussian  v = v + tscale * zT                                          */
/*     sign flip v = -v where the element is selected (all when p >= 1)       */
/*     rescale   v = scale * v                                                */
/*  output: h = fp16(v), round to nearest even.                               */
/* ------------------------------------------------------------------------ */
enum { ORC_NOISE_ELEMENTWISE = 0, ORC_NOISE_BLOCK = 1 };
enum { ORC_DIST_GAUSS = 0, ORC_DIST_T3 = 1 };
enum { ORC_T_ADD = 1, ORC_T_FLIP = 2, ORC_T_SCALE = 4 };
enum { ORC_BASE_BENIGN = 0, ORC_BASE_CLEAN = 1 };

/* Flip threshold: an element flips when its uniform 32-bit word u satisfies
 * u < floor(p 2^32); p >= 1 flips every element. */
static int flip_selected(double p, uint32_t u)
{
    if (p >= 1.0)
        return 1;
    if (!(p > 0.0))
        return 0;
    double thr = floor(p * 4294967296.0);
    return (double)u < thr;
}

/* Elements [e0, e0 + count) of block (s, c); ref and h hold just that range. */
/* Eq. 2: the benign output v = a + sc * zb of element e of block (s, c).
 * redraw != 0 draws the noise from the ALT streams: an independent benign
 * recompute of the same stage (Section 4.5, recompute ceiling and
 * noisy-reference ablation). */
static float benign_value(uint32_t s, uint32_t c, uint32_t e, uint64_t seed, uint32_t cfg_id,
                          int benign_mode, int benign_dist, float sigma_f, float bscale,
                          int redraw, float a, float base)
{
    uint32_t st_benign = redraw ? ST_ALT : ST_BENIGN;
    uint32_t st_t12 = redraw ? ST_ALT_T12 : ST_T12;
    uint32_t st_t3 = redraw ? ST_ALT_T3 : ST_T3;
    float sc = (benign_mode == ORC_NOISE_BLOCK) ? bscale : r32((double)sigma_f * fabs((double)a));
    float zb = normal1(seed, st_benign, cfg_id, s, c, e);
    if (benign_dist == ORC_DIST_T3) {
        float z1, z2;
        normal2(seed, st_t12, cfg_id, s, c, e, &z1, &z2);
        float z3 = normal1(seed, st_t3, cfg_id, s, c, e);
        float q = r32((double)r32((double)r32((double)z1 * z1) + (double)r32((double)z2 * z2)) +
                      (double)r32((double)z3 * z3));
        zb = (q == 0.0f) ? 0.0f : r32((double)zb / (double)r32(sqrt((double)q)));
    }
    return r32((double)base + (double)r32((double)sc * (double)zb));
}

/* Eq. 3: the tampering of a malicious stage applied to its benign output v,
 * or to the noise-free output `base` for the clean base, in this order:
 * Gaussian, sign flip, rescale. */
static float tamper_value(uint32_t s, uint32_t c, uint32_t e, uint64_t seed, uint32_t cfg_id,
                          uint32_t tamper, int tamper_base, float tscale, double flip_p,
                          float scale_f, float base, float v)
{
    if (tamper_base == ORC_BASE_CLEAN)
        v = base;
    if (tamper & ORC_T_ADD) {
        float zt = normal1(seed, ST_TADD, cfg_id, s, c, e);
        v = r32((double)v + (double)r32((double)tscale * (double)zt));
    }
    if (tamper & ORC_T_FLIP) {
        uint32_t u = word1(seed, ST_TFLIP, cfg_id, s, c, e);
        if (flip_selected(flip_p, u))
            v = -v;
    }
    if (tamper & ORC_T_SCALE)
        v = r32((double)scale_f * (double)v);
    return v;
}

int orc_sim_range_ex(uint32_t s, uint32_t c, uint64_t e0, uint64_t count, uint64_t seed,
                     uint32_t cfg_id, int benign_mode, int benign_dist, double sigma_b,
                     float bscale, int malicious, uint32_t tamper, int tamper_base, float tscale,
                     double flip_p, double scale, int redraw, const float* ref, uint16_t* h)
{
    float sigma_f = r32(sigma_b);
    float scale_f = r32(scale);
    for (uint64_t k = 0; k < count; ++k) {
        uint32_t e = (uint32_t)(e0 + k);
        float a = ref[k];
        float v = benign_value(s, c, e, seed, cfg_id, benign_mode, benign_dist, sigma_f, bscale,
                               redraw, a, a);

        if (malicious)
            v = tamper_value(s, c, e, seed, cfg_id, tamper, tamper_base, tscale, flip_p, scale_f,
                             a, v);
        h[k] = orc_f16_rne(v);
    }
    return 0;
}

/* Propagation model (Sections 4.4, 5.3-5.5: depth, position, collusion,
 * frontier).  Eq. 2 feeds stage i the live h_{i-1}; with a carry gain g the
 * live error of the previous stage, d = fp32(h_{s-1} - a_{s-1}), enters
 * stage s as u = fp32(a + fp32(g d)) (u = a for stage 0).  The benign step is
 * v = fp32(u + fp32(sc zb)) with sc from |a| (or the block scale), the clean
 * base of a malicious stage is u, and h = fp16(v).  Stages run in order for
 * each canary and element; g = 0 is the independent live pass. */
/* Noise-free output u of stage s under the propagation model: its reference
 * a plus the carried live error g d of the stage before (a at stage 0). */
static float carried_input(uint32_t s, float a, float g, float d)
{
    return (s == 0) ? a : r32((double)a + (double)r32((double)g * (double)d));
}

/* Canary c of the arrays is the run's canary c0 + c: that global index keys
 * its noise (c0 = 0 for a whole run). */
int orc_canary_sim_chain_at(uint32_t c0, uint32_t S, uint32_t C, uint32_t T, uint32_t H,
                            uint64_t seed, uint32_t cfg_id, int benign_mode, int benign_dist,
                            double sigma_b, const float* bscale, uint64_t mal_mask,
                            uint32_t tamper, int tamper_base, const float* tscale, double flip_p,
                            double scale, int redraw, double carry, const float* ref, uint16_t* h)
{
    uint64_t n = (uint64_t)T * H;
    float sigma_f = r32(sigma_b);
    float scale_f = r32(scale);
    float g = r32(carry);
    for (uint32_t c = 0; c < C; ++c)
        for (uint64_t k = 0; k < n; ++k) {
            uint32_t e = (uint32_t)k;
            float d = 0.0f;
            for (uint32_t s = 0; s < S; ++s) {
                uint64_t b = (uint64_t)s * C + c;
                float a = ref[b * n + k];
                float u = carried_input(s, a, g, d);
                float v = benign_value(s, c0 + c, e, seed, cfg_id, benign_mode, benign_dist,
                                       sigma_f, bscale ? bscale[b] : 0.0f, redraw, a, u);
                if (s < 64 && ((mal_mask >> s) & 1u))
                    v = tamper_value(s, c0 + c, e, seed, cfg_id, tamper, tamper_base,
                                     tscale ? tscale[b] : 0.0f, flip_p, scale_f, u, v);
                uint16_t hb = orc_f16_rne(v);
                h[b * n + k] = hb;
                d = r32(orc_f16_value(hb) - (double)a);
            }
        }
    return 0;
}

int orc_canary_sim_chain(uint32_t S, uint32_t C, uint32_t T, uint32_t H, uint64_t seed,
                         uint32_t cfg_id, int benign_mode, int benign_dist, double sigma_b,
                         const float* bscale, uint64_t mal_mask, uint32_t tamper,
                         int tamper_base, const float* tscale, double flip_p, double scale,
                         int redraw, double carry, const float* ref, uint16_t* h)
{
    return orc_canary_sim_chain_at(0, S, C, T, H, seed, cfg_id, benign_mode, benign_dist, sigma_b,
                                   bscale, mal_mask, tamper, tamper_base, tscale, flip_p, scale,
                                   redraw, carry, ref, h);
}

/* Exact-norm Gaussian tamper of Section 3.2, tau(v) = v + eps ||v|| N / ||N||,
 * for block (s, c): vv = sum v^2 over the untampered output (the benign
 * a + delta, or a for the clean base) and zz = sum z^2 over the TAMPER_ADD
 * normals, in fp64; the scale of those normals is fp32(eps sqrt(vv / zz)). */
float orc_tamper_scale_exact_block(uint32_t s, uint32_t c, uint32_t T, uint32_t H, uint64_t seed,
                                   uint32_t cfg_id, int benign_mode, int benign_dist,
                                   double sigma_b, float bscale, int tamper_base, int redraw,
                                   double eps, const float* ref, double* vv_out, double* zz_out)
{
    float sigma_f = r32(sigma_b);
    double vv = 0.0, zz = 0.0;
    uint64_t n = (uint64_t)T * H;
    for (uint64_t k = 0; k < n; ++k) {
        uint32_t e = (uint32_t)k;
        float a = ref[k];
        float v = (tamper_base == ORC_BASE_CLEAN)
                      ? a
                      : benign_value(s, c, e, seed, cfg_id, benign_mode, benign_dist, sigma_f,
                                     bscale, redraw, a, a);
        float z = normal1(seed, ST_TADD, cfg_id, s, c, e);
        vv += (double)v * (double)v;
        zz += (double)z * (double)z;
    }
    if (vv_out)
        *vv_out = vv;
    if (zz_out)
        *zz_out = zz;
    return zz > 0.0 ? r32(eps * sqrt(vv / zz)) : 0.0f;
}

/* The same exact-norm tamper under the propagation model (carry g > 0).
 * For a malicious stage m the untampered output v is the stage's benign
 * output given the live error carried in from stage m - 1 (the clean base:
 * the noise-free u), so it depends on everything upstream, earlier
 * malicious stages included.  The scales are therefore found stage by stage
 * in pipeline order: for each malicious stage m, every element of the block
 * is walked through stages 0 .. m as the propagation model walks it (earlier
 * malicious stages tampered with the scales already found and the run's
 * other tamper settings), and vv = sum v^2 at stage m, zz = sum z^2 of its
 * TAMPER_ADD normals give tscale[m][c] = fp32(eps sqrt(vv / zz)).  Entries
 * of benign stages are 0 (norms 0 as well).  Canary c of the arrays is the
 * run's canary c0 + c.  tscale, norms: [S][C] and [S][C][2] outputs. */
int orc_tamper_scale_exact_chain_at(uint32_t c0, uint32_t S, uint32_t C, uint32_t T, uint32_t H,
                                    uint64_t seed, uint32_t cfg_id, int benign_mode,
                                    int benign_dist, double sigma_b, const float* bscale,
                                    uint64_t mal_mask, uint32_t tamper, int tamper_base,
                                    double flip_p, double scale, int redraw, double carry,
                                    double eps, const float* ref, float* tscale, double* norms)
{
    uint64_t n = (uint64_t)T * H;
    float sigma_f = r32(sigma_b);
    float scale_f = r32(scale);
    float g = r32(carry);
    for (uint64_t b = 0; b < (uint64_t)S * C; ++b) {
        tscale[b] = 0.0f;
        if (norms) {
            norms[2 * b] = 0.0;
            norms[2 * b + 1] = 0.0;
        }
    }
    for (uint32_t c = 0; c < C; ++c)
        for (uint32_t m = 0; m < S && m < 64; ++m) {
            if (!((mal_mask >> m) & 1u))
                continue;
            double vv = 0.0, zz = 0.0;
            for (uint64_t k = 0; k < n; ++k) {
                uint32_t e = (uint32_t)k;
                float d = 0.0f;
                for (uint32_t s = 0; s <= m; ++s) {
                    uint64_t b = (uint64_t)s * C + c;
                    float a = ref[b * n + k];
                    float u = carried_input(s, a, g, d);
                    float v = benign_value(s, c0 + c, e, seed, cfg_id, benign_mode, benign_dist,
                                           sigma_f, bscale ? bscale[b] : 0.0f, redraw, a, u);
                    if (s == m) {
                        float vt = (tamper_base == ORC_BASE_CLEAN) ? u : v;
                        float z = normal1(seed, ST_TADD, cfg_id, s, c0 + c, e);
                        vv += (double)vt * (double)vt;
                        zz += (double)z * (double)z;
                        break;
                    }
                    if ((mal_mask >> s) & 1u)
                        v = tamper_value(s, c0 + c, e, seed, cfg_id, tamper, tamper_base,
                                         tscale[b], flip_p, scale_f, u, v);
                    d = r32(orc_f16_value(orc_f16_rne(v)) - (double)a);
                }
            }
            uint64_t bm = (uint64_t)m * C + c;
            tscale[bm] = zz > 0.0 ? r32(eps * sqrt(vv / zz)) : 0.0f;
            if (norms) {
                norms[2 * bm] = vv;
                norms[2 * bm + 1] = zz;
            }
        }
    return 0;
}

int orc_sim_range(uint32_t s, uint32_t c, uint64_t e0, uint64_t count, uint64_t seed,
                  uint32_t cfg_id, int benign_mode, int benign_dist, double sigma_b, float bscale,
                  int malicious, uint32_t tamper, int tamper_base, float tscale, double flip_p,
                  double scale, const float* ref, uint16_t* h)
{
    return orc_sim_range_ex(s, c, e0, count, seed, cfg_id, benign_mode, benign_dist, sigma_b,
                            bscale, malicious, tamper, tamper_base, tscale, flip_p, scale, 0, ref,
                            h);
}

int orc_sim_block(uint32_t s, uint32_t c, uint32_t T, uint32_t H, uint64_t seed, uint32_t cfg_id,
                  int benign_mode, int benign_dist, double sigma_b, float bscale, int malicious,
                  uint32_t tamper, int tamper_base, float tscale, double flip_p, double scale,
                  const float* ref, uint16_t* h)
{
    return orc_sim_range(s, c, 0, (uint64_t)T * H, seed, cfg_id, benign_mode, benign_dist,
                         sigma_b, bscale, malicious, tamper, tamper_base, tscale, flip_p, scale,
                         ref, h);
}

/* Whole live array [S][C][T][H].  tscale and bscale are [S][C] (may be NULL
 * when unused); bit s of mal_mask marks shard s malicious. */
int orc_canary_sim(uint32_t S, uint32_t C, uint32_t T, uint32_t H, uint64_t seed, uint32_t cfg_id,
                   int benign_mode, int benign_dist, double sigma_b, const float* bscale,
                   uint64_t mal_mask, uint32_t tamper, int tamper_base, const float* tscale,
                   double flip_p, double scale, int redraw, const float* ref, uint16_t* h)
{
    uint64_t n = (uint64_t)T * H;
    for (uint32_t s = 0; s < S; ++s)
        for (uint32_t c = 0; c < C; ++c) {
            uint64_t b = (uint64_t)s * C + c;
            int mal = s < 64 && ((mal_mask >> s) & 1u);
            orc_sim_range_ex(s, c, 0, n, seed, cfg_id, benign_mode, benign_dist, sigma_b,
                             bscale ? bscale[b] : 0.0f, mal, tamper, tamper_base,
                             tscale ? tscale[b] : 0.0f, flip_p, scale, redraw, ref + b * n,
                             h + b * n);
        }
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Relative-L2 mismatch, Eq. 4:  m = ||h - a||_F / ||a||_F over the T x d    */
/* block, with h the fp16 live activation (widened exactly) and a the fp32    */
/* reference.  D = sum (h - a)^2 and R = sum a^2 in fp64, index order.        */
/* Degenerate block: R = 0 gives m = 0 when D = 0 and +inf otherwise.         */
/* ------------------------------------------------------------------------ */
double orc_drift_block(uint64_t n, const uint16_t* h, const float* a, double* D_out, double* R_out)
{
    double D = 0.0, R = 0.0;
    for (uint64_t e = 0; e < n; ++e) {
        double hv = orc_f16_value(h[e]);
        double av = (double)a[e];
        double d = hv - av;
        D += d * d;
        R += av * av;
    }
    if (D_out)
        *D_out = D;
    if (R_out)
        *R_out = R;
    if (R == 0.0)
        return D == 0.0 ? 0.0 : INFINITY;
    return sqrt(D / R);
}

/* Scores of every block, written as [C][S] (one canary's k scores adjacent,
 * as Eq. 5 ranks them), both as fp64 and as fp32. */
void orc_drift_score(uint32_t S, uint32_t C, uint32_t T, uint32_t H, const uint16_t* h,
                     const float* ref, double* score64, float* score32, double* num_den)
{
    uint64_t n = (uint64_t)T * H;
    for (uint32_t s = 0; s < S; ++s)
        for (uint32_t c = 0; c < C; ++c) {
            uint64_t b = (uint64_t)s * C + c;
            double D, R;
            double m = orc_drift_block(n, h + b * n, ref + b * n, &D, &R);
            uint64_t o = (uint64_t)c * S + s;
            if (score64)
                score64[o] = m;
            if (score32)
                score32[o] = r32(m);
            if (num_den) {
                num_den[2 * o] = D;
                num_den[2 * o + 1] = R;
            }
        }
}

/* Relative-L2 mismatch against an fp16 reference r (Eq. 4 with the stored
 * fp32 reference replaced by a second live pass: the noisy-reference
 * ablation and the redundant-recompute ceiling of Section 4.5). */
double orc_drift_block_f16ref(uint64_t n, const uint16_t* h, const uint16_t* r, double* D_out,
                              double* R_out)
{
    double D = 0.0, R = 0.0;
    for (uint64_t e = 0; e < n; ++e) {
        double hv = orc_f16_value(h[e]);
        double rv = orc_f16_value(r[e]);
        double d = hv - rv;
        D += d * d;
        R += rv * rv;
    }
    if (D_out)
        *D_out = D;
    if (R_out)
        *R_out = R;
    if (R == 0.0)
        return D == 0.0 ? 0.0 : INFINITY;
    return sqrt(D / R);
}

void orc_drift_score_f16ref(uint32_t S, uint32_t C, uint32_t T, uint32_t H, const uint16_t* h,
                            const uint16_t* r, double* score64, float* score32)
{
    uint64_t n = (uint64_t)T * H;
    for (uint32_t s = 0; s < S; ++s)
        for (uint32_t c = 0; c < C; ++c) {
            uint64_t b = (uint64_t)s * C + c;
            double m = orc_drift_block_f16ref(n, h + b * n, r + b * n, NULL, NULL);
            uint64_t o = (uint64_t)c * S + s;
            if (score64)
                score64[o] = m;
            if (score32)
                score32[o] = r32(m);
        }
}

/* Cosine mismatch, the metric ablation of Section 4.4:
 *   m~ = 1 - (h . a) / (||h|| ||a||),
 * with the three sums in extended precision (long double) from exact
 * products.  A block where h or a is all zero has no angle; it scores 0 when
 * both are zero and 1 otherwise. */
double orc_cosine_block(uint64_t n, const uint16_t* h, const float* a)
{
    long double hh = 0.0L, aa = 0.0L, ha = 0.0L;
    for (uint64_t e = 0; e < n; ++e) {
        long double hv = (long double)orc_f16_value(h[e]);
        long double av = (long double)a[e];
        hh += hv * hv;
        aa += av * av;
        ha += hv * av;
    }
    if (hh == 0.0L || aa == 0.0L)
        return (hh == 0.0L && aa == 0.0L) ? 0.0 : 1.0;
    return (double)(1.0L - ha / sqrtl(hh * aa));
}

/* The same against an fp16 reference r (a second live pass). */
double orc_cosine_block_f16ref(uint64_t n, const uint16_t* h, const uint16_t* r)
{
    long double hh = 0.0L, rr = 0.0L, hr = 0.0L;
    for (uint64_t e = 0; e < n; ++e) {
        long double hv = (long double)orc_f16_value(h[e]);
        long double rv = (long double)orc_f16_value(r[e]);
        hh += hv * hv;
        rr += rv * rv;
        hr += hv * rv;
    }
    if (hh == 0.0L || rr == 0.0L)
        return (hh == 0.0L && rr == 0.0L) ? 0.0 : 1.0;
    return (double)(1.0L - hr / sqrtl(hh * rr));
}

void orc_cosine_score(uint32_t S, uint32_t C, uint32_t T, uint32_t H, const uint16_t* h,
                      const float* ref, double* score64, float* score32)
{
    uint64_t n = (uint64_t)T * H;
    for (uint32_t s = 0; s < S; ++s)
        for (uint32_t c = 0; c < C; ++c) {
            uint64_t b = (uint64_t)s * C + c;
            double m = orc_cosine_block(n, h + b * n, ref + b * n);
            uint64_t o = (uint64_t)c * S + s;
            if (score64)
                score64[o] = m;
            if (score32)
                score32[o] = r32(m);
        }
}

/* ------------------------------------------------------------------------ */
/* Detection AUROC.                                                          */
/* Score order: the numeric order, -0 ties +0, and NaN above every number    */
/* (+inf included), NaN tying NaN.  Eq. 5 ranks the stage with the larger    */
/* mismatch as the more suspicious one; a block whose mismatch is not a      */
/* number (a NaN in the activations it returned) has no finite agreement     */
/* with the reference at all, so it ranks as the most suspicious, and a      */
/* single corrupted element cannot hide a stage below the benign ones.       */
/* ------------------------------------------------------------------------ */
static int score_cmp(float x, float y)
{
    int nx = isnan(x), ny = isnan(y);
    if (nx || ny)
        return nx && ny ? 0 : (nx ? 1 : -1);
    if (x > y)
        return 1;
    if (x < y)
        return -1;
    return 0;
}

int orc_score_cmp(float x, float y) { return score_cmp(x, y); }

enum { ORC_AUROC_CONTROL = 1, ORC_AUROC_POOLED = 2, ORC_CTRL_INCLUDE_TRUE = 4, ORC_AUROC_RANDOM = 8 };

/* Random-baseline score of (canary t, stage s) (Section 4.5): Uniform[0, 1)
 * with 24 random bits, u = (w >> 8) 2^-24, w = Philox word 0 of counter
 * (t, s, 0, RANDOM|cfg_id). */
float orc_random_score(uint64_t seed, uint32_t cfg_id, uint32_t t, uint32_t s)
{
    uint32_t w[4];
    philox_at(seed, t, s, 0, ST_RANDOM, cfg_id, w);
    return (float)((double)(w[0] >> 8) * 0x1p-24);
}

/* Scrambled-label stage for canary t (Section 4.5): a uniformly chosen
 * benign stage j* != i*.  With benign stages b_0 < b_1 < ... < b_{B-1},
 * u = Philox((t, 0, 0, SCRAMBLE|cfg_id))[0] and j* = b_{u mod B}.
 * Returns -1 when there is no benign stage. */
int orc_scramble_jstar(uint32_t S, uint64_t pos_mask, uint64_t seed, uint32_t cfg_id, uint32_t t)
{
    uint32_t benign[64];
    uint32_t B = 0;
    for (uint32_t j = 0; j < S && j < 64; ++j)
        if (!((pos_mask >> j) & 1u))
            benign[B++] = j;
    if (B == 0)
        return -1;
    uint32_t w[4];
    philox_at(seed, t, 0, 0, ST_SCRAMBLE, cfg_id, w);
    return (int)benign[w[0] % B];
}

/* Eq. 5 per canary: for each canary t of one configuration (scores [C][S],
 * positives = shards in pos_mask), out[t][0..5] = the counts whose ratio is
 * A^(t): G_t, E_t (positive i beats / ties negative j, over all such pairs
 * of that canary), then the same two for the scrambled-label control (the
 * chosen benign stage j* against the others, Section 4.5) and for the
 * random baseline (every score replaced by its uniform, Section 4.5).  The
 * control and baseline entries are 0 unless their flag is set.  Draws use
 * the canary's global index canary_base + t. */
int orc_auroc_canaries(uint32_t S, uint32_t C, const float* scores, uint64_t pos_mask,
                       uint64_t seed, uint32_t cfg_id, uint32_t canary_base, uint32_t flags,
                       uint32_t* out)
{
    if (S > 64)
        return 1;
    for (uint32_t t = 0; t < C; ++t) {
        const float* m = scores + (uint64_t)t * S;
        const uint32_t tg = canary_base + t;
        uint32_t* o = out + (uint64_t)t * 6;
        for (int k = 0; k < 6; ++k)
            o[k] = 0;
        for (uint32_t i = 0; i < S; ++i) {
            if (!((pos_mask >> i) & 1u))
                continue;
            for (uint32_t j = 0; j < S; ++j) {
                if ((pos_mask >> j) & 1u)
                    continue;
                int r = score_cmp(m[i], m[j]);
                o[0] += (r > 0);
                o[1] += (r == 0);
                if (flags & ORC_AUROC_RANDOM) {
                    int q = score_cmp(orc_random_score(seed, cfg_id, tg, i),
                                      orc_random_score(seed, cfg_id, tg, j));
                    o[4] += (q > 0);
                    o[5] += (q == 0);
                }
            }
        }
        if (flags & ORC_AUROC_CONTROL) {
            const int skip_true = !(flags & ORC_CTRL_INCLUDE_TRUE);
            int js = orc_scramble_jstar(S, pos_mask, seed, cfg_id, tg);
            if (js >= 0)
                for (uint32_t j = 0; j < S; ++j) {
                    if (j == (uint32_t)js)
                        continue;
                    if (skip_true && ((pos_mask >> j) & 1u))
                        continue;
                    int r = score_cmp(m[js], m[j]);
                    o[2] += (r > 0);
                    o[3] += (r == 0);
                }
        }
    }
    return 0;
}

/* One configuration: scores [C][S] (fp32), positives = shards in pos_mask.
 * counts[0..5] = G, E, pairs (Eq. 5 summed over canaries: G counts
 *   m_i > m_j, E counts m_i == m_j, over i in M, j not in M),
 *   then the same three for the scrambled-label control;
 * pooled[0..2] = G, E, pairs over all positive/negative score pairs of the
 *   configuration (the Mann-Whitney U of all C*S scores pooled). */
int orc_auroc_config(uint32_t S, uint32_t C, const float* scores, uint64_t pos_mask,
                     uint64_t seed, uint32_t cfg_id, uint32_t flags, uint64_t* counts,
                     uint64_t* pooled, uint64_t* baseline)
{
    if (S > 64)
        return 1;
    for (int k = 0; k < 6; ++k)
        counts[k] = 0;
    if (pooled)
        for (int k = 0; k < 3; ++k)
            pooled[k] = 0;
    if (baseline)
        for (int k = 0; k < 3; ++k)
            baseline[k] = 0;

    for (uint32_t t = 0; t < C; ++t) {
        const float* m = scores + (uint64_t)t * S;
        for (uint32_t i = 0; i < S; ++i) {
            if (!((pos_mask >> i) & 1u))
                continue;
            for (uint32_t j = 0; j < S; ++j) {
                if ((pos_mask >> j) & 1u)
                    continue;
                int r = score_cmp(m[i], m[j]);
                counts[0] += (r > 0);
                counts[1] += (r == 0);
                counts[2] += 1;
            }
        }
        if (flags & ORC_AUROC_CONTROL) {
            int js = orc_scramble_jstar(S, pos_mask, seed, cfg_id, t);
            if (js >= 0) {
                for (uint32_t j = 0; j < S; ++j) {
                    if (j == (uint32_t)js)
                        continue;
                    if (!(flags & ORC_CTRL_INCLUDE_TRUE) && ((pos_mask >> j) & 1u))
                        continue;
                    int r = score_cmp(m[js], m[j]);
                    counts[3] += (r > 0);
                    counts[4] += (r == 0);
                    counts[5] += 1;
                }
            }
        }
    }

    /* Random baseline: Eq. 5 counts with every score replaced by a uniform. */
    if (baseline && (flags & ORC_AUROC_RANDOM)) {
        for (uint32_t t = 0; t < C; ++t)
            for (uint32_t i = 0; i < S; ++i) {
                if (!((pos_mask >> i) & 1u))
                    continue;
                float ui = orc_random_score(seed, cfg_id, t, i);
                for (uint32_t j = 0; j < S; ++j) {
                    if ((pos_mask >> j) & 1u)
                        continue;
                    int r = score_cmp(ui, orc_random_score(seed, cfg_id, t, j));
                    baseline[0] += (r > 0);
                    baseline[1] += (r == 0);
                    baseline[2] += 1;
                }
            }
    }

    if (pooled && (flags & ORC_AUROC_POOLED)) {
        for (uint32_t tp = 0; tp < C; ++tp)
            for (uint32_t i = 0; i < S; ++i) {
                if (!((pos_mask >> i) & 1u))
                    continue;
                float p = scores[(uint64_t)tp * S + i];
                for (uint32_t tn = 0; tn < C; ++tn)
                    for (uint32_t j = 0; j < S; ++j) {
                        if ((pos_mask >> j) & 1u)
                            continue;
                        int r = score_cmp(p, scores[(uint64_t)tn * S + j]);
                        pooled[0] += (r > 0);
                        pooled[1] += (r == 0);
                        pooled[2] += 1;
                    }
            }
    }
    return 0;
}
