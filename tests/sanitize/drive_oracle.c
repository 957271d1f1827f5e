/* Drives every oracle routine on small and degenerate shapes under
 * AddressSanitizer and UndefinedBehaviorSanitizer (built by
 * tests/test_sanitizers.py).  Exits 0 when every call returns; any
 * out-of-bounds access, use of freed memory, signed overflow or other
 * undefined behaviour aborts the run with the sanitizer's report. */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

void orc_philox(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4]);
float orc_z16(uint32_t w0, uint32_t w1);
uint16_t orc_f16_rne(float x);
double orc_f16_value(uint16_t bits);
void orc_f16_rne_range(uint64_t start, uint64_t count, uint16_t* out);
int orc_outlier_gain(uint32_t H, uint32_t n_out, float big, uint64_t seed, uint32_t ref_set_id,
                     float* gain);
void orc_ref_synth(uint32_t S, uint32_t C, uint32_t T, uint32_t H, uint64_t seed,
                   uint32_t ref_set_id, const float* gain, float* out);
void orc_ref_stats(uint32_t S, uint32_t C, uint32_t T, uint32_t H, const float* ref,
                   double* sumsq, double* sumabs);
void orc_block_scales(uint64_t nblocks, uint32_t T, uint32_t H, const double* sumsq,
                      const double* sumabs, double eps, double sigma_b, float* tscale,
                      float* bscale);
int orc_canary_sim(uint32_t S, uint32_t C, uint32_t T, uint32_t H, uint64_t seed, uint32_t cfg_id,
                   int benign_mode, int benign_dist, double sigma_b, const float* bscale,
                   uint64_t mal_mask, uint32_t tamper, int tamper_base, const float* tscale,
                   double flip_p, double scale, int redraw, const float* ref, uint16_t* h);
int orc_canary_sim_chain(uint32_t S, uint32_t C, uint32_t T, uint32_t H, uint64_t seed,
                         uint32_t cfg_id, int benign_mode, int benign_dist, double sigma_b,
                         const float* bscale, uint64_t mal_mask, uint32_t tamper,
                         int tamper_base, const float* tscale, double flip_p, double scale,
                         int redraw, double carry, const float* ref, uint16_t* h);
float orc_tamper_scale_exact_block(uint32_t s, uint32_t c, uint32_t T, uint32_t H, uint64_t seed,
                                   uint32_t cfg_id, int benign_mode, int benign_dist,
                                   double sigma_b, float bscale, int tamper_base, int redraw,
                                   double eps, const float* ref, double* vv, double* zz);
void orc_drift_score(uint32_t S, uint32_t C, uint32_t T, uint32_t H, const uint16_t* h,
                     const float* ref, double* score64, float* score32, double* num_den);
void orc_drift_score_f16ref(uint32_t S, uint32_t C, uint32_t T, uint32_t H, const uint16_t* h,
                            const uint16_t* r, double* score64, float* score32);
void orc_cosine_score(uint32_t S, uint32_t C, uint32_t T, uint32_t H, const uint16_t* h,
                      const float* ref, double* score64, float* score32);
double orc_cosine_block_f16ref(uint64_t n, const uint16_t* h, const uint16_t* r);
float orc_random_score(uint64_t seed, uint32_t cfg_id, uint32_t t, uint32_t s);
int orc_scramble_jstar(uint32_t S, uint64_t pos_mask, uint64_t seed, uint32_t cfg_id, uint32_t t);
int orc_auroc_config(uint32_t S, uint32_t C, const float* scores, uint64_t pos_mask,
                     uint64_t seed, uint32_t cfg_id, uint32_t flags, uint64_t* counts,
                     uint64_t* pooled, uint64_t* baseline);

static void* xmalloc(size_t n) { void* p = malloc(n ? n : 1); if (!p) abort(); return p; }

static void one_shape(uint32_t S, uint32_t C, uint32_t T, uint32_t H) {
    size_t n = (size_t)S * C * T * H, nb = (size_t)S * C;
    float* gain = xmalloc(sizeof(float) * H);
    float* ref = xmalloc(sizeof(float) * n);
    uint16_t* h = xmalloc(sizeof(uint16_t) * n);
    uint16_t* r = xmalloc(sizeof(uint16_t) * n);
    double* q = xmalloc(sizeof(double) * nb);
    double* m = xmalloc(sizeof(double) * nb);
    float* ts = xmalloc(sizeof(float) * nb);
    float* bs = xmalloc(sizeof(float) * nb);
    double* s64 = xmalloc(sizeof(double) * nb);
    float* s32 = xmalloc(sizeof(float) * nb);
    double* nd = xmalloc(sizeof(double) * 2 * nb);
    uint64_t mal = S >= 64 ? (1ull << 63) | 1ull : (S > 1 ? 1ull << (S / 2) : 1ull);
    if (orc_outlier_gain(H, H / 8, 20.0f, 7, 1, gain)) abort();
    orc_ref_synth(S, C, T, H, 7, 1, gain, ref);
    orc_ref_stats(S, C, T, H, ref, q, m);
    orc_block_scales(nb, T, H, q, m, 0.05, 1e-2, ts, bs);
    for (int dist = 0; dist < 2; ++dist)
        for (int mode = 0; mode < 2; ++mode) {
            orc_canary_sim(S, C, T, H, 3, 5, mode, dist, 1e-2, bs, mal, 7, 0, ts, 0.3, 1.1, 0,
                           ref, h);
            orc_canary_sim(S, C, T, H, 3, 5, mode, dist, 1e-2, bs, mal, 7, 1, ts, 1.0, 1.1, 1,
                           ref, r);
            orc_canary_sim_chain(S, C, T, H, 3, 5, mode, dist, 1e-2, bs, mal, 7, 0, ts, 0.3,
                                 1.1, 0, 0.7, ref, h);
        }
    if (nb && T * H)
        (void)orc_tamper_scale_exact_block(0, 0, T, H, 3, 5, 1, 1, 1e-2, bs[0], 0, 0, 0.05, ref,
                                           NULL, NULL);
    orc_drift_score(S, C, T, H, h, ref, s64, s32, nd);
    orc_drift_score_f16ref(S, C, T, H, h, r, s64, s32);
    orc_cosine_score(S, C, T, H, h, ref, s64, s32);
    if (nb && T * H) (void)orc_cosine_block_f16ref((uint64_t)T * H, h, r);
    if (S <= 64) {
        uint64_t counts[6], pooled[3], base[3];
        for (uint32_t flags = 0; flags < 16; ++flags)
            if (orc_auroc_config(S, C, s32, mal, 3, 5, flags, counts, pooled, base)) abort();
    }
    free(gain); free(ref); free(h); free(r); free(q); free(m); free(ts); free(bs);
    free(s64); free(s32); free(nd);
}

int main(void) {
    uint32_t ctr[4] = {1, 2, 3, 4}, key[2] = {5, 6}, out[4];
    orc_philox(ctr, key, out);
    (void)orc_z16(0, 0); (void)orc_z16(0xFFFFFFFFu, 0xFFFFFFFFu);
    const float specials[] = {0.0f, -0.0f, INFINITY, -INFINITY, NAN, 65504.0f, 65520.0f, 1e30f,
                              5.96e-8f, 1e-45f, -3.0e-5f};
    for (size_t i = 0; i < sizeof(specials) / sizeof(specials[0]); ++i)
        (void)orc_f16_value(orc_f16_rne(specials[i]));
    uint16_t buf[4096];
    orc_f16_rne_range(0x7F7FF000u, 4096, buf);
    orc_f16_rne_range(0xFFFFF000u, 4096, buf);
    for (uint32_t b = 0; b < 65536; ++b) (void)orc_f16_value((uint16_t)b);
    (void)orc_random_score(1, 2, 3, 4);
    (void)orc_scramble_jstar(8, 0xFF, 1, 2, 3);   /* no benign stage */
    (void)orc_scramble_jstar(64, 1, 1, 2, 3);
    /* shapes: ordinary, ragged, single element rows, empty, S = 64 */
    one_shape(4, 3, 5, 16);
    one_shape(3, 2, 1, 8);
    one_shape(2, 0, 4, 8);
    one_shape(2, 2, 0, 8);
    one_shape(64, 2, 2, 8);
    return 0;
}
