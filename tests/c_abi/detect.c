/* The detector driven from C through include/cdt.h alone: device buffers
 * from hipMalloc, one stream, no Python.  Synthetic references, a live pass
 * with a Gaussian tamper on the middle shard, Eq. 4 scores and the Eqs. 5-6
 * counts with the scrambled-label control, printed for the test that runs
 * this program (tests/test_gpu_c_abi.py) to compare with the oracle.
 *
 * Usage: detect S C T H seed eps sigma_b
 * Output: "scores" and C*S fp32 scores in [C][S] order (%.9g), then
 *         "counts" and the six counts.  Exit status 0 on success. */
#include <hip/hip_runtime_api.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "cdt.h"

#define HIP_OK(x)                                                               \
    do {                                                                        \
        hipError_t e_ = (x);                                                    \
        if (e_ != hipSuccess) {                                                 \
            fprintf(stderr, "%s: %s\n", #x, hipGetErrorString(e_));             \
            return 2;                                                           \
        }                                                                       \
    } while (0)
#define CDT_OK_(x)                                                              \
    do {                                                                        \
        int r_ = (x);                                                           \
        if (r_ != CDT_OK) {                                                     \
            fprintf(stderr, "%s: [%d] %s\n", #x, r_, cdt_last_error());         \
            return 3;                                                           \
        }                                                                       \
    } while (0)

int main(int argc, char** argv) {
    if (argc != 8) {
        fprintf(stderr, "usage: detect S C T H seed eps sigma_b\n");
        return 1;
    }
    const uint32_t S = (uint32_t)atoi(argv[1]), C = (uint32_t)atoi(argv[2]);
    const uint32_t T = (uint32_t)atoi(argv[3]), H = (uint32_t)atoi(argv[4]);
    const uint64_t seed = strtoull(argv[5], NULL, 10);
    const double eps = atof(argv[6]), sigma_b = atof(argv[7]);
    if (cdt_version() != CDT_INTERFACE_VERSION) {
        fprintf(stderr, "libcdt interface version %d, this header declares %d\n", cdt_version(),
                CDT_INTERFACE_VERSION);
        return 1;
    }
    const size_t n = (size_t)S * C * T * H, nb = (size_t)S * C;
    const uint64_t mal = 1ull << (S / 2);
    hipStream_t st;
    HIP_OK(hipStreamCreate(&st));
    float *gain, *ref, *tscale, *score;
    uint16_t* h;
    double *sumsq, *sumabs;
    void *ws, *auroc_ws;
    uint64_t* counts;
    const size_t ws_bytes = cdt_reduce_workspace_bytes(S, C, T, H) + 16;
    const size_t auroc_bytes = cdt_auroc_workspace_bytes(1) + 16;
    HIP_OK(hipMalloc((void**)&gain, sizeof(float) * H));
    HIP_OK(hipMalloc((void**)&ref, sizeof(float) * n));
    HIP_OK(hipMalloc((void**)&h, sizeof(uint16_t) * n));
    HIP_OK(hipMalloc((void**)&tscale, sizeof(float) * nb));
    HIP_OK(hipMalloc((void**)&score, sizeof(float) * nb));
    HIP_OK(hipMalloc((void**)&sumsq, sizeof(double) * nb));
    HIP_OK(hipMalloc((void**)&sumabs, sizeof(double) * nb));
    HIP_OK(hipMalloc(&ws, ws_bytes));
    HIP_OK(hipMalloc(&auroc_ws, auroc_bytes));
    HIP_OK(hipMalloc((void**)&counts, sizeof(uint64_t) * 6));

    CDT_OK_(cdt_outlier_gain(H, (uint32_t)(0.01 * H + 0.5), 20.0f, seed, 0, gain, st));
    CDT_OK_(cdt_ref_synth(S, C, T, H, seed, 0, 0, gain, ref, st));
    CDT_OK_(cdt_ref_stats(S, C, T, H, ref, sumsq, sumabs, ws, ws_bytes, st));
    CDT_OK_(cdt_block_scales(nb, T, H, sumsq, sumabs, eps, 0.0, tscale, NULL, st));
    cdt_sim_params p;
    memset(&p, 0, sizeof(p));
    p.seed = seed;
    p.cfg_id = 1;
    p.benign_mode = CDT_NOISE_ELEMENTWISE;
    p.benign_dist = CDT_DIST_GAUSS;
    p.tamper = CDT_T_ADD;
    p.tamper_base = CDT_BASE_BENIGN;
    p.mal_mask = mal;
    p.sigma_b = sigma_b;
    p.scale = 1.0;
    p.tscale = tscale;
    CDT_OK_(cdt_canary_sim(S, C, T, H, &p, ref, h, st));
    CDT_OK_(cdt_drift_score(S, C, T, H, h, ref, score, NULL, ws, ws_bytes, st));
    cdt_auroc_cfg cfg;
    memset(&cfg, 0, sizeof(cfg));
    cfg.S = S;
    cfg.C = C;
    cfg.pos_mask = mal;
    cfg.cfg_id = 1;
    CDT_OK_(cdt_auroc(1, &cfg, score, nb, seed, CDT_AUROC_CONTROL, counts, NULL, NULL, auroc_ws,
                      auroc_bytes, st));

    float* score_h = (float*)malloc(sizeof(float) * nb);
    uint64_t counts_h[6];
    HIP_OK(hipMemcpyAsync(score_h, score, sizeof(float) * nb, hipMemcpyDeviceToHost, st));
    HIP_OK(hipMemcpyAsync(counts_h, counts, sizeof(counts_h), hipMemcpyDeviceToHost, st));
    HIP_OK(hipStreamSynchronize(st));
    printf("scores");
    for (size_t i = 0; i < nb; ++i) printf(" %.9g", score_h[i]);
    printf("\ncounts");
    for (int i = 0; i < 6; ++i) printf(" %llu", (unsigned long long)counts_h[i]);
    printf("\n");
    free(score_h);
    hipFree(gain); hipFree(ref); hipFree(h); hipFree(tscale); hipFree(score);
    hipFree(sumsq); hipFree(sumabs); hipFree(ws); hipFree(auroc_ws); hipFree(counts);
    HIP_OK(hipStreamDestroy(st));
    return 0;
}
