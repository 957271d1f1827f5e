// Drives the argument checks of the C ABI with bad and edge-case arguments
// under AddressSanitizer and UndefinedBehaviorSanitizer on the host side
// (built by tests/test_sanitizers.py; no GPU is touched).  Every call here
// must be rejected, or return at once for an empty shape, before any HIP
// call; the driver exits non-zero if one is accepted.
#include <stdio.h>
#include <string.h>

#include "cdt.h"

static int bad = 0;

static void expect(int got, int want, const char* what) {
    if (got != want) {
        fprintf(stderr, "%s: got %d, want %d (%s)\n", what, got, want, cdt_last_error());
        bad = 1;
    }
}

int main() {
    void* p = reinterpret_cast<void*>(16);   // aligned, never dereferenced
    void* q = reinterpret_cast<void*>(8);    // misaligned
    float* fp = static_cast<float*>(p);
    uint16_t* hp = static_cast<uint16_t*>(p);
    expect(cdt_version(), CDT_INTERFACE_VERSION, "version");
    expect(cdt_outlier_gain(40000, 1, 20.f, 0, 0, fp, nullptr), CDT_ELIMIT, "gain H");
    expect(cdt_outlier_gain(16, 17, 20.f, 0, 0, fp, nullptr), CDT_EINVAL, "gain n_out");
    expect(cdt_ref_synth(2, 2, 3, 12, 0, 0, 0, fp, fp, nullptr), CDT_EINVAL, "synth H%8");
    expect(cdt_ref_synth(2, 3, 3, 16, 0, 0, 0xFFFFFFFEu, fp, fp, nullptr), CDT_ELIMIT, "base");
    expect(cdt_ref_synth(2, 2, 3, 16, 0, 0, 0, static_cast<float*>(q), fp, nullptr), CDT_EALIGN,
           "synth align");
    expect(cdt_ref_synth(2, 0, 3, 16, 0, 0, 0, nullptr, nullptr, nullptr), CDT_OK, "synth empty");
    expect(cdt_ref_stats(2, 2, 3, 16, fp, nullptr, nullptr, p, 1 << 20, nullptr), CDT_EINVAL,
           "stats null");
    expect(cdt_block_scales(4, 2, 8, nullptr, nullptr, 0.1, 0.0, fp, nullptr, nullptr),
           CDT_EINVAL, "scales null");
    cdt_sim_params sp;
    memset(&sp, 0, sizeof(sp));
    sp.sigma_b = 1e-3;
    sp.scale = 1.0;
    sp.cfg_id = 1u << 24;
    expect(cdt_canary_sim(4, 2, 2, 16, &sp, fp, hp, nullptr), CDT_ELIMIT, "sim cfg_id");
    sp.cfg_id = 0;
    sp.carry = 2.0;
    expect(cdt_canary_sim(4, 2, 2, 16, &sp, fp, hp, nullptr), CDT_EINVAL, "sim carry");
    sp.carry = 0.0;
    sp.reserved = 1;
    expect(cdt_canary_sim(4, 2, 2, 16, &sp, fp, hp, nullptr), CDT_EINVAL, "sim reserved");
    sp.reserved = 0;
    expect(cdt_canary_sim(65, 2, 2, 16, &sp, fp, hp, nullptr), CDT_ELIMIT, "sim S");
    expect(cdt_canary_sim(4, 2, 2, 16, nullptr, fp, hp, nullptr), CDT_EINVAL, "sim params");
    expect(cdt_sim_score(4, 2, 2, 16, &sp, fp, nullptr, fp, nullptr, p, 1, nullptr), CDT_EINVAL,
           "fused ws");
    expect(cdt_tamper_scale_exact(4, 2, 2, 16, &sp, fp, -1.0, fp, nullptr, p, 1 << 20, nullptr),
           CDT_EINVAL, "exact eps");
    expect(cdt_drift_score(2, 2, 3, 16, hp, fp, fp, nullptr, p, 15, nullptr), CDT_EINVAL,
           "drift ws");
    expect(cdt_drift_score(2, 2, 1u << 16, 1u << 16, hp, fp, fp, nullptr, p, 1 << 20, nullptr),
           CDT_ELIMIT, "drift T*H");
    expect(cdt_drift_score_f16ref(2, 2, 3, 16, static_cast<uint16_t*>(q), hp, fp, nullptr, p,
                                  1 << 20, nullptr), CDT_EALIGN, "f16ref align");
    expect(cdt_cosine_score(0, 2, 3, 16, nullptr, nullptr, nullptr, nullptr, nullptr, 0, nullptr),
           CDT_OK, "cosine empty");
    expect(cdt_drift_read_stream(2, 2, 3, 16, hp, fp, p, 15, nullptr), CDT_EINVAL, "read ws");
    expect(cdt_drift_read_stream(2, 2, 3, 16, static_cast<uint16_t*>(q), fp, p, 1 << 20, nullptr),
           CDT_EALIGN, "read align");
    expect(cdt_drift_read_stream(2, 2, 0, 16, nullptr, nullptr, nullptr, 0, nullptr), CDT_OK,
           "read empty");
    cdt_auroc_cfg cfgs[2];
    memset(cfgs, 0, sizeof(cfgs));
    cfgs[0].S = 8; cfgs[0].C = 4; cfgs[0].pos_mask = 1;
    cfgs[1].S = 8; cfgs[1].C = 4; cfgs[1].score_off = 30; cfgs[1].pos_mask = 1;
    uint64_t* up = static_cast<uint64_t*>(p);
    expect(cdt_auroc(2, cfgs, fp, 60, 0, 0, up, nullptr, nullptr, p, 64, nullptr), CDT_EINVAL,
           "auroc outside");
    expect(cdt_auroc(2, cfgs, fp, 64, 0, 16, up, nullptr, nullptr, p, 64, nullptr), CDT_EINVAL,
           "auroc flags");
    cfgs[1].S = 65;
    expect(cdt_auroc_upload(2, cfgs, 1000, 0, p, 64, nullptr), CDT_ELIMIT, "upload S");
    expect(cdt_auroc_launch(2, q, fp, 64, 0, 0, up, nullptr, nullptr, nullptr), CDT_EALIGN,
           "launch align");
    expect(cdt_auroc_launch(2, p, fp, 64, 0, 2, up, nullptr, nullptr, nullptr), CDT_EINVAL,
           "launch pooled");
    expect(cdt_drift_score_noalloc(16, 1024, 256, 8192, hp, fp, fp, nullptr, nullptr), CDT_ELIMIT,
           "noalloc scratch");
    expect(cdt_drift_score_noalloc(2, 2, 3, 16, static_cast<uint16_t*>(q), fp, fp, nullptr,
                                   nullptr), CDT_EALIGN, "noalloc align");
    expect(cdt_auroc_values(2, nullptr, nullptr, nullptr, static_cast<double*>(p), nullptr),
           CDT_EINVAL, "values counts");
    expect(cdt_auroc_values((1u << 24) + 1, up, nullptr, nullptr, static_cast<double*>(p),
                            nullptr), CDT_ELIMIT, "values n_cfg");
    sp.carry = 0.5;
    expect(cdt_tamper_scale_exact(65, 2, 2, 16, &sp, fp, 0.1, fp, nullptr, p, 1 << 20, nullptr),
           CDT_ELIMIT, "exact chain S");
    expect(cdt_tamper_scale_exact(4, 2, 2, 16, &sp, fp, 0.1, nullptr, nullptr, p, 1 << 20,
                                  nullptr), CDT_EINVAL, "exact chain tscale");
    sp.carry = 0.0;
    if (cdt_last_error()[0] == '\0') bad = 1;
    return bad;
}
