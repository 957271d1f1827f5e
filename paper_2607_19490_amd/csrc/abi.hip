// C ABI of libcdt: argument validation, workspace sizing, launches and
// error reporting.  Every check runs on the host before any HIP call, so a
// rejected call touches no device state.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <mutex>
#include <vector>

#include "cdt.h"
#include "cdt_launch.hpp"
#include "cdt_rank.hpp"

namespace {

thread_local char g_error[512] = "";

int fail(int code, const char* fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_error, sizeof(g_error), fmt, ap);
    va_end(ap);
    return code;
}

int ok() {
    g_error[0] = '\0';
    return CDT_OK;
}

int device_status(hipError_t e, const char* what) {
    if (e != hipSuccess) return fail(CDT_EDEVICE, "%s: %s", what, hipGetErrorString(e));
    return ok();
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

constexpr uint64_t kMaxBlockElems = 1ull << 32;  // element index e must fit 32 bits
constexpr uint64_t kMaxBlocks = 1ull << 32;      // (shard, canary) blocks per call
constexpr uint64_t kMaxElems = 1ull << 40;       // elements per call
constexpr uint32_t kMaxId = 1u << 24;            // counter id field
constexpr uint32_t kMaxOutlierH = 32768;
constexpr uint32_t kMaxPooled = 16384;

// Shape checks common to every activation call.  Beyond the per-block limit,
// the block count must fit 32 bits and the whole array 2^40 elements (4 TiB
// of fp32, far beyond one device), so that every size derived from the
// shape (workspace bytes, grids, offsets) is exact in 64 bits.
int check_shape(const char* fn, uint32_t S, uint32_t C, uint32_t T, uint32_t H) {
    if (H % 8 != 0) return fail(CDT_EINVAL, "%s: H=%u must be a multiple of 8", fn, H);
    const uint64_t n = static_cast<uint64_t>(T) * H;
    if (n >= kMaxBlockElems)
        return fail(CDT_ELIMIT, "%s: T*H=%llu must be below 2^32", fn,
                    static_cast<unsigned long long>(n));
    const uint64_t nblocks = static_cast<uint64_t>(S) * C;
    if (nblocks > kMaxBlocks)
        return fail(CDT_ELIMIT, "%s: S*C=%llu above 2^32", fn,
                    static_cast<unsigned long long>(nblocks));
    if (n > 0 && nblocks > kMaxElems / n)
        return fail(CDT_ELIMIT, "%s: S*C*T*H above 2^40", fn);
    return CDT_OK;
}

bool empty(uint32_t S, uint32_t C, uint32_t T, uint32_t H) {
    return static_cast<uint64_t>(S) * C * T * H == 0;
}

// Global canary indices canary_base .. canary_base + C - 1 fit the 32-bit
// counter word.
bool canaries_fit(uint32_t canary_base, uint64_t C) {
    return static_cast<uint64_t>(canary_base) + C <= (1ull << 32);
}

}  // namespace

extern "C" {

int cdt_version(void) { return 11; }

const char* cdt_last_error(void) { return g_error; }

int cdt_outlier_gain(uint32_t H, uint32_t n_out, float big, uint64_t seed, uint32_t ref_set_id,
                     float* gain, void* stream) {
    if (H > kMaxOutlierH) return fail(CDT_ELIMIT, "cdt_outlier_gain: H=%u above %u", H, kMaxOutlierH);
    if (n_out > H) return fail(CDT_EINVAL, "cdt_outlier_gain: n_out=%u above H=%u", n_out, H);
    if (ref_set_id >= kMaxId) return fail(CDT_ELIMIT, "cdt_outlier_gain: ref_set_id >= 2^24");
    if (!isfinite(big)) return fail(CDT_EINVAL, "cdt_outlier_gain: gain must be finite");
    if (H == 0) return ok();
    if (!gain) return fail(CDT_EINVAL, "cdt_outlier_gain: gain is NULL");
    return device_status(cdt::launch_outlier_gain(H, n_out, big, seed, ref_set_id, gain,
                                                  static_cast<hipStream_t>(stream)),
                         "cdt_outlier_gain");
}

int cdt_ref_synth(uint32_t S, uint32_t C, uint32_t T, uint32_t H, uint64_t seed,
                  uint32_t ref_set_id, uint32_t canary_base, const float* gain, float* ref,
                  void* stream) {
    int rc = check_shape("cdt_ref_synth", S, C, T, H);
    if (rc) return rc;
    if (ref_set_id >= kMaxId) return fail(CDT_ELIMIT, "cdt_ref_synth: ref_set_id >= 2^24");
    if (!canaries_fit(canary_base, C))
        return fail(CDT_ELIMIT, "cdt_ref_synth: canary_base + C above 2^32");
    if (empty(S, C, T, H)) return ok();
    if (!gain || !ref) return fail(CDT_EINVAL, "cdt_ref_synth: NULL array");
    if (!aligned16(gain) || !aligned16(ref))
        return fail(CDT_EALIGN, "cdt_ref_synth: arrays must be 16-byte aligned");
    return device_status(cdt::launch_ref_synth(S, C, T, H, seed, ref_set_id, canary_base, gain,
                                               ref, static_cast<hipStream_t>(stream)),
                         "cdt_ref_synth");
}

size_t cdt_reduce_workspace_bytes(uint32_t S, uint32_t C, uint32_t T, uint32_t H) {
    const uint64_t n = static_cast<uint64_t>(T) * H;
    const uint64_t cpb = cdt::reduce_chunks_per_block(n);
    return static_cast<size_t>(cpb * S * C * cdt::kReduceMaxSums * sizeof(double));
}

int cdt_ref_stats(uint32_t S, uint32_t C, uint32_t T, uint32_t H, const float* ref,
                  double* sumsq, double* sumabs, void* ws, size_t ws_bytes, void* stream) {
    int rc = check_shape("cdt_ref_stats", S, C, T, H);
    if (rc) return rc;
    if (static_cast<uint64_t>(S) * C == 0) return ok();
    if (!sumsq || !sumabs) return fail(CDT_EINVAL, "cdt_ref_stats: NULL output");
    const size_t need = cdt_reduce_workspace_bytes(S, C, T, H);
    if (static_cast<uint64_t>(T) * H > 0) {
        if (!ref) return fail(CDT_EINVAL, "cdt_ref_stats: ref is NULL");
        if (!aligned16(ref)) return fail(CDT_EALIGN, "cdt_ref_stats: ref must be 16-byte aligned");
    }
    if (need > 0 && (!ws || ws_bytes < need))
        return fail(CDT_EINVAL, "cdt_ref_stats: workspace of %zu bytes needed, %zu given", need,
                    ws ? ws_bytes : 0);
    if (ws && !aligned16(ws)) return fail(CDT_EALIGN, "cdt_ref_stats: ws must be 16-byte aligned");
    return device_status(cdt::launch_ref_stats(S, C, T, H, ref, sumsq, sumabs, ws,
                                               static_cast<hipStream_t>(stream)),
                         "cdt_ref_stats");
}

int cdt_block_scales(uint64_t nblocks, uint32_t T, uint32_t H, const double* sumsq,
                     const double* sumabs, double eps, double sigma_b, float* tscale,
                     float* bscale, void* stream) {
    if (!(eps >= 0.0) || !isfinite(eps) || !(sigma_b >= 0.0) || !isfinite(sigma_b))
        return fail(CDT_EINVAL, "cdt_block_scales: eps and sigma_b must be finite and >= 0");
    if (nblocks == 0 || (!tscale && !bscale)) return ok();
    if (tscale && !sumsq) return fail(CDT_EINVAL, "cdt_block_scales: tscale needs sumsq");
    if (bscale && !sumabs) return fail(CDT_EINVAL, "cdt_block_scales: bscale needs sumabs");
    if (nblocks > (1ull << 40)) return fail(CDT_ELIMIT, "cdt_block_scales: too many blocks");
    return device_status(cdt::launch_block_scales(nblocks, T, H, sumsq, sumabs, eps, sigma_b,
                                                  tscale, bscale,
                                                  static_cast<hipStream_t>(stream)),
                         "cdt_block_scales");
}

namespace {

// Validation of the live-pass parameters shared by cdt_canary_sim and
// cdt_sim_score; fills the launch description on success.
int check_sim(const char* fn, uint32_t S, uint32_t C, uint32_t T, uint32_t H,
              const cdt_sim_params* p, cdt::SimLaunch* L) {
    int rc = check_shape(fn, S, C, T, H);
    if (rc) return rc;
    if (!p) return fail(CDT_EINVAL, "%s: params is NULL", fn);
    if (S > 64) return fail(CDT_ELIMIT, "%s: S=%u above 64", fn, S);
    if (p->cfg_id >= kMaxId) return fail(CDT_ELIMIT, "%s: cfg_id >= 2^24", fn);
    if (p->benign_mode > CDT_NOISE_BLOCK) return fail(CDT_EINVAL, "%s: bad benign_mode", fn);
    if (p->benign_dist > CDT_DIST_T3) return fail(CDT_EINVAL, "%s: bad benign_dist", fn);
    if (p->tamper & ~7u) return fail(CDT_EINVAL, "%s: bad tamper flags", fn);
    if (p->tamper_base > CDT_BASE_CLEAN) return fail(CDT_EINVAL, "%s: bad tamper_base", fn);
    if (p->redraw > 1) return fail(CDT_EINVAL, "%s: redraw must be 0 or 1", fn);
    if (!(p->sigma_b >= 0.0) || !isfinite(p->sigma_b))
        return fail(CDT_EINVAL, "%s: sigma_b must be finite and >= 0", fn);
    if (!(p->flip_p >= 0.0 && p->flip_p <= 1.0))
        return fail(CDT_EINVAL, "%s: flip_p must lie in [0, 1]", fn);
    if (!isfinite(p->scale)) return fail(CDT_EINVAL, "%s: scale must be finite", fn);
    if (!(p->carry >= 0.0 && p->carry <= 1.0))
        return fail(CDT_EINVAL, "%s: carry must lie in [0, 1]", fn);
    if (p->reserved != 0) return fail(CDT_EINVAL, "%s: reserved must be 0", fn);
    if (!canaries_fit(p->canary_base, C))
        return fail(CDT_ELIMIT, "%s: canary_base + C above 2^32", fn);
    const uint64_t mal = p->mal_mask & (S >= 64 ? ~0ull : ((1ull << S) - 1ull));
    if (!empty(S, C, T, H)) {
        if (p->benign_mode == CDT_NOISE_BLOCK && !p->bscale)
            return fail(CDT_EINVAL, "%s: BLOCK noise needs bscale", fn);
        if (mal && (p->tamper & CDT_T_ADD) && !p->tscale)
            return fail(CDT_EINVAL, "%s: Gaussian tamper needs tscale", fn);
    }
    L->S = S;
    L->C = C;
    L->T = T;
    L->H = H;
    L->seed = p->seed;
    L->cfg_id = p->cfg_id;
    L->benign_mode = p->benign_mode;
    L->benign_dist = p->benign_dist;
    L->tamper = p->tamper;
    L->tamper_base = p->tamper_base;
    L->redraw = p->redraw;
    L->mal_mask = mal;
    L->sigma_b = static_cast<float>(p->sigma_b);
    // Flip selection: u < floor(p 2^32) with p < 1 (so the threshold fits 32
    // bits); p == 1 flips every element.
    L->flip_all = p->flip_p >= 1.0;
    L->flip_thr = L->flip_all ? 0u : static_cast<uint32_t>(floor(p->flip_p * 4294967296.0));
    L->scale = static_cast<float>(p->scale);
    L->carry = static_cast<float>(p->carry);
    L->canary_base = p->canary_base;
    L->bscale = p->bscale;
    L->tscale = p->tscale;
    return CDT_OK;
}

}  // namespace

int cdt_canary_sim(uint32_t S, uint32_t C, uint32_t T, uint32_t H, const cdt_sim_params* p,
                   const float* ref, uint16_t* h, void* stream) {
    cdt::SimLaunch L;
    int rc = check_sim("cdt_canary_sim", S, C, T, H, p, &L);
    if (rc) return rc;
    if (empty(S, C, T, H)) return ok();
    if (!ref || !h) return fail(CDT_EINVAL, "cdt_canary_sim: NULL array");
    if (!aligned16(ref) || !aligned16(h))
        return fail(CDT_EALIGN, "cdt_canary_sim: arrays must be 16-byte aligned");
    return device_status(cdt::launch_canary_sim(L, ref, h, static_cast<hipStream_t>(stream)),
                         "cdt_canary_sim");
}

size_t cdt_sim_batch_workspace_bytes(uint32_t n_jobs) {
    return (cdt::sim_batch_table_bytes(n_jobs) + 255) & ~static_cast<size_t>(255);
}

int cdt_canary_sim_batch(uint32_t n_jobs, const cdt_sim_job* jobs, void* ws, size_t ws_bytes,
                         void* stream) {
    const char* fn = "cdt_canary_sim_batch";
    if (n_jobs == 0) return ok();
    if (n_jobs > (1u << 16)) return fail(CDT_ELIMIT, "%s: n_jobs above 65536", fn);
    if (!jobs) return fail(CDT_EINVAL, "%s: NULL jobs", fn);
    std::vector<cdt::SimLaunch> runs(n_jobs);
    std::vector<const float*> refs(n_jobs);
    std::vector<uint16_t*> hs(n_jobs);
    int dist = -1, mode = -1;
    for (uint32_t j = 0; j < n_jobs; ++j) {
        const cdt_sim_job& J = jobs[j];
        int rc = check_sim(fn, J.S, J.C, J.T, J.H, J.p, &runs[j]);
        if (rc) return rc;
        if (runs[j].carry != 0.0f)
            return fail(CDT_EINVAL, "%s: job %u: the propagation model (carry > 0) runs "
                                    "through cdt_canary_sim", fn, j);
        if (empty(J.S, J.C, J.T, J.H)) continue;
        if (dist < 0) {
            dist = static_cast<int>(runs[j].benign_dist);
            mode = static_cast<int>(runs[j].benign_mode);
        } else if (dist != static_cast<int>(runs[j].benign_dist) ||
                   mode != static_cast<int>(runs[j].benign_mode)) {
            return fail(CDT_EINVAL, "%s: job %u: every job must use the same benign noise "
                                    "distribution and mode", fn, j);
        }
        if (!J.ref || !J.h) return fail(CDT_EINVAL, "%s: job %u has a NULL array", fn, j);
        if (!aligned16(J.ref) || !aligned16(J.h))
            return fail(CDT_EALIGN, "%s: job %u arrays must be 16-byte aligned", fn, j);
        refs[j] = J.ref;
        hs[j] = J.h;
    }
    if (dist < 0) return ok();
    const size_t need = cdt_sim_batch_workspace_bytes(n_jobs);
    if (!ws || ws_bytes < need)
        return fail(CDT_EINVAL, "%s: workspace of %zu bytes needed, %zu given", fn, need,
                    ws ? ws_bytes : 0);
    if (!aligned16(ws)) return fail(CDT_EALIGN, "%s: ws must be 16-byte aligned", fn);
    return device_status(cdt::launch_canary_sim_batch(n_jobs, runs.data(), refs.data(), hs.data(),
                                                      ws, static_cast<hipStream_t>(stream)),
                         fn);
}

int cdt_canary_sim_stream(uint32_t S, uint32_t C, uint32_t T, uint32_t H, const float* ref,
                          uint16_t* h, void* stream) {
    const char* fn = "cdt_canary_sim_stream";
    int rc = check_shape(fn, S, C, T, H);
    if (rc) return rc;
    if (empty(S, C, T, H)) return ok();
    if (!ref || !h) return fail(CDT_EINVAL, "%s: NULL array", fn);
    if (!aligned16(ref) || !aligned16(h))
        return fail(CDT_EALIGN, "%s: arrays must be 16-byte aligned", fn);
    return device_status(cdt::launch_canary_sim_stream(S, C, T, H, ref, h,
                                                       static_cast<hipStream_t>(stream)),
                         fn);
}

int cdt_sim_score(uint32_t S, uint32_t C, uint32_t T, uint32_t H, const cdt_sim_params* p,
                  const float* ref, uint16_t* h, float* score, double* num_den, void* ws,
                  size_t ws_bytes, void* stream) {
    cdt::SimLaunch L;
    int rc = check_sim("cdt_sim_score", S, C, T, H, p, &L);
    if (rc) return rc;
    if (L.carry != 0.0f)
        return fail(CDT_EINVAL, "cdt_sim_score: the propagation model (carry > 0) needs "
                                "cdt_canary_sim then cdt_drift_score");
    if (static_cast<uint64_t>(S) * C == 0) return ok();
    if (!score) return fail(CDT_EINVAL, "cdt_sim_score: score is NULL");
    if (static_cast<uint64_t>(T) * H > 0) {
        if (!ref) return fail(CDT_EINVAL, "cdt_sim_score: ref is NULL");
        if (!aligned16(ref) || (h && !aligned16(h)))
            return fail(CDT_EALIGN, "cdt_sim_score: arrays must be 16-byte aligned");
    }
    const size_t need = cdt_reduce_workspace_bytes(S, C, T, H);
    if (need > 0 && (!ws || ws_bytes < need))
        return fail(CDT_EINVAL, "cdt_sim_score: workspace of %zu bytes needed, %zu given", need,
                    ws ? ws_bytes : 0);
    if (ws && !aligned16(ws)) return fail(CDT_EALIGN, "cdt_sim_score: ws must be 16-byte aligned");
    return device_status(cdt::launch_sim_score(L, ref, h, score, num_den, ws,
                                               static_cast<hipStream_t>(stream)),
                         "cdt_sim_score");
}

int cdt_tamper_scale_exact(uint32_t S, uint32_t C, uint32_t T, uint32_t H,
                           const cdt_sim_params* p, const float* ref, double eps, float* tscale,
                           double* norms, void* ws, size_t ws_bytes, void* stream) {
    const char* fn = "cdt_tamper_scale_exact";
    if (!p) return fail(CDT_EINVAL, "%s: params is NULL", fn);
    if (!(eps >= 0.0) || !isfinite(eps)) return fail(CDT_EINVAL, "%s: eps must be finite and >= 0", fn);
    // Independent stages: the tamper settings do not enter the norms.  Under
    // the propagation model they shape the earlier malicious stages, whose
    // Gaussian scales are the ones this call writes first (tscale).
    const bool chain = p->carry != 0.0;
    cdt_sim_params q = *p;
    if (chain) {
        q.tscale = tscale;
    } else {
        q.tamper = 0;
        q.tscale = nullptr;
    }
    cdt::SimLaunch L;
    int rc = check_sim(fn, S, C, T, H, &q, &L);
    if (rc) return rc;
    if (static_cast<uint64_t>(S) * C == 0) return ok();
    if (!tscale) return fail(CDT_EINVAL, "%s: tscale is NULL", fn);
    if (static_cast<uint64_t>(T) * H > 0) {
        if (!ref) return fail(CDT_EINVAL, "%s: ref is NULL", fn);
        if (!aligned16(ref)) return fail(CDT_EALIGN, "%s: ref must be 16-byte aligned", fn);
    }
    const size_t need = cdt_reduce_workspace_bytes(S, C, T, H);
    if (need > 0 && (!ws || ws_bytes < need))
        return fail(CDT_EINVAL, "%s: workspace of %zu bytes needed, %zu given", fn, need,
                    ws ? ws_bytes : 0);
    if (ws && !aligned16(ws)) return fail(CDT_EALIGN, "%s: ws must be 16-byte aligned", fn);
    if (chain)
        return device_status(cdt::launch_tamper_scale_exact_chain(
                                 L, ref, eps, tscale, norms, ws, static_cast<hipStream_t>(stream)),
                             fn);
    return device_status(cdt::launch_tamper_scale_exact(L, ref, eps, tscale, norms, ws,
                                                        static_cast<hipStream_t>(stream)),
                         fn);
}

namespace {

int drift_common(const char* fn, cdt::DriftMetric metric, uint32_t S, uint32_t C, uint32_t T,
                 uint32_t H, const uint16_t* h, const void* ref, float* score, double* sums,
                 void* ws, size_t ws_bytes, void* stream) {
    int rc = check_shape(fn, S, C, T, H);
    if (rc) return rc;
    if (static_cast<uint64_t>(S) * C == 0) return ok();
    if (!score) return fail(CDT_EINVAL, "%s: score is NULL", fn);
    if (static_cast<uint64_t>(T) * H > 0) {
        if (!h || !ref) return fail(CDT_EINVAL, "%s: NULL array", fn);
        if (!aligned16(h) || !aligned16(ref))
            return fail(CDT_EALIGN, "%s: arrays must be 16-byte aligned", fn);
    }
    const size_t need = cdt_reduce_workspace_bytes(S, C, T, H);
    if (need > 0 && (!ws || ws_bytes < need))
        return fail(CDT_EINVAL, "%s: workspace of %zu bytes needed, %zu given", fn, need,
                    ws ? ws_bytes : 0);
    if (ws && !aligned16(ws)) return fail(CDT_EALIGN, "%s: ws must be 16-byte aligned", fn);
    return device_status(cdt::launch_drift(metric, S, C, T, H, h, ref, score, sums, ws,
                                           static_cast<hipStream_t>(stream)),
                         fn);
}

}  // namespace

int cdt_drift_score(uint32_t S, uint32_t C, uint32_t T, uint32_t H, const uint16_t* h,
                    const float* ref, float* score, double* num_den, void* ws, size_t ws_bytes,
                    void* stream) {
    return drift_common("cdt_drift_score", cdt::DriftMetric::kL2, S, C, T, H, h, ref, score,
                        num_den, ws, ws_bytes, stream);
}

}  // extern "C"

// ---------------------------------------------------------------------------
// cdt_drift_score_noalloc: Eq. 4 with its per-chunk partial sums in a fixed
// array of the library's own device memory, for callers that cannot
// allocate.  Each GPU the library runs on holds its own copy of `scratch`
// until the process ends.  In host code `scratch` names a host-side stand-in,
// not device memory: its device address is looked up once per device, with
// that device current, and only that address is ever passed to a kernel.
// ---------------------------------------------------------------------------
static __device__ __align__(256) double scratch[CDT_NOALLOC_SCRATCH_BYTES / sizeof(double)];

namespace {

constexpr int kMaxScratchDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxScratchDevices] = {};

// Device address of the current device's `scratch` (looked up on its first
// use on that device).  The kernels run on `stream`'s device, so a stream of
// another device is refused: its kernels would reach into this device's
// array.
int scratch_of_current_device(const char* fn, hipStream_t stream, void** out) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return device_status(e, fn);
    if (dev < 0 || dev >= kMaxScratchDevices)
        return fail(CDT_ELIMIT, "%s: device %d beyond the %d the library serves", fn, dev,
                    kMaxScratchDevices);
    if (stream != nullptr && stream != hipStreamLegacy && stream != hipStreamPerThread) {
        hipDevice_t sdev = -1;
        e = hipStreamGetDevice(stream, &sdev);
        if (e != hipSuccess) return device_status(e, fn);
        if (sdev != dev)
            return fail(CDT_EINVAL, "%s: stream of device %d while device %d is current", fn,
                        static_cast<int>(sdev), dev);
    }
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return device_status(e, fn);
        if (!p) return fail(CDT_EDEVICE, "%s: no device address for the scratch array", fn);
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return CDT_OK;
}

}  // namespace

extern "C" {

int cdt_drift_score_noalloc(uint32_t S, uint32_t C, uint32_t T, uint32_t H, const uint16_t* h,
                            const float* ref, float* score, double* num_den, void* stream) {
    const char* fn = "cdt_drift_score_noalloc";
    int rc = check_shape(fn, S, C, T, H);
    if (rc) return rc;
    if (static_cast<uint64_t>(S) * C == 0) return ok();
    // Scratch in use: one (D, R) fp64 pair per chunk when a block spans
    // several chunks; a block of one chunk is scored directly.
    const uint64_t n = static_cast<uint64_t>(T) * H;
    const uint64_t cpb = cdt::reduce_chunks_per_block(n);
    const uint64_t need = cpb > 1 ? cpb * S * C * 2 * sizeof(double) : 0;
    if (need > CDT_NOALLOC_SCRATCH_BYTES)
        return fail(CDT_ELIMIT, "%s: this shape needs %llu bytes of scratch, above the %u the "
                                "library holds; use cdt_drift_score with a workspace", fn,
                    static_cast<unsigned long long>(need), CDT_NOALLOC_SCRATCH_BYTES);
    if (!score) return fail(CDT_EINVAL, "%s: score is NULL", fn);
    if (n > 0) {
        if (!h || !ref) return fail(CDT_EINVAL, "%s: NULL array", fn);
        if (!aligned16(h) || !aligned16(ref))
            return fail(CDT_EALIGN, "%s: arrays must be 16-byte aligned", fn);
    }
    void* ws = nullptr;
    rc = scratch_of_current_device(fn, static_cast<hipStream_t>(stream), &ws);
    if (rc) return rc;
    return device_status(cdt::launch_drift(cdt::DriftMetric::kL2, S, C, T, H, h, ref, score,
                                           num_den, ws, static_cast<hipStream_t>(stream)),
                         fn);
}

}  // extern "C"

namespace {

constexpr uint32_t kMaxDriftJobs = 1u << 16;

size_t align256(size_t x) { return (x + 255) & ~static_cast<size_t>(255); }

// Device table of a batched Eq. 4 launch (jobs with no block dropped), the
// partial sums laid out one job after another behind it in the workspace.
struct DriftBatchPlan {
    std::vector<cdt::DriftJobDev> table;
    std::vector<cdt::BatchGroupDev> groups;
    uint64_t total_iters = 0, total_blocks = 0, partial_doubles = 0;
};

// Shapes only (no pointers): what cdt_drift_batch_workspace_bytes sizes.
int plan_drift_batch(const char* fn, uint32_t n_jobs, const cdt_drift_job* jobs,
                     DriftBatchPlan* plan, bool check_arrays) {
    if (n_jobs > kMaxDriftJobs) return fail(CDT_ELIMIT, "%s: n_jobs above %u", fn, kMaxDriftJobs);
    if (n_jobs > 0 && !jobs) return fail(CDT_EINVAL, "%s: NULL jobs", fn);
    for (uint32_t j = 0; j < n_jobs; ++j) {
        const cdt_drift_job& J = jobs[j];
        int rc = check_shape(fn, J.S, J.C, J.T, J.H);
        if (rc) return rc;
        const uint64_t nb = static_cast<uint64_t>(J.S) * J.C;
        if (nb == 0) continue;  // nothing to score
        const uint64_t n = static_cast<uint64_t>(J.T) * J.H;
        if (check_arrays) {
            if (!J.score) return fail(CDT_EINVAL, "%s: job %u has a NULL score", fn, j);
            if (n > 0) {
                if (!J.h || !J.ref) return fail(CDT_EINVAL, "%s: job %u has a NULL array", fn, j);
                if (!aligned16(J.h) || !aligned16(J.ref))
                    return fail(CDT_EALIGN, "%s: job %u arrays must be 16-byte aligned", fn, j);
            }
        }
        cdt::DriftJobDev d{};
        d.h = J.h;
        d.ref = J.ref;
        d.score = J.score;
        d.sums = J.num_den;
        d.cpb = cdt::reduce_chunks_per_block(n);
        d.block_begin = plan->total_blocks;
        d.n8 = static_cast<uint32_t>(n / 8);
        d.S = J.S;
        d.C = J.C;
        d.direct = d.cpb == 1;
        const uint64_t chunks = d.cpb * nb;
        if (!d.direct) {
            d.partial = reinterpret_cast<double*>(static_cast<uintptr_t>(plan->partial_doubles));
            plan->partial_doubles += chunks * 2;
        }
        plan->total_blocks += nb;
        plan->table.push_back(d);
    }
    // jobs in a row over one reference array in one layout share its chunks
    // (BatchGroupDev)
    const uint32_t nt = static_cast<uint32_t>(plan->table.size());
    std::vector<cdt::BatchKey> keys(nt);
    for (uint32_t j = 0; j < nt; ++j) {
        const cdt::DriftJobDev& d = plan->table[j];
        keys[j] = cdt::BatchKey{d.ref, d.cpb * d.S * d.C, d.S, d.C, d.n8};
    }
    plan->groups.resize(nt);
    uint32_t ng = 0;
    plan->total_iters = cdt::plan_batch_groups(nt, keys.data(),
                                               cdt::kDriftJobsPerIter, cdt::kDriftJobMajorFrom,
                                               plan->groups.data(), &ng);
    plan->groups.resize(ng);
    if (plan->total_blocks > kMaxBlocks * 16)
        return fail(CDT_ELIMIT, "%s: the batch holds too many blocks", fn);
    return CDT_OK;
}

// Workspace: the job table, the group table, then the partial sums.
size_t batch_groups_offset(const DriftBatchPlan& plan) {
    return align256(plan.table.size() * sizeof(cdt::DriftJobDev));
}

// (room for one group per job, so that the size depends on the shapes only)
size_t batch_partials_offset(const DriftBatchPlan& plan) {
    return batch_groups_offset(plan) + align256(plan.table.size() * sizeof(cdt::BatchGroupDev));
}

size_t batch_bytes(const DriftBatchPlan& plan) {
    return batch_partials_offset(plan) + plan.partial_doubles * sizeof(double);
}

}  // namespace

extern "C" {

size_t cdt_drift_batch_workspace_bytes(uint32_t n_jobs, const cdt_drift_job* jobs) {
    DriftBatchPlan plan;
    if (plan_drift_batch("cdt_drift_batch_workspace_bytes", n_jobs, jobs, &plan, false))
        return 0;
    return batch_bytes(plan);
}

}  // extern "C"

namespace {

// The batched Eq. 4's set-up shared by the launch and its read-stream aid:
// plan the jobs, check ws, and copy the job and group tables into it (with
// the partial-sum addresses filled in).  *launch is false when there is no
// work.
int stage_drift_batch(const char* fn, uint32_t n_jobs, const cdt_drift_job* jobs, void* ws,
                      size_t ws_bytes, hipStream_t st, DriftBatchPlan* plan, bool* launch) {
    *launch = false;
    int rc = plan_drift_batch(fn, n_jobs, jobs, plan, true);
    if (rc) return rc;
    if (plan->table.empty()) return ok();
    const size_t need = batch_bytes(*plan);
    if (!ws || ws_bytes < need)
        return fail(CDT_EINVAL, "%s: workspace of %zu bytes needed, %zu given", fn, need,
                    ws ? ws_bytes : 0);
    if (!aligned16(ws)) return fail(CDT_EALIGN, "%s: ws must be 16-byte aligned", fn);
    // partial offsets -> addresses behind the tables in ws; the two tables
    // go up in one copy, staged contiguously in pageable host memory (such a
    // copy completes before hipMemcpyAsync returns, so `staged` may go)
    char* base = static_cast<char*>(ws);
    double* partials = reinterpret_cast<double*>(base + batch_partials_offset(*plan));
    for (cdt::DriftJobDev& d : plan->table)
        if (!d.direct) d.partial = partials + reinterpret_cast<uintptr_t>(d.partial);
    std::vector<char> staged(batch_partials_offset(*plan), 0);
    memcpy(staged.data(), plan->table.data(), plan->table.size() * sizeof(cdt::DriftJobDev));
    memcpy(staged.data() + batch_groups_offset(*plan), plan->groups.data(),
           plan->groups.size() * sizeof(cdt::BatchGroupDev));
    const hipError_t e = hipMemcpyAsync(ws, staged.data(), staged.size(), hipMemcpyHostToDevice,
                                        st);
    if (e != hipSuccess) return device_status(e, fn);
    *launch = true;
    return CDT_OK;
}

}  // namespace

extern "C" {

int cdt_drift_score_batch(uint32_t n_jobs, const cdt_drift_job* jobs, void* ws, size_t ws_bytes,
                          void* stream) {
    const char* fn = "cdt_drift_score_batch";
    hipStream_t st = static_cast<hipStream_t>(stream);
    DriftBatchPlan plan;
    bool launch = false;
    int rc = stage_drift_batch(fn, n_jobs, jobs, ws, ws_bytes, st, &plan, &launch);
    if (rc || !launch) return rc;
    char* base = static_cast<char*>(ws);
    return device_status(
        cdt::launch_drift_batch(
            reinterpret_cast<const cdt::DriftJobDev*>(base),
            static_cast<uint32_t>(plan.table.size()),
            reinterpret_cast<const cdt::BatchGroupDev*>(base + batch_groups_offset(plan)),
            static_cast<uint32_t>(plan.groups.size()), plan.total_iters, plan.total_blocks, st),
        fn);
}

int cdt_drift_read_stream_batch(uint32_t n_jobs, const cdt_drift_job* jobs, void* ws,
                                size_t ws_bytes, void* stream) {
    const char* fn = "cdt_drift_read_stream_batch";
    hipStream_t st = static_cast<hipStream_t>(stream);
    DriftBatchPlan plan;
    bool launch = false;
    int rc = stage_drift_batch(fn, n_jobs, jobs, ws, ws_bytes, st, &plan, &launch);
    if (rc || !launch) return rc;
    char* base = static_cast<char*>(ws);
    return device_status(
        cdt::launch_drift_batch_read_stream(
            reinterpret_cast<const cdt::DriftJobDev*>(base),
            reinterpret_cast<const cdt::BatchGroupDev*>(base + batch_groups_offset(plan)),
            static_cast<uint32_t>(plan.groups.size()), plan.total_iters, st),
        fn);
}

int cdt_drift_read_stream(uint32_t S, uint32_t C, uint32_t T, uint32_t H, const uint16_t* h,
                          const float* ref, void* ws, size_t ws_bytes, void* stream) {
    const char* fn = "cdt_drift_read_stream";
    int rc = check_shape(fn, S, C, T, H);
    if (rc) return rc;
    if (static_cast<uint64_t>(S) * C * T * H == 0) return ok();
    if (!h || !ref) return fail(CDT_EINVAL, "%s: NULL array", fn);
    if (!aligned16(h) || !aligned16(ref))
        return fail(CDT_EALIGN, "%s: arrays must be 16-byte aligned", fn);
    const size_t need = cdt_reduce_workspace_bytes(S, C, T, H);
    if (!ws || ws_bytes < need)
        return fail(CDT_EINVAL, "%s: workspace of %zu bytes needed, %zu given", fn, need,
                    ws ? ws_bytes : 0);
    if (!aligned16(ws)) return fail(CDT_EALIGN, "%s: ws must be 16-byte aligned", fn);
    return device_status(cdt::launch_drift_read_stream(S, C, T, H, h, ref, ws,
                                                       static_cast<hipStream_t>(stream)),
                         fn);
}

int cdt_drift_score_f16ref(uint32_t S, uint32_t C, uint32_t T, uint32_t H, const uint16_t* h,
                           const uint16_t* r, float* score, double* num_den, void* ws,
                           size_t ws_bytes, void* stream) {
    return drift_common("cdt_drift_score_f16ref", cdt::DriftMetric::kL2HalfRef, S, C, T, H, h, r,
                        score, num_den, ws, ws_bytes, stream);
}

int cdt_cosine_score(uint32_t S, uint32_t C, uint32_t T, uint32_t H, const uint16_t* h,
                     const float* ref, float* score, double* sums, void* ws, size_t ws_bytes,
                     void* stream) {
    return drift_common("cdt_cosine_score", cdt::DriftMetric::kCosine, S, C, T, H, h, ref, score,
                        sums, ws, ws_bytes, stream);
}

int cdt_cosine_score_f16ref(uint32_t S, uint32_t C, uint32_t T, uint32_t H, const uint16_t* h,
                            const uint16_t* r, float* score, double* sums, void* ws,
                            size_t ws_bytes, void* stream) {
    return drift_common("cdt_cosine_score_f16ref", cdt::DriftMetric::kCosineHalfRef, S, C, T, H,
                        h, r, score, sums, ws, ws_bytes, stream);
}

size_t cdt_auroc_workspace_bytes(uint32_t n_cfg) {
    return static_cast<size_t>(n_cfg) * sizeof(cdt_auroc_cfg);
}

namespace {

// Host checks of a configuration table against n_scores scores and flags.
int check_auroc_table(const char* fn, uint32_t n_cfg, const cdt_auroc_cfg* cfgs,
                      uint64_t n_scores, uint32_t flags) {
    if (flags & ~15u) return fail(CDT_EINVAL, "%s: bad flags", fn);
    if (!cfgs) return fail(CDT_EINVAL, "%s: NULL cfgs", fn);
    if (n_cfg > (1u << 24)) return fail(CDT_ELIMIT, "%s: n_cfg above 2^24", fn);
    for (uint32_t g = 0; g < n_cfg; ++g) {
        const cdt_auroc_cfg& c = cfgs[g];
        if (c.S > 64) return fail(CDT_ELIMIT, "%s: cfg %u has S=%u above 64", fn, g, c.S);
        if (c.cfg_id >= kMaxId) return fail(CDT_ELIMIT, "%s: cfg %u cfg_id >= 2^24", fn, g);
        if (!canaries_fit(c.canary_base, c.C))
            return fail(CDT_ELIMIT, "%s: cfg %u canary_base + C above 2^32", fn, g);
        const uint64_t len = static_cast<uint64_t>(c.S) * c.C;
        if ((flags & CDT_AUROC_POOLED) && len > kMaxPooled)
            return fail(CDT_ELIMIT, "%s: cfg %u has C*S=%llu above %u for pooled ranking", fn,
                        g, static_cast<unsigned long long>(len), kMaxPooled);
        if (c.C > (1u << 30)) return fail(CDT_ELIMIT, "%s: cfg %u C above 2^30", fn, g);
        if (c.score_off > n_scores || len > n_scores - c.score_off)
            return fail(CDT_EINVAL, "%s: cfg %u table [%llu, +%llu) outside %llu scores", fn, g,
                        static_cast<unsigned long long>(c.score_off),
                        static_cast<unsigned long long>(len),
                        static_cast<unsigned long long>(n_scores));
    }
    return CDT_OK;
}

// Host checks of the output arrays of one scoring launch.
int check_auroc_outputs(const char* fn, uint32_t flags, uint64_t* counts, uint64_t* pooled,
                        uint64_t* baseline) {
    if (flags & ~15u) return fail(CDT_EINVAL, "%s: bad flags", fn);
    if (!counts) return fail(CDT_EINVAL, "%s: NULL counts", fn);
    if ((flags & CDT_AUROC_POOLED) && !pooled)
        return fail(CDT_EINVAL, "%s: pooled counts requested but pooled is NULL", fn);
    if ((flags & CDT_AUROC_RANDOM) && !baseline)
        return fail(CDT_EINVAL, "%s: baseline counts requested but baseline is NULL", fn);
    return CDT_OK;
}

// Copy a validated table (held in library-owned pageable memory, see
// validated_table) into the device buffer `table` on `st`.  A copy from
// pageable host memory completes before hipMemcpyAsync returns, so the host
// table may be released afterwards.
int upload_table(const char* fn, const std::vector<cdt_auroc_cfg>& cfgs, void* table,
                 size_t table_bytes, hipStream_t st) {
    const size_t need = cdt_auroc_workspace_bytes(static_cast<uint32_t>(cfgs.size()));
    if (!table || table_bytes < need)
        return fail(CDT_EINVAL, "%s: workspace of %zu bytes needed, %zu given", fn, need,
                    table ? table_bytes : 0);
    if (!aligned16(table)) return fail(CDT_EALIGN, "%s: ws must be 16-byte aligned", fn);
    const hipError_t e = hipMemcpyAsync(table, cfgs.data(), need, hipMemcpyHostToDevice, st);
    if (e != hipSuccess) return device_status(e, fn);
    return CDT_OK;
}

// The caller's table copied once into library memory and validated there:
// what is checked is what is uploaded, even if the caller's memory changes
// meanwhile, and the caller may reuse it (pinned or not) once the call
// returns.
int validated_table(const char* fn, uint32_t n_cfg, const cdt_auroc_cfg* cfgs,
                    uint64_t n_scores, uint32_t flags, std::vector<cdt_auroc_cfg>* out) {
    if (!cfgs) return fail(CDT_EINVAL, "%s: NULL cfgs", fn);
    if (n_cfg > (1u << 24)) return fail(CDT_ELIMIT, "%s: n_cfg above 2^24", fn);
    out->assign(cfgs, cfgs + n_cfg);
    return check_auroc_table(fn, n_cfg, out->data(), n_scores, flags);
}

}  // namespace

int cdt_auroc(uint32_t n_cfg, const cdt_auroc_cfg* cfgs, const float* scores, uint64_t n_scores,
              uint64_t seed, uint32_t flags, uint64_t* counts, uint64_t* pooled,
              uint64_t* baseline, void* ws, size_t ws_bytes, void* stream) {
    static_assert(sizeof(cdt_auroc_cfg) == sizeof(cdt::AurocCfgDev), "cfg layout");
    if (flags & ~15u) return fail(CDT_EINVAL, "cdt_auroc: bad flags");
    if (n_cfg == 0) return ok();
    int rc = check_auroc_outputs("cdt_auroc", flags, counts, pooled, baseline);
    if (rc) return rc;
    std::vector<cdt_auroc_cfg> table;
    rc = validated_table("cdt_auroc", n_cfg, cfgs, n_scores, flags, &table);
    if (rc) return rc;
    if (!scores) {
        for (const cdt_auroc_cfg& c : table)
            if (static_cast<uint64_t>(c.S) * c.C > 0)
                return fail(CDT_EINVAL, "cdt_auroc: scores is NULL");
    }
    hipStream_t st = static_cast<hipStream_t>(stream);
    rc = upload_table("cdt_auroc", table, ws, ws_bytes, st);
    if (rc) return rc;
    return device_status(cdt::launch_auroc(n_cfg, static_cast<const cdt::AurocCfgDev*>(ws),
                                           scores, n_scores, seed, flags, counts, pooled,
                                           baseline, st),
                         "cdt_auroc");
}

int cdt_auroc_upload(uint32_t n_cfg, const cdt_auroc_cfg* cfgs, uint64_t n_scores,
                     uint32_t flags, void* table, size_t table_bytes, void* stream) {
    if (flags & ~15u) return fail(CDT_EINVAL, "cdt_auroc_upload: bad flags");
    if (n_cfg == 0) return ok();
    std::vector<cdt_auroc_cfg> staged;
    int rc = validated_table("cdt_auroc_upload", n_cfg, cfgs, n_scores, flags, &staged);
    if (rc) return rc;
    rc = upload_table("cdt_auroc_upload", staged, table, table_bytes,
                      static_cast<hipStream_t>(stream));
    if (rc) return rc;
    return ok();
}

int cdt_auroc_launch(uint32_t n_cfg, const void* table, const float* scores, uint64_t n_scores,
                     uint64_t seed, uint32_t flags, uint64_t* counts, uint64_t* pooled,
                     uint64_t* baseline, void* stream) {
    if (flags & ~15u) return fail(CDT_EINVAL, "cdt_auroc_launch: bad flags");
    if (n_cfg == 0) return ok();
    if (n_cfg > (1u << 24)) return fail(CDT_ELIMIT, "cdt_auroc_launch: n_cfg above 2^24");
    int rc = check_auroc_outputs("cdt_auroc_launch", flags, counts, pooled, baseline);
    if (rc) return rc;
    if (!table || !scores) return fail(CDT_EINVAL, "cdt_auroc_launch: NULL table or scores");
    if (!aligned16(table)) return fail(CDT_EALIGN, "cdt_auroc_launch: table must be 16-byte aligned");
    return device_status(cdt::launch_auroc(n_cfg, static_cast<const cdt::AurocCfgDev*>(table),
                                           scores, n_scores, seed, flags, counts, pooled,
                                           baseline, static_cast<hipStream_t>(stream)),
                         "cdt_auroc_launch");
}

size_t cdt_auroc_canaries_workspace_bytes(uint32_t n_cfg) {
    return align256(static_cast<size_t>(n_cfg) * sizeof(cdt_auroc_cfg)) +
           static_cast<size_t>(n_cfg) * sizeof(uint64_t);
}

int cdt_auroc_canaries(uint32_t n_cfg, const cdt_auroc_cfg* cfgs, const float* scores,
                       uint64_t n_scores, uint64_t seed, uint32_t flags, uint32_t* per_canary,
                       void* ws, size_t ws_bytes, void* stream) {
    const char* fn = "cdt_auroc_canaries";
    if (flags & ~(CDT_AUROC_CONTROL | CDT_CTRL_INCLUDE_TRUE | CDT_AUROC_RANDOM))
        return fail(CDT_EINVAL, "%s: bad flags (the pooled ranking has no per-canary form)", fn);
    if (n_cfg == 0) return ok();
    std::vector<cdt_auroc_cfg> table;
    int rc = validated_table(fn, n_cfg, cfgs, n_scores, flags, &table);
    if (rc) return rc;
    // each configuration's canaries follow the previous ones' in per_canary
    const size_t table_bytes = align256(static_cast<size_t>(n_cfg) * sizeof(cdt_auroc_cfg));
    std::vector<char> staged(cdt_auroc_canaries_workspace_bytes(n_cfg), 0);
    memcpy(staged.data(), table.data(), n_cfg * sizeof(cdt_auroc_cfg));
    uint64_t* offsets = reinterpret_cast<uint64_t*>(staged.data() + table_bytes);
    uint64_t total = 0;
    bool any_scores = false;
    for (uint32_t g = 0; g < n_cfg; ++g) {
        offsets[g] = total;
        total += table[g].C;
        any_scores = any_scores || static_cast<uint64_t>(table[g].S) * table[g].C > 0;
    }
    if (total == 0) return ok();
    if (!per_canary) return fail(CDT_EINVAL, "%s: per_canary is NULL", fn);
    if (any_scores && !scores) return fail(CDT_EINVAL, "%s: scores is NULL", fn);
    if (!ws || ws_bytes < staged.size())
        return fail(CDT_EINVAL, "%s: workspace of %zu bytes needed, %zu given", fn, staged.size(),
                    ws ? ws_bytes : 0);
    if (!aligned16(ws)) return fail(CDT_EALIGN, "%s: ws must be 16-byte aligned", fn);
    hipStream_t st = static_cast<hipStream_t>(stream);
    // from pageable host memory: the copy completes before the call returns
    const hipError_t e = hipMemcpyAsync(ws, staged.data(), staged.size(), hipMemcpyHostToDevice,
                                        st);
    if (e != hipSuccess) return device_status(e, fn);
    char* base = static_cast<char*>(ws);
    return device_status(
        cdt::launch_auroc_canaries(n_cfg, reinterpret_cast<const cdt::AurocCfgDev*>(base),
                                   reinterpret_cast<const uint64_t*>(base + table_bytes), scores,
                                   n_scores, seed, flags, per_canary, st),
        fn);
}

int cdt_auroc_values(uint32_t n_cfg, const uint64_t* counts, const uint64_t* pooled,
                     const uint64_t* baseline, double* values, void* stream) {
    if (n_cfg == 0) return ok();
    if (n_cfg > (1u << 24)) return fail(CDT_ELIMIT, "cdt_auroc_values: n_cfg above 2^24");
    if (!counts || !values) return fail(CDT_EINVAL, "cdt_auroc_values: NULL counts or values");
    return device_status(cdt::launch_auroc_values(n_cfg, counts, pooled, baseline, values,
                                                  static_cast<hipStream_t>(stream)),
                         "cdt_auroc_values");
}

}  // extern "C"
