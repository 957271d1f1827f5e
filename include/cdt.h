/*
 * cdt.h -- C ABI of libcdt, the canary-versus-reference activation drift
 * detector of "Integrity of peer-to-peer distributed LLM inference under
 * malicious nodes" (Cihangiroglu & Nocera), on AMD Instinct MI355X (gfx950).
 *
 * Vocabulary (Section 3): a pipeline of k stages ("shards", S here) hands
 * T x d activations (d = H here) from stage to stage; the verifier holds fp32
 * reference activations a*_i for n canaries (C here) and compares the fp16
 * activations h_i each stage returns for them.  A block is one (shard,
 * canary) pair: T*H elements.
 *
 * Layouts (row-major, contiguous):
 *   activations  ref[S][C][T][H] fp32,  h[S][C][T][H] fp16 (as uint16 bits)
 *   per block    [S][C]  (block statistics and scales)
 *   scores       [C][S]  (one canary's k mismatches adjacent, as Eq. 5 ranks)
 *
 * Conventions for every call:
 *   - Array pointers are DEVICE pointers (hipMalloc or torch allocations)
 *     owned by the caller, unless a comment says "host".  The library never
 *     allocates or frees memory.
 *   - Calls are asynchronous on `stream` (a hipStream_t passed as void*,
 *     NULL = the default stream).  The calls that take a HOST table
 *     (cdt_auroc, cdt_auroc_upload, cdt_auroc_canaries and the batched
 *     launches) copy it from library-held pageable memory, a copy that is
 *     complete when the call returns; nothing else waits on the host.
 *   - Arguments are validated before any device work; on failure nothing is
 *     launched and an error code is returned.  cdt_last_error() gives a
 *     per-thread description of the last failure.
 *   - Results are deterministic: fixed reduction orders, no atomics.
 *   - activations need H % 8 == 0, T*H < 2^32, S*C <= 2^32,
 *     S*C*T*H <= 2^40 and 16-byte aligned pointers; S <= 64 wherever a
 *     shard bit mask is involved (CDT_ELIMIT otherwise).
 *   - Empty shapes (S, C, T or H zero) are valid and do no work, except
 *     that drift scores of empty blocks are written as 0.
 *   - Canary sharding: every generated value and every per-canary random
 *     draw is keyed by the canary's global index canary_base + c.  A caller
 *     holding canaries [c0, c0 + C) of a larger run passes canary_base = c0
 *     and gets bit for bit those canaries' references, live activations,
 *     scores and per-canary counts of the whole run; the integer counts of
 *     cdt_auroc add up exactly over such slices (not the pooled ranking,
 *     which compares canaries with each other).  canary_base + C <= 2^32.
 */
#ifndef CDT_H
#define CDT_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Return codes. */
#define CDT_OK 0
#define CDT_EINVAL 1  /* null pointer, bad enum, bad size or workspace too small */
#define CDT_EALIGN 2  /* array pointer not 16-byte aligned                       */
#define CDT_ELIMIT 3  /* shape beyond a documented limit                          */
#define CDT_EDEVICE 4 /* HIP launch or runtime error                             */

/* Random streams (fourth Philox counter word = stream << 24 | id). */
#define CDT_STREAM_REF 0
#define CDT_STREAM_BENIGN 1
#define CDT_STREAM_T12 2
#define CDT_STREAM_T3 3
#define CDT_STREAM_TAMPER_ADD 4
#define CDT_STREAM_TAMPER_FLIP 5
#define CDT_STREAM_SCRAMBLE 6
#define CDT_STREAM_RANDOM 7
#define CDT_STREAM_OUTLIER 8
#define CDT_STREAM_ALT 9
#define CDT_STREAM_ALT_T12 10
#define CDT_STREAM_ALT_T3 11

/* Interface version; changes whenever a layout, a generator rule or the set
 * of entry points changes (11: cdt_drift_read_stream_batch added; 10:
 * cdt_auroc_canaries added; 9: batched live
 * pass and Eq. 4, the live-pass stream aid, exact-norm scales under the
 * propagation model; 8:
 * cdt_drift_score_noalloc added; 7: cdt_auroc_values added, NaN scores
 * rank above every number).  cdt_version() returns the library's, which a
 * caller compares with the CDT_INTERFACE_VERSION of the header it was
 * built with. */
#define CDT_INTERFACE_VERSION 11
int cdt_version(void);

/* Description of the last error on the calling thread ("" if none). */
const char* cdt_last_error(void);

/* ------------------------------------------------------------------------ */
/* Synthetic references (the verifier's offline fp32 pass, Eq. 1 and        */
/* Section 3.3; no model weights, so a seeded stand-in)                     */
/* ------------------------------------------------------------------------ */

/* Outlier channel gains gain[H] (fp32, device): the n_out channels j with the
 * smallest (w_j, j), w_j = Philox4x32-10 word 0 of counter
 * (j, 0, 0, OUTLIER<<24 | ref_set_id) under key (lo32 seed, hi32 seed), get
 * gain `big`; every other channel gets 1.  Needs n_out <= H <= 32768 and
 * ref_set_id < 2^24. */
int cdt_outlier_gain(uint32_t H, uint32_t n_out, float big, uint64_t seed, uint32_t ref_set_id,
                     float* gain, void* stream);

/* ref[s][c][t][j] = fp32(z * gain[j]) with z the unit normal of element
 * e = t*H + j drawn from stream REF (id = ref_set_id): Philox call
 * q = e/2 of counter (q, c, s, REF<<24 | ref_set_id), words 0-1 for even e
 * and 2-3 for odd e, made into z by the Irwin-Hall rule
 *   n = sum of the four 16-bit halves of the two words - 131070,
 *   z = fp32(n) * fp32(sqrt(3 / (2^32 - 1))).
 * c in the counter is the global canary index canary_base + c.
 * gain: [H] fp32 (device). */
int cdt_ref_synth(uint32_t S, uint32_t C, uint32_t T, uint32_t H, uint64_t seed,
                  uint32_t ref_set_id, uint32_t canary_base, const float* gain, float* ref,
                  void* stream);

/* Workspace (device bytes) needed by cdt_ref_stats, the four block
 * reductions (cdt_drift_score, cdt_drift_score_f16ref, cdt_cosine_score,
 * cdt_cosine_score_f16ref), cdt_sim_score and cdt_tamper_scale_exact for
 * this shape: per-block partial sums (up to three fp64 per chunk of 32768
 * elements).  Calls on one stream may share one workspace; calls that can
 * overlap (different streams) need their own. */
size_t cdt_reduce_workspace_bytes(uint32_t S, uint32_t C, uint32_t T, uint32_t H);

/* Per-block reference statistics in fp64: sumsq[s][c] = sum a^2 and
 * sumabs[s][c] = sum |a| over the block (mu_i of Eq. 2 is sumabs / (T H)).
 * ws: device workspace of at least cdt_reduce_workspace_bytes bytes. */
int cdt_ref_stats(uint32_t S, uint32_t C, uint32_t T, uint32_t H, const float* ref,
                  double* sumsq, double* sumabs, void* ws, size_t ws_bytes, void* stream);

/* Per-block scales, each computed in fp64 and rounded once to fp32:
 *   tscale[b] = eps * sqrt(sumsq[b] / (T H))       (Gaussian tamper: eps rms)
 *   bscale[b] = sigma_b * (sumabs[b] / (T H))      (Eq. 2: sigma_hw mu_i)
 * Either output may be NULL.  nblocks = S*C. */
int cdt_block_scales(uint64_t nblocks, uint32_t T, uint32_t H, const double* sumsq,
                     const double* sumabs, double eps, double sigma_b, float* tscale,
                     float* bscale, void* stream);

/* ------------------------------------------------------------------------ */
/* Live pass simulation (Eqs. 2-3)                                           */
/* ------------------------------------------------------------------------ */
#define CDT_NOISE_ELEMENTWISE 0 /* delta ~ N(0, (sigma_b |a|)^2) per element      */
#define CDT_NOISE_BLOCK 1       /* delta ~ N(0, bscale^2): Eq. 2, sigma_hw mu_i    */
#define CDT_DIST_GAUSS 0        /* unit normal (Irwin-Hall stand-in)              */
#define CDT_DIST_T3 1           /* unit-variance Student-t, 3 degrees of freedom  */
#define CDT_T_ADD 1             /* Gaussian tamper: v + tscale * z                */
#define CDT_T_FLIP 2            /* sign flip of a selected fraction (all: -v)     */
#define CDT_T_SCALE 4           /* rescale: (1 + alpha) v                         */
#define CDT_BASE_BENIGN 0       /* tamper the benign output a + delta             */
#define CDT_BASE_CLEAN 1        /* tamper the clean a (Eq. 3 read literally)      */

typedef struct cdt_sim_params {
    uint64_t seed;          /* Philox key (lo32, hi32)                            */
    uint32_t cfg_id;        /* counter id of the noise streams, < 2^24             */
    uint32_t benign_mode;   /* CDT_NOISE_*                                         */
    uint32_t benign_dist;   /* CDT_DIST_*                                          */
    uint32_t tamper;        /* OR of CDT_T_* (all three: Gaussian, flip, rescale) */
    uint32_t tamper_base;   /* CDT_BASE_*                                          */
    uint32_t redraw;        /* 0: benign noise from BENIGN/T12/T3; 1: from ALT/    */
                            /* ALT_T12/ALT_T3, an independent benign recompute of  */
                            /* the same stage (Section 4.5: recompute ceiling and  */
                            /* noisy-reference ablation)                           */
    uint64_t mal_mask;      /* bit s set: shard s is malicious (tampers)           */
    double sigma_b;         /* ELEMENTWISE noise level (used as fp32(sigma_b))     */
    double flip_p;          /* flip probability in [0, 1]; 1 flips every element   */
    double scale;           /* rescale factor 1 + alpha (used as fp32(scale))      */
    const float* bscale;    /* device [S][C], BLOCK mode, else may be NULL         */
    const float* tscale;    /* device [S][C], needed with CDT_T_ADD                */
    double carry;           /* propagation gain g in [0, 1] (used as fp32(g)); 0:  */
                            /* independent stages                                  */
    uint32_t canary_base;   /* global index of canary 0 (0 for a whole run)        */
    uint32_t reserved;      /* must be 0                                           */
} cdt_sim_params;

/* h = fp16_rne(v) for every element, with (one fp32 operation per step, in
 * this order, no fused multiply-add):
 *   sc = fp32(sigma_b) * |a|  (ELEMENTWISE)   or  bscale[s][c]  (BLOCK)
 *   zb = z_BENIGN, or for T3: q = (z1*z1 + z2*z2) + z3*z3 with z1, z2 from
 *        one T12 call (q = e) and z3 from stream T3, zb = q == 0 ? 0 :
 *        z_BENIGN / sqrt(q)
 *   v  = a + sc * zb
 * and on malicious shards, starting from v (BENIGN base) or a (CLEAN base):
 *   ADD   v = v + tscale[s][c] * z_TAMPER_ADD
 *   FLIP  v = -v if flip_p >= 1 or u < floor(flip_p 2^32), u = word e%4 of
 *         TAMPER_FLIP call q = e/4
 *   SCALE v = fp32(scale) * v
 * One-normal streams use call q = e/2 like cdt_ref_synth; every counter is
 * (q, canary_base + c, s, stream<<24 | cfg_id).  p: host struct, read
 * during the call.
 * Needs S <= 64.
 *
 * Propagation model (carry g > 0; the depth, position, collusion and
 * frontier substudies of Sections 4.4 and 5.3-5.5): stage s sees the live
 * error of stage s-1, d = fp32(h_{s-1} - a_{s-1}), as the paper's Eq. 2
 * feeds f_i the live h_{i-1}.  Its noise-free output is u = fp32(a +
 * fp32(g * d)) (u = a for stage 0); the benign step is v = u + sc * zb (sc
 * still from |a|), the clean base is u, and the tamper follows as above.
 * g = 0 gives the independent stages exactly. */
int cdt_canary_sim(uint32_t S, uint32_t C, uint32_t T, uint32_t H, const cdt_sim_params* p,
                   const float* ref, uint16_t* h, void* stream);

/* The live pass of several runs in one launch (the factorial sweep generates
 * the configurations of a reference set together): job j writes its own h
 * from its ref with its own parameters, bitwise as cdt_canary_sim would.
 * The chunks of all jobs form one grid, so short runs share the launch's
 * ramp-up and tail.  Consecutive jobs that read the same ref array in the
 * same shape are generated together, so that each
 * reference chunk is read from HBM about once for all of them: with fewer
 * than 8 such jobs their work is walked chunk by chunk, the jobs of a chunk
 * one after another (re-reads from L2); with 8 or more, each XCD takes its
 * own jobs over the same reference offsets (re-reads from the last-level
 * cache).  Order the jobs so that runs sharing references are adjacent.
 * Every job must use the same benign_dist and benign_mode and carry 0
 * (CDT_EINVAL otherwise); their shapes, tamper settings and scales may
 * differ.  jobs and each p: HOST, read during the call (the job and group
 * tables are copied into ws on `stream` from library-held host memory, a
 * copy a stream capture must not record: call it outside captures).  At
 * most 65536 jobs.
 * ws: cdt_sim_batch_workspace_bytes(n_jobs) device bytes. */
typedef struct cdt_sim_job {
    uint32_t S, C, T, H;
    const cdt_sim_params* p;  /* host                            */
    const float* ref;         /* device fp32 [S][C][T][H]        */
    uint16_t* h;              /* device fp16 bits [S][C][T][H]   */
} cdt_sim_job;

size_t cdt_sim_batch_workspace_bytes(uint32_t n_jobs);
int cdt_canary_sim_batch(uint32_t n_jobs, const cdt_sim_job* jobs, void* ws, size_t ws_bytes,
                         void* stream);

/* Measurement aid for the live pass's memory bound: reads ref and writes h
 * exactly as cdt_canary_sim does for Gaussian noise on independent stages
 * (the same chunks, loads, prefetch and stores), with the live-pass
 * arithmetic replaced by h = fp16_rne(a), no random numbers drawn.  Its rate
 * is what the memory system delivers for the live pass's 4 B-read and
 * 2 B-write access pattern.  Errors as cdt_canary_sim. */
int cdt_canary_sim_stream(uint32_t S, uint32_t C, uint32_t T, uint32_t H, const float* ref,
                          uint16_t* h, void* stream);

/* Per-block scale of the exact-norm Gaussian tamper of Section 3.2,
 * tau(v) = v + eps ||v||_F N / ||N||_F: with v the untampered output of the
 * block (a + delta, formed exactly as cdt_canary_sim forms it, or a itself
 * for the clean base) and N its TAMPER_ADD normals,
 *   tscale[s][c] = fp32( eps * sqrt( sum v^2 / sum N^2 ) )   (fp64 sums),
 * so that cdt_canary_sim's Gaussian tamper, given this tscale, adds a
 * perturbation of norm eps ||v|| (up to rounding).  p gives the benign
 * settings, seed and cfg_id of the run (its tamper fields are ignored).
 *
 * Under the propagation model (p->carry > 0) v is a malicious stage's
 * untampered output given the live error carried in from the stage before
 * (the clean base: its noise-free u), so it depends on every stage
 * upstream.  The scales are found for the malicious stages (p->mal_mask) in
 * pipeline order: for stage m, every element is walked through stages
 * 0 .. m as cdt_canary_sim walks it, the earlier malicious stages tampered
 * with p's tamper settings and the Gaussian scales this call has already
 * written to tscale, and tscale[m][c] is formed as above from stage m's
 * sums.  Entries of benign stages are set to 0 (norms too).  Passing the
 * result as tscale to cdt_canary_sim with the same p then runs the paper's
 * attack, every colluder at exactly eps ||v||.
 * norms: optional device [S][C][2] fp64 (sum v^2, sum N^2), or NULL.
 * ws: cdt_reduce_workspace_bytes bytes. */
int cdt_tamper_scale_exact(uint32_t S, uint32_t C, uint32_t T, uint32_t H,
                           const cdt_sim_params* p, const float* ref, double eps, float* tscale,
                           double* norms, void* ws, size_t ws_bytes, void* stream);

/* The live pass and Eq. 4 in one launch (the simulation study's fast path):
 * every reference element is read once, its live fp16 value formed exactly
 * as cdt_canary_sim forms it, and scored at once as cdt_drift_score scores
 * it.  score / num_den are bitwise those of cdt_canary_sim followed by
 * cdt_drift_score.  h: device [S][C][T][H] fp16 bits written as well, or
 * NULL to skip the store.  ws: cdt_reduce_workspace_bytes bytes.
 * Needs S <= 64. */
int cdt_sim_score(uint32_t S, uint32_t C, uint32_t T, uint32_t H, const cdt_sim_params* p,
                  const float* ref, uint16_t* h, float* score, double* num_den, void* ws,
                  size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------ */
/* Relative-L2 mismatch, Eq. 4                                               */
/* ------------------------------------------------------------------------ */

/* score[c][s] = fp32( sqrt( sum (h - a)^2 / sum a^2 ) ) over block (s, c), the
 * sums accumulated in fp64 from the exactly widened fp16 h and fp32 a; a
 * block with sum a^2 = 0 scores 0 if h = a there and +inf otherwise.
 * num_den: optional device [C][S][2] fp64 (sum (h-a)^2, sum a^2), or NULL.
 * ws: device workspace of at least cdt_reduce_workspace_bytes bytes.
 * h and ref are read once each; nothing else touches HBM in bulk. */
int cdt_drift_score(uint32_t S, uint32_t C, uint32_t T, uint32_t H, const uint16_t* h,
                    const float* ref, float* score, double* num_den, void* ws, size_t ws_bytes,
                    void* stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): exactly
 * cdt_drift_score (same kernels, same results bit for bit) with no workspace
 * argument.  The per-chunk partial sums go to a fixed scratch array of
 * CDT_NOALLOC_SCRATCH_BYTES in the library's own device memory, which each
 * GPU the library runs on holds until the process ends.  A shape needs
 * 16 bytes per chunk of 32768 elements when its blocks span more than one
 * chunk (S*C*ceil(T*H/32768) chunks; the 16 x 256 x 256 x 8192 shape needs
 * 4 MiB) and none otherwise; a shape beyond the limit returns CDT_ELIMIT and
 * launches nothing.  No memory is allocated or freed, and every partial sum
 * is written before it is read, so nothing needs clearing between calls.
 * All calls on one GPU share its array: calls that can overlap there (on
 * different streams, or from several threads without ordering) race and
 * must be serialised by the caller.  The first call on a device looks up
 * the array's device address (with that device current).  `stream` must
 * belong to the current device (CDT_EINVAL otherwise): the array used is
 * the current device's. */
#define CDT_NOALLOC_SCRATCH_BYTES 8388608u
int cdt_drift_score_noalloc(uint32_t S, uint32_t C, uint32_t T, uint32_t H, const uint16_t* h,
                            const float* ref, float* score, double* num_den, void* stream);

/* Eq. 4 over several arrays in one launch (the factorial sweep scores the
 * configurations of a reference set together; several runs against one
 * reference set): job j scores its own h[S][C][T][H] against its ref into
 * its score[C][S] (num_den optional), bitwise as cdt_drift_score would.  The
 * chunks of all jobs form one grid, so short arrays share the launch's
 * ramp-up and tail instead of paying one each, and one combine launch
 * finishes every block.  Consecutive jobs that read the same ref array in
 * the same shape share its reads: one workgroup scores a chunk
 * of up to 8 of them, reading the reference chunk once, so a group of up to
 * 8 jobs moves 2k + 4 bytes per element instead of 6k (larger groups read
 * the chunk once per 8 jobs, the repeats mostly from L2).  Order the jobs so
 * that arrays scored against one reference are adjacent.  jobs: HOST array,
 * validated and copied into ws during the call (reusable when the call
 * returns; the copy comes from library-held host memory, so a stream
 * capture must not record the call); jobs with S*C = 0 are skipped.  At
 * most 65536 jobs.
 * ws: cdt_drift_batch_workspace_bytes(n_jobs, jobs) device bytes (the job
 * and group tables and every job's partial sums); calls that can overlap
 * need their own. */
typedef struct cdt_drift_job {
    uint32_t S, C, T, H;
    const uint16_t* h;   /* device fp16 bits [S][C][T][H]      */
    const float* ref;    /* device fp32 [S][C][T][H]           */
    float* score;        /* device fp32 [C][S] (written)        */
    double* num_den;     /* device fp64 [C][S][2] or NULL       */
} cdt_drift_job;

/* Workspace bytes for cdt_drift_score_batch on these jobs (0 if a job's
 * shape is invalid; shapes only, pointers are not looked at). */
size_t cdt_drift_batch_workspace_bytes(uint32_t n_jobs, const cdt_drift_job* jobs);
int cdt_drift_score_batch(uint32_t n_jobs, const cdt_drift_job* jobs, void* ws, size_t ws_bytes,
                          void* stream);

/* Measurement aid for the batched Eq. 4's memory bound: the same checks,
 * tables, grid, chunks, loads, lane exchange and order as
 * cdt_drift_score_batch on the same arguments, with the arithmetic replaced
 * by an XOR fold of the loaded words; it writes nothing (a fold equal to a
 * fixed 32-bit sentinel would overwrite one score, which does not occur in
 * practice). */
int cdt_drift_read_stream_batch(uint32_t n_jobs, const cdt_drift_job* jobs, void* ws,
                                size_t ws_bytes, void* stream);

/* Measurement aid for Eq. 4's memory bound: reads h and ref exactly as
 * cdt_drift_score does (the same chunks, loads, lane exchange and order)
 * and computes nothing from them, so its rate is what the memory system
 * delivers for the drift kernel's access pattern.  Produces no result: ws
 * (cdt_reduce_workspace_bytes bytes, 16-byte aligned) may be overwritten.
 * Errors as cdt_drift_score. */
int cdt_drift_read_stream(uint32_t S, uint32_t C, uint32_t T, uint32_t H, const uint16_t* h,
                          const float* ref, void* ws, size_t ws_bytes, void* stream);

/* Relative-L2 mismatch against an fp16 reference r (Eq. 4 with the stored
 * fp32 reference replaced by a second live pass, Section 4.5: the
 * noisy-reference ablation and the redundant-recompute ceiling):
 * score[c][s] = fp32( sqrt( sum (h - r)^2 / sum r^2 ) ), sums in fp64.
 * r: device [S][C][T][H] fp16 bits.  Otherwise as cdt_drift_score. */
int cdt_drift_score_f16ref(uint32_t S, uint32_t C, uint32_t T, uint32_t H, const uint16_t* h,
                           const uint16_t* r, float* score, double* num_den, void* ws,
                           size_t ws_bytes, void* stream);

/* Cosine mismatch, the metric ablation of Section 4.4:
 * score[c][s] = fp32(1 - h.a / (||h|| ||a||)).  With d = h - a, A = sum a^2,
 * P = sum a d, D = sum d^2 (fp64, from exactly widened operands) and
 * Hn = A + 2P + D = ||h||^2, it is evaluated as
 *   (A D - P^2) / (sqrt(A Hn) (sqrt(A Hn) + A + P))      when A + P > 0,
 *   1 - (A + P) / sqrt(A Hn)                              otherwise,
 * the same value without the cancellation of 1 - cos near 0.  A block with
 * h or a all zero scores 0 if both are zero, else 1.
 * sums: optional device [C][S][3] fp64 (D, A, P), or NULL. */
int cdt_cosine_score(uint32_t S, uint32_t C, uint32_t T, uint32_t H, const uint16_t* h,
                     const float* ref, float* score, double* sums, void* ws, size_t ws_bytes,
                     void* stream);

/* The cosine mismatch against an fp16 reference r (a second live pass, as
 * in cdt_drift_score_f16ref): the cosine row of the recompute ceiling. */
int cdt_cosine_score_f16ref(uint32_t S, uint32_t C, uint32_t T, uint32_t H, const uint16_t* h,
                            const uint16_t* r, float* score, double* sums, void* ws,
                            size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------ */
/* Detection AUROC, Eqs. 5-6, the Mann-Whitney form and the scrambled-label  */
/* control of Section 4.5, batched over configurations                       */
/* ------------------------------------------------------------------------ */
#define CDT_AUROC_CONTROL 1     /* also count the scrambled-label control        */
#define CDT_AUROC_POOLED 2      /* also rank all C*S scores of a config together  */
#define CDT_CTRL_INCLUDE_TRUE 4 /* control keeps the true malicious shards as negatives */
#define CDT_AUROC_RANDOM 8      /* also count the random baseline                  */

typedef struct cdt_auroc_cfg {
    uint32_t S, C;       /* shards (<= 64) and canaries of this configuration     */
    uint64_t score_off;  /* element offset of its [C][S] table in `scores`       */
    uint64_t pos_mask;   /* malicious shards (the positives of the ranking)      */
    uint32_t cfg_id;     /* counter id of the SCRAMBLE stream (< 2^24)            */
    uint32_t canary_base; /* global index of canary 0 (0 for a whole run)          */
} cdt_auroc_cfg;

/* Bytes of device workspace cdt_auroc needs for n_cfg configurations. */
size_t cdt_auroc_workspace_bytes(uint32_t n_cfg);

/* For each configuration g (cfgs: HOST array of n_cfg entries, validated and
 * copied into ws during the call):
 *   counts[g][0..2] = G, E, pairs with G = #{(t, i in M, j not in M):
 *       m_ti > m_tj}, E the ties (Eq. 5 summed over canaries; Eq. 6 as
 *       printed is G / pairs, the Mann-Whitney value (G + E/2) / pairs);
 *   counts[g][3..5] = the same for the scrambled-label control (if
 *       CDT_AUROC_CONTROL, else 0): per canary t a benign shard j*, the
 *       (u mod B)-th benign shard in increasing order, u = Philox word 0
 *       of counter (canary_base + t, 0, 0, SCRAMBLE<<24 | cfg_id), B the
 *       number of benign shards, ranked against the benign shards other
 *       than j* (all other shards with CDT_CTRL_INCLUDE_TRUE);
 *   pooled[g][0..2] = G, E, pairs over every positive score against every
 *       negative score of the configuration (if CDT_AUROC_POOLED; needs
 *       C*S <= 16384; pooled may be NULL otherwise);
 *   baseline[g][0..2] = G, E, pairs of Eq. 5 with every score replaced by
 *       the random-baseline score of Section 4.5, u(t, s) = (w >> 8) 2^-24,
 *       w = Philox word 0 of counter (canary_base + t, s, 0, RANDOM<<24 |
 *       cfg_id) (if CDT_AUROC_RANDOM; baseline may be NULL otherwise).
 * Score order: the numeric order with -0 tying +0, and NaN above every
 * number (+inf included), NaN tying NaN: a block whose Eq. 4 mismatch is
 * not a number ranks as the most suspicious stage.
 * counts: device [n_cfg][6] uint64; scores: device fp32; n_scores bounds
 * every configuration's table. */
int cdt_auroc(uint32_t n_cfg, const cdt_auroc_cfg* cfgs, const float* scores, uint64_t n_scores,
              uint64_t seed, uint32_t flags, uint64_t* counts, uint64_t* pooled,
              uint64_t* baseline, void* ws, size_t ws_bytes, void* stream);

/* cdt_auroc in two parts, for a fixed set of configurations scored again and
 * again (a serving loop, or a stream capture replayed as a HIP graph).
 *
 * cdt_auroc_upload validates the HOST table cfgs exactly as cdt_auroc does,
 * against n_scores scores and the flags the launches will use, and copies
 * it into the device buffer `table` (cdt_auroc_workspace_bytes(n_cfg)
 * bytes, 16-byte aligned) on `stream`.  The table is copied into library
 * host memory before it is checked, so cfgs (pinned or not) may be reused
 * as soon as the call returns.
 *
 * cdt_auroc_launch scores `scores` against an uploaded table: it only
 * launches kernels (no copies, no host reads of device memory), so a stream
 * capture can record it.  Results are those of cdt_auroc with the same
 * arguments.  The kernels check every configuration again against the
 * n_scores given here (S <= 64, its table inside the scores, C*S <= 16384
 * for the pooled ranking); a configuration that fails writes 2^64 - 1 to
 * all its counts instead of being read. */
int cdt_auroc_upload(uint32_t n_cfg, const cdt_auroc_cfg* cfgs, uint64_t n_scores,
                     uint32_t flags, void* table, size_t table_bytes, void* stream);
int cdt_auroc_launch(uint32_t n_cfg, const void* table, const float* scores, uint64_t n_scores,
                     uint64_t seed, uint32_t flags, uint64_t* counts, uint64_t* pooled,
                     uint64_t* baseline, void* stream);

/* Eq. 6 from the counts above, on the device, in fp64: for configuration g
 *   values[g][0] = G / pairs           (Eq. 6 as printed: a tie counts 0)
 *   values[g][1] = (G + E/2) / pairs   (the Mann-Whitney reading stated after
 *                                       Eq. 6: a tie counts one half)
 *   values[g][2..3] the same for the scrambled-label control (counts[g][3..5]),
 *   values[g][4..5] the same for the pooled ranking (pooled[g][0..2]),
 *   values[g][6..7] the same for the random baseline (baseline[g][0..2]).
 * A ratio over zero pairs, or over counts holding the out-of-bounds marker
 * 2^64 - 1, is NaN; so are the pooled or baseline entries when that array is
 * NULL.  counts: device [n_cfg][6]; pooled, baseline: device [n_cfg][3] or
 * NULL; values: device [n_cfg][8] fp64 (written, caller-owned). */
int cdt_auroc_values(uint32_t n_cfg, const uint64_t* counts, const uint64_t* pooled,
                     const uint64_t* baseline, double* values, void* stream);

/* Eq. 5 per canary: the counts behind each canary's A^(t) = G_t / (|M| |N|)
 * (Eq. 6 is their mean), the paper's per-canary view of the detector against
 * its controls (Section 4.5).  For configuration g of cfgs (HOST array,
 * validated exactly as cdt_auroc validates it and copied into ws during the
 * call, so a stream capture must not record it) and each of its canaries t:
 *   per_canary[o_g + t][0..1] = G_t, E_t: positive shard i beats / ties
 *       negative shard j, over that canary's pairs (i in M, j not in M);
 *   per_canary[o_g + t][2..3] = the same for the scrambled-label control
 *       (its chosen benign stage against the others, as in cdt_auroc), 0
 *       without CDT_AUROC_CONTROL;
 *   per_canary[o_g + t][4..5] = the same with the random-baseline scores, 0
 *       without CDT_AUROC_RANDOM;
 * with o_g = C_0 + ... + C_{g-1}.  Summed over a configuration's canaries
 * they give cdt_auroc's counts.  Same score order as cdt_auroc.
 * flags: CDT_AUROC_CONTROL, CDT_CTRL_INCLUDE_TRUE, CDT_AUROC_RANDOM
 * (CDT_AUROC_POOLED has no per-canary form: CDT_EINVAL).
 * per_canary: device uint32 [sum of C][6] (written, caller-owned).
 * ws: cdt_auroc_canaries_workspace_bytes(n_cfg) device bytes, 16-byte
 * aligned (the table and the canary offsets). */
size_t cdt_auroc_canaries_workspace_bytes(uint32_t n_cfg);
int cdt_auroc_canaries(uint32_t n_cfg, const cdt_auroc_cfg* cfgs, const float* scores,
                       uint64_t n_scores, uint64_t seed, uint32_t flags, uint32_t* per_canary,
                       void* ws, size_t ws_bytes, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* CDT_H */
