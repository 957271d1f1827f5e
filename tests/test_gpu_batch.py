"""Batched launches against the single-run calls, through the C ABI: the
batched live pass (cdt_canary_sim_batch) and the batched Eq. 4
(cdt_drift_score_batch) must give every job's output bit for bit as
cdt_canary_sim / cdt_drift_score give it, over jobs of mixed shapes (one
and several chunks per block, ragged tails, empty jobs) and parameters;
one job of each batch is also checked against the oracle.  Jobs that share
a reference array (Eq. 4 reads a reference chunk once per unit of up to 8
of them) are covered with groups of 1 to 15 jobs, every unit size from 1 to
8 among them.  And the live pass's stream aid (cdt_canary_sim_stream)
writes exactly fp16(a)."""
import numpy as np
import pytest

import oracle
from paper_2607_19490_amd import inputs
from tests.gpu_util import announce, h_bits, rel_err, require_gpu, to_dev

pytestmark = pytest.mark.gpu

DRIFT_RTOL = 1e-5


@pytest.fixture(scope="module")
def gpu():
    return require_gpu()


DRIFT_SHAPES = [(16, 4, 4, 32768), (4, 8, 16, 256), (3, 5, 7, 264), (2, 3, 41, 1000),
                (0, 3, 4, 16), (2, 2, 0, 16), (1, 1, 130, 8192), (5, 2, 1, 8)]


def test_drift_score_batch_equals_single(gpu):
    torch, cdt = gpu
    announce("drift_score_batch over 8 jobs")
    jobs, host = [], []
    for k, shape in enumerate(DRIFT_SHAPES):
        S, C, T, H = shape
        a = inputs.ref_normal(shape, seed=200 + k, outlier_frac=0.01)
        h = inputs.live_near(a, seed=300 + k, rel=1e-3, flip_frac=0.001)
        hd, ad = to_dev(torch, h).view(torch.float16), to_dev(torch, a)
        sc = torch.full((C, S), -1.0, dtype=torch.float32, device="cuda")
        nd = torch.full((C, S, 2), -1.0, dtype=torch.float64, device="cuda")
        jobs.append((hd, ad, sc, nd if k % 2 == 0 else None))
        host.append((h, a))
    cdt.drift_score_batch(jobs)
    singles = []
    for hd, ad, sc, nd in jobs:
        nd1 = torch.empty((sc.shape[0], sc.shape[1], 2), dtype=torch.float64, device="cuda")
        singles.append((cdt.drift_score(hd, ad, num_den=nd1), nd1))
    torch.cuda.synchronize()
    for k, ((hd, ad, sc, nd), (want, nd1)) in enumerate(zip(jobs, singles)):
        assert torch.equal(sc, want), f"job {k} {DRIFT_SHAPES[k]}: scores differ"
        if nd is not None:
            assert torch.equal(nd, nd1), f"job {k}: sums differ"
    h, a = host[3]
    s64, _, _ = oracle.drift_score(h, a)
    assert rel_err(jobs[3][2].cpu().numpy(), s64) < DRIFT_RTOL


SIM_JOBS = [
    ((4, 8, 16, 256), dict(cfg_id=1, sigma_b=1e-3, mal_mask=1 << 2, tamper=1, eps=0.05)),
    ((8, 6, 9, 1000), dict(cfg_id=2, sigma_b=1e-4, mal_mask=1 << 4, tamper=2, flip_p=0.02)),
    ((2, 3, 41, 1000), dict(cfg_id=3, sigma_b=1e-2, mal_mask=1, tamper=4, scale=1.05)),
    ((16, 2, 40, 4096), dict(cfg_id=4, sigma_b=1e-3, mal_mask=(1 << 8) | (1 << 15), tamper=7,
                             eps=0.1, flip_p=0.1, scale=1.1)),
    ((0, 2, 3, 16), dict(cfg_id=5)),
    ((3, 5, 7, 264), dict(cfg_id=6, sigma_b=0.0, tamper_base=1, mal_mask=2, tamper=1, eps=0.2)),
]


@pytest.mark.parametrize("dist,mode", [(0, 0), (1, 1)], ids=["gauss_elementwise", "t3_block"])
def test_canary_sim_batch_equals_single(gpu, dist, mode):
    torch, cdt = gpu
    announce(f"canary_sim_batch dist={dist} mode={mode}")
    jobs, singles, host = [], [], []
    for k, (shape, kw) in enumerate(SIM_JOBS):
        S, C, T, H = shape
        kw = dict(kw, seed=0xABCDEF12345 + k, benign_dist=dist, benign_mode=mode)
        eps = kw.pop("eps", 0.0)
        ref = oracle.ref_synth(S, C, T, H, 40 + k, 0, oracle.outlier_gain(H, max(1, H // 100),
                                                                          20.0, 40 + k, 0))
        q, m = oracle.ref_stats(ref)
        ts, bs = oracle.block_scales(T, H, q, m, eps, kw.get("sigma_b", 1e-3))
        ref_d = to_dev(torch, ref)
        kw.update(bscale=to_dev(torch, bs), tscale=to_dev(torch, ts))
        h = torch.empty((S, C, T, H), dtype=torch.float16, device="cuda")
        jobs.append((ref_d, h, kw))
        singles.append(cdt.canary_sim(ref_d, **kw))
        host.append((ref, bs, ts, kw))
    cdt.canary_sim_batch(jobs)
    torch.cuda.synchronize()
    for k, ((ref_d, h, kw), want) in enumerate(zip(jobs, singles)):
        assert torch.equal(h.view(torch.int16), want.view(torch.int16)), f"job {k} differs"
    ref, bs, ts, kw = host[1]
    kw_o = {key: v for key, v in kw.items() if key not in ("bscale", "tscale")}
    want = oracle.canary_sim(ref, bscale=bs, tscale=ts, **kw_o)
    np.testing.assert_array_equal(h_bits(jobs[1][1]), want)


# Jobs over shared references, in the order given: consecutive jobs over one
# reference array form a group (Eq. 4: units of up to 8 jobs per reference
# read; the live pass: chunk-major below 8 jobs, job-major from 8 on); a
# reference that comes back after another one starts a new group.  Per
# entry: (reference index, shape index).  Groups of 1, 2, 3, 4, 5, 6, 9
# (8 + 1) and 15 (8 + 7) jobs, so every unit size from 1 to 8 is scored,
# ragged shapes among them.
SHARED_ORDER = ([(0, 0), (0, 0), (0, 0), (1, 1), (1, 1), (0, 0), (2, 2), (3, 3), (3, 3), (2, 2)]
                + [(1, 1)] * 6 + [(3, 3)] * 9 + [(0, 0)] * 4 + [(2, 2)] * 5 + [(1, 1)] * 15)
SHARED_SHAPES = [(16, 4, 4, 32768), (3, 5, 7, 264), (4, 8, 16, 256), (2, 3, 41, 1000)]


def test_drift_score_batch_shared_references(gpu):
    """Groups of jobs over one reference (several chunks per block, one chunk
    per block, ragged tails; groups of 1 to 15 jobs, a reference coming back
    after another) score every job as the single launch does, bit for bit."""
    torch, cdt = gpu
    announce("drift_score_batch over shared references")
    refs = []
    for k, shape in enumerate(SHARED_SHAPES):
        refs.append(to_dev(torch, inputs.ref_normal(shape, seed=500 + k, outlier_frac=0.01)))
    jobs = []
    for k, (r, si) in enumerate(SHARED_ORDER):
        S, C, T, H = SHARED_SHAPES[si]
        a = refs[r].cpu().numpy()
        h = to_dev(torch, inputs.live_near(a, seed=600 + k, rel=1e-3, flip_frac=0.001))
        sc = torch.full((C, S), -1.0, dtype=torch.float32, device="cuda")
        nd = torch.full((C, S, 2), -1.0, dtype=torch.float64, device="cuda")
        jobs.append((h.view(torch.float16), refs[r], sc, nd))
    cdt.drift_score_batch(jobs)
    for k, (hd, ad, sc, nd) in enumerate(jobs):
        nd1 = torch.empty_like(nd)
        want = cdt.drift_score(hd, ad, num_den=nd1)
        torch.cuda.synchronize()
        assert torch.equal(sc, want), f"job {k}: scores differ"
        assert torch.equal(nd, nd1), f"job {k}: sums differ"


def test_drift_score_batch_special_values(gpu):
    """Non-finite, extreme and degenerate operands in a group of 9 runs over
    one shared reference (a unit of 8 and one of 1; two chunks per block,
    the second ragged): fp16 infinities and NaNs in h, infinite reference
    elements, fp16 subnormals, values near the fp16 limit, and an all-zero
    reference block that one run matches exactly (score 0) and the others
    do not (+inf).  Every run's scores and sums equal the single launch's
    bit for bit, NaNs included."""
    torch, cdt = gpu
    announce("drift_score_batch special values")
    S, C, T, H = 6, 3, 5, 7000
    a = inputs.ref_normal((S, C, T, H), seed=31)
    a[3] *= np.float32(1e-6)
    a[4] *= np.float32(6e4 / np.abs(a[4]).max())
    a[5, 2] = 0.0
    a[2, 1, 4, 39] = np.inf
    a[5, 0, 0, 0] = np.inf
    ad = to_dev(torch, a)
    jobs = []
    for j in range(9):
        h = inputs.live_near(a, seed=40 + j, rel=1e-2)
        h[0, j % C, 1, 3 + j] = 0x7C00
        h[1, (j + 1) % C, 2, 5] = 0xFC00 if j % 2 else 0x7E00
        h[2, 1, 4, 39] = 0x7C00
        h[5, 2] = 0
        if j:
            h[5, 2, j % T, 17 * j] = 0x3C00  # 1.0 where the reference is 0
        sc = torch.full((C, S), -1.0, dtype=torch.float32, device="cuda")
        nd = torch.full((C, S, 2), -1.0, dtype=torch.float64, device="cuda")
        jobs.append((to_dev(torch, h).view(torch.float16), ad, sc, nd))
    cdt.drift_score_batch(jobs)
    for j, (hd, _, sc, nd) in enumerate(jobs):
        nd1 = torch.empty_like(nd)
        want = cdt.drift_score(hd, ad, num_den=nd1)
        torch.cuda.synchronize()
        assert torch.equal(sc.view(torch.int32), want.view(torch.int32)), f"run {j}: scores"
        assert torch.equal(nd.view(torch.int64), nd1.view(torch.int64)), f"run {j}: sums"
        s_ = sc.cpu().numpy()
        assert (s_[2, 5] == 0.0) if j == 0 else np.isposinf(s_[2, 5]), (j, s_[2, 5])
        assert np.isnan(s_[1, 2]) and np.all(np.isfinite(s_[:, 3:5])), j


@pytest.mark.parametrize("dist", [0, 1], ids=["gauss", "t3"])
def test_canary_sim_batch_special_references(gpu, dist):
    """A group of 9 runs (different tampers and scales) over one reference
    holding infinities, NaNs, values beyond the fp16 range and fp32
    subnormals: the batched live pass writes every run's activations bit
    for bit as one launch per run does, NaN payloads included."""
    torch, cdt = gpu
    announce(f"canary_sim_batch special references dist={dist}")
    S, C, T, H = 4, 3, 5, 4096  # 20480 elements per block: one partial live-pass chunk
    ref = inputs.ref_normal((S, C, T, H), seed=33)
    flat = ref.reshape(-1)
    specials = [np.inf, -np.inf, np.nan, 1e30, -7e4, 65519.0, 1e-40, -1e-45, 0.0, -0.0]
    flat[::997][:len(specials)] = np.array(specials, np.float32)
    ref[S // 2, 1, 2, :8] = np.float32(1e6)
    q, m = oracle.ref_stats(ref)
    ts, bs = oracle.block_scales(T, H, q, m, 0.05, 1e-2)
    rd, tsd, bsd = to_dev(torch, ref), to_dev(torch, ts), to_dev(torch, bs)
    jobs = []
    for j in range(9):
        kw = dict(seed=6, cfg_id=50 + j, sigma_b=1e-2, benign_dist=dist, mal_mask=1 << (j % S),
                  tamper=(1, 2, 4, 7)[j % 4], tscale=tsd, bscale=bsd, flip_p=0.25,
                  scale=1.5)
        jobs.append((rd, torch.empty((S, C, T, H), dtype=torch.float16, device="cuda"), kw))
    cdt.canary_sim_batch(jobs)
    for j, (_, hb, kw) in enumerate(jobs):
        one = cdt.canary_sim(rd, **kw)
        torch.cuda.synchronize()
        assert torch.equal(hb.view(torch.int16), one.view(torch.int16)), f"run {j}"
    bits = h_bits(jobs[0][1])
    assert np.any((bits & 0x7C00) == 0x7C00)  # the specials reached the output


def test_drift_read_stream_batch_writes_nothing(gpu):
    """The batched Eq. 4's read-stream aid runs the same launch's loads over
    mixed groups (units of 8, 3 and 1; one and several chunks per block)
    and leaves every score and sum untouched."""
    torch, cdt = gpu
    announce("drift_read_stream_batch")
    jobs = []
    for k, (r, si) in enumerate(SHARED_ORDER[:12] + [(2, 2)] * 8):
        S, C, T, H = SHARED_SHAPES[si]
        a = to_dev(torch, inputs.ref_normal((S, C, T, H), seed=700 + r))
        h = to_dev(torch, inputs.live_near(a.cpu().numpy(), seed=800 + k, rel=1e-3))
        jobs.append((h.view(torch.float16), a,
                     torch.full((C, S), -1.0, dtype=torch.float32, device="cuda"),
                     torch.full((C, S, 2), -1.0, dtype=torch.float64, device="cuda")))
    b = cdt.drift_batch(jobs)
    cdt.drift_read_stream_batch(b)
    torch.cuda.synchronize()
    for k, (_, _, sc, nd) in enumerate(jobs):
        assert bool((sc == -1.0).all()) and bool((nd == -1.0).all()), k
    cdt.drift_score_batch(b)  # the same batch object still scores
    torch.cuda.synchronize()
    assert all(bool((sc >= 0).all()) for _, _, sc, _ in jobs)


def test_batches_share_only_identical_layouts(gpu):
    """Jobs that pass one reference array in different shapes with the same
    chunk count (and even different element counts) must not share its
    reads: each is scored, and generated, in its own layout."""
    torch, cdt = gpu
    announce("batches over one reference array in different shapes")
    pairs = [((1, 2, 4, 16384), (2, 2, 2, 16384)),   # 4 chunks each, same size
             ((1, 1, 5, 8192), (2, 1, 1, 8192))]      # 2 chunks each, sizes differ
    for sa, sb in pairs:
        na = int(np.prod(sa))
        flat = to_dev(torch, inputs.ref_normal((na,), seed=900 + na, outlier_frac=0.01))
        ra = flat.view(*sa)
        rb = flat[:int(np.prod(sb))].view(*sb)
        jobs = []
        for k, (shape, ref) in enumerate(((sa, ra), (sb, rb))):
            S, C, T, H = shape
            h = to_dev(torch, inputs.live_near(ref.cpu().numpy(), seed=910 + k, rel=1e-3))
            sc = torch.full((C, S), -1.0, dtype=torch.float32, device="cuda")
            jobs.append((h.view(torch.float16), ref, sc, None))
        cdt.drift_score_batch(jobs)
        for hd, ad, sc, _ in jobs:
            want = cdt.drift_score(hd, ad)
            torch.cuda.synchronize()
            assert torch.equal(sc, want), (sa, sb)
        sims = []
        for k, (shape, ref) in enumerate(((sa, ra), (sb, rb))):
            kw = dict(seed=5, cfg_id=20 + k, sigma_b=1e-3)
            sims.append((ref, torch.empty(shape, dtype=torch.float16, device="cuda"), kw))
        cdt.canary_sim_batch(sims)
        for ref, h, kw in sims:
            want = cdt.canary_sim(ref, **kw)
            torch.cuda.synchronize()
            assert torch.equal(h.view(torch.int16), want.view(torch.int16)), (sa, sb)


@pytest.mark.parametrize("dist", [0, 1], ids=["gauss", "t3"])
def test_canary_sim_batch_shared_references(gpu, dist):
    """The live pass of groups of runs over one reference (different
    configurations, attackers and tampers per run) equals one launch per
    run, bit for bit."""
    torch, cdt = gpu
    announce(f"canary_sim_batch over shared references dist={dist}")
    refs, scales = [], []
    for k, (S, C, T, H) in enumerate(SHARED_SHAPES):
        ref = oracle.ref_synth(S, C, T, H, 70 + k, 0, oracle.outlier_gain(H, max(1, H // 100),
                                                                          20.0, 70 + k, 0))
        q, m = oracle.ref_stats(ref)
        ts, _ = oracle.block_scales(T, H, q, m, 0.05, 1e-3)
        refs.append(to_dev(torch, ref))
        scales.append(to_dev(torch, ts))
    jobs, singles = [], []
    for k, (r, si) in enumerate(SHARED_ORDER):
        S, C, T, H = SHARED_SHAPES[si]
        kw = dict(seed=77, cfg_id=10 + k, sigma_b=1e-3, benign_dist=dist,
                  mal_mask=1 << (k % S), tamper=(1, 2, 4, 7)[k % 4], tscale=scales[r],
                  flip_p=0.05, scale=1.05)
        h = torch.empty((S, C, T, H), dtype=torch.float16, device="cuda")
        jobs.append((refs[r], h, kw))
        singles.append(cdt.canary_sim(refs[r], **kw))
    cdt.canary_sim_batch(jobs)
    torch.cuda.synchronize()
    for k, ((_, h, _), want) in enumerate(zip(jobs, singles)):
        assert torch.equal(h.view(torch.int16), want.view(torch.int16)), f"job {k} differs"


def test_canary_sim_batch_rejects_mixed_noise(gpu):
    torch, cdt = gpu
    ref = torch.zeros((2, 2, 2, 16), dtype=torch.float32, device="cuda")
    h = torch.empty((2, 2, 2, 16), dtype=torch.float16, device="cuda")
    with pytest.raises(cdt.CdtError):
        cdt.canary_sim_batch([(ref, h, dict(seed=0, cfg_id=0)),
                              (ref, h, dict(seed=0, cfg_id=1, benign_dist=1))])


@pytest.mark.parametrize("shape", [(4, 8, 16, 256), (3, 5, 41, 1000), (2, 2, 9, 8000)])
def test_canary_sim_stream_is_fp16_of_reference(gpu, shape):
    torch, cdt = gpu
    announce(f"canary_sim_stream {shape}")
    a = inputs.ref_normal(shape, seed=7, outlier_frac=0.05) * np.float32(300.0)
    ad = to_dev(torch, a)
    h = cdt.canary_sim_stream(ad)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(h_bits(h), oracle.f16_rne(a))
