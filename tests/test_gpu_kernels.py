"""GPU parity of every libcdt kernel against the CPU oracle, through the C ABI.

Bar: bit-exact for generated activations (fp32 references, fp16 live
activations), outlier channels and AUROC counts; 1e-5 relative for drift
scores (Eq. 4); the fp64 sums within the bound of two n-term fp64 sums.  Shapes span several
chunks, ragged tails, single-element blocks and empty inputs.
"""

import numpy as np
import pytest

import oracle
from paper_2607_19490_amd import inputs
from tests.gpu_util import announce, h_bits, rel_err, require_gpu, to_dev, ulp_diff_f32

pytestmark = pytest.mark.gpu

DRIFT_RTOL = 1e-5  # tolerance stated for drift scores

# (S, C, T, H): tiny, ragged (T*H not a multiple of any chunk), multi-chunk
# with a partial last chunk, and single-group blocks
SHAPES = [(4, 8, 16, 256), (3, 5, 7, 264), (2, 3, 41, 1000), (5, 2, 1, 8), (1, 1, 130, 8192)]

# Blocks of 3000 and 9000 eight-element groups: a workgroup step of 2048
# groups that is whole, then one that is partial, inside one chunk; and two
# whole chunks followed by a chunk shorter than one step.  The whole steps
# read the fp32 reference in contiguous runs and exchange quads across lanes;
# the partial ones read it directly.
EXCHANGE_TAIL_SHAPES = [(2, 3, 5, 4800), (1, 2, 9, 8000)]


@pytest.fixture(scope="module")
def gpu():
    return require_gpu()


# ----------------------------------------------------------------------------
# generator
# ----------------------------------------------------------------------------
@pytest.mark.parametrize("H,n_out", [(8, 1), (256, 0), (264, 3), (4096, 41), (8192, 82)])
def test_outlier_gain(gpu, H, n_out):
    torch, cdt = gpu
    announce(f"outlier_gain H={H} n_out={n_out}")
    g = cdt.outlier_gain(H, n_out, 20.0, 7, 3)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(g.cpu().numpy(), oracle.outlier_gain(H, n_out, 20.0, 7, 3))


@pytest.mark.parametrize("shape", SHAPES)
def test_ref_synth(gpu, shape):
    torch, cdt = gpu
    S, C, T, H = shape
    announce(f"ref_synth {shape}")
    gain = oracle.outlier_gain(H, max(1, H // 100), 20.0, 1, 2)
    ref = cdt.ref_synth(S, C, T, H, 11, 2, to_dev(torch, gain))
    torch.cuda.synchronize()
    np.testing.assert_array_equal(ref.cpu().numpy(), oracle.ref_synth(S, C, T, H, 11, 2, gain))


def test_fp16_conversion_exhaustive(gpu):
    """Every fp32 bit pattern, fed through the live pass with zero noise
    (block mode, scale 0: v = a + 0 z), must come out as its IEEE
    round-to-nearest-even fp16.  All 2^32 inputs are checked against torch's
    device conversion (a library routine), and a sample of each slab against
    numpy's.  Zeros are compared by magnitude, since a + (+-0) can flip a
    zero's sign; NaN is compared by class."""
    torch, cdt = gpu
    n, H = 1 << 28, 8192
    T = n // H
    bs = torch.zeros((1, 1), dtype=torch.float32, device="cuda")
    h = torch.empty((1, 1, T, H), dtype=torch.float16, device="cuda")
    rng = np.random.default_rng(0)
    for start in range(0, 1 << 32, n):
        announce(f"fp16 conversion inputs [{start:#x}, {start + n:#x})")
        idx = torch.arange(start, start + n, dtype=torch.int64, device="cuda")
        x = torch.where(idx >= 1 << 31, idx - (1 << 32), idx).to(torch.int32)
        del idx
        x = x.view(torch.float32).view(1, 1, T, H)
        cdt.canary_sim(x, out=h, seed=1, cfg_id=0, benign_mode=1, sigma_b=0.0, bscale=bs)
        got = h.view(torch.int16).reshape(-1)
        want = x.to(torch.float16).view(torch.int16).reshape(-1)
        same = got == want
        zeros = ((got & 0x7FFF) == 0) & ((want & 0x7FFF) == 0)
        nans = torch.isnan(x.reshape(-1)) & torch.isnan(h.reshape(-1))
        bad = int((~(same | zeros | nans)).sum())
        assert bad == 0, f"{bad} inputs in [{start:#x}, {start + n:#x}) differ"
        pick = np.sort(rng.integers(0, n, 1 << 14))
        xs = x.reshape(-1)[torch.from_numpy(pick).cuda()].cpu().numpy()
        gs = got[torch.from_numpy(pick).cuda()].cpu().numpy().view(np.uint16)
        with np.errstate(over="ignore"):  # values past the fp16 range round to inf
            ws = xs.astype(np.float16).view(np.uint16)
        ok = (gs == ws) | (((gs & 0x7FFF) == 0) & ((ws & 0x7FFF) == 0)) | np.isnan(xs)
        assert ok.all()
        del x, got, want, same, zeros, nans
    torch.cuda.synchronize()


@pytest.mark.parametrize("shape", SHAPES + EXCHANGE_TAIL_SHAPES)
def test_ref_stats_and_block_scales(gpu, shape):
    torch, cdt = gpu
    S, C, T, H = shape
    announce(f"ref_stats {shape}")
    ref = oracle.ref_synth(S, C, T, H, 5, 0, oracle.outlier_gain(H, 1, 20.0, 5, 0))
    q, m = cdt.ref_stats(to_dev(torch, ref))
    torch.cuda.synchronize()
    q_o, m_o = oracle.ref_stats(ref)
    tol = max(1e-14, 2 * T * H * 2.0**-53)  # two fp64 sums of n non-negative terms
    assert rel_err(q.cpu().numpy(), q_o) < tol
    assert rel_err(m.cpu().numpy(), m_o) < tol
    # block scales from identical fp64 statistics: same fp32 result
    ts, bs = cdt.block_scales(to_dev(torch, q_o), to_dev(torch, m_o), T, H, 0.05, 2e-3)
    torch.cuda.synchronize()
    ts_o, bs_o = oracle.block_scales(T, H, q_o, m_o, 0.05, 2e-3)
    assert ulp_diff_f32(ts.cpu().numpy(), ts_o).max() == 0
    assert ulp_diff_f32(bs.cpu().numpy(), bs_o).max() == 0


SIM_CASES = {
    "gauss_add": dict(sigma_b=1e-3, tamper=1, eps=0.05),
    "t3_flip": dict(benign_dist=1, sigma_b=2e-2, tamper=2, flip_p=0.3),
    "block_scale": dict(benign_mode=1, sigma_b=2e-3, tamper=4, scale=1.05),
    "mixed": dict(sigma_b=1e-4, tamper=7, eps=0.1, flip_p=0.1, scale=1.1),
    "mixed_clean": dict(sigma_b=1e-2, tamper=7, eps=0.02, flip_p=0.02, scale=1.02,
                        tamper_base=1),
    "full_flip": dict(benign_mode=1, sigma_b=2e-3, tamper=2, flip_p=1.0),
    "t3_block_add": dict(benign_mode=1, benign_dist=1, sigma_b=0.1, tamper=1, eps=0.2),
    "no_noise": dict(sigma_b=0.0, tamper=0),
}


@pytest.mark.parametrize("case", sorted(SIM_CASES))
@pytest.mark.parametrize("shape", SHAPES[:3] + [(64, 2, 3, 16), (1, 2, 9, 8000), (1, 1, 130, 8192)])
def test_canary_sim(gpu, case, shape):
    torch, cdt = gpu
    S, C, T, H = shape
    kw = dict(SIM_CASES[case])
    announce(f"canary_sim {case} {shape}")
    eps = kw.pop("eps", 0.0)
    gain = oracle.outlier_gain(H, max(1, H // 100), 20.0, 3, 1)
    ref = oracle.ref_synth(S, C, T, H, 3, 1, gain)
    q, m = oracle.ref_stats(ref)
    ts, bs = oracle.block_scales(T, H, q, m, eps, kw.get("sigma_b", 0.0))
    mal = (1 << (S // 2)) | (1 << (S - 1))  # two colluders
    h = cdt.canary_sim(to_dev(torch, ref), seed=0xDEADBEEF12345, cfg_id=77, mal_mask=mal,
                       bscale=to_dev(torch, bs), tscale=to_dev(torch, ts), **kw)
    torch.cuda.synchronize()
    want = oracle.canary_sim(ref, seed=0xDEADBEEF12345, cfg_id=77, mal_mask=mal, bscale=bs,
                             tscale=ts, **kw)
    got = h_bits(h)
    bad = int((got != want).sum())
    assert bad == 0, f"{bad} of {want.size} fp16 words differ"


# ----------------------------------------------------------------------------
# Eq. 4
# ----------------------------------------------------------------------------
@pytest.mark.parametrize("shape", SHAPES + [(16, 4, 4, 32768)] + EXCHANGE_TAIL_SHAPES)
def test_drift_score(gpu, shape):
    torch, cdt = gpu
    S, C, T, H = shape
    announce(f"drift_score {shape}")
    a = inputs.ref_normal(shape, seed=S * 1000 + H, outlier_frac=0.01)
    h = inputs.live_near(a, seed=7, rel=1e-3, flip_frac=0.001)
    nd = torch.empty((C, S, 2), dtype=torch.float64, device="cuda")
    sc = cdt.drift_score(to_dev(torch, h).view(torch.float16), to_dev(torch, a), num_den=nd)
    torch.cuda.synchronize()
    s64, s32, nd_o = oracle.drift_score(h, a)
    assert rel_err(sc.cpu().numpy(), s64) < DRIFT_RTOL
    # both sides add n non-negative fp64 terms (in different orders): each
    # sum is within (n - 1) 2^-53 of the exact one, relative
    assert rel_err(nd.cpu().numpy(), nd_o) < max(1e-14, 2 * T * H * 2.0**-53)
    assert ulp_diff_f32(sc.cpu().numpy(), s32).max() <= 1


@pytest.mark.parametrize("shape", [(4, 8, 16, 256)] + EXCHANGE_TAIL_SHAPES)
def test_drift_read_stream(gpu, shape):
    """The compute-free read of Eq. 4's stream runs on ragged shapes, leaves
    its inputs untouched, and a drift_score after it (same workspace) still
    matches the oracle."""
    torch, cdt = gpu
    S, C, T, H = shape
    announce(f"drift_read_stream {shape}")
    a = inputs.ref_normal(shape, seed=11, outlier_frac=0.01)
    h = inputs.live_near(a, seed=12, rel=1e-3, flip_frac=0.001)
    h_d, a_d = to_dev(torch, h).view(torch.float16), to_dev(torch, a)
    ws = cdt.workspace(S, C, T, H, a_d)
    cdt.drift_read_stream(h_d, a_d, ws=ws)
    sc = cdt.drift_score(h_d, a_d, ws=ws)
    torch.cuda.synchronize()
    assert np.array_equal(h_d.view(torch.int16).cpu().numpy().view(np.uint16), h)
    assert np.array_equal(a_d.cpu().numpy(), a)
    s64, _, _ = oracle.drift_score(h, a)
    assert rel_err(sc.cpu().numpy(), s64) < DRIFT_RTOL


def test_drift_exact_special_cases(gpu):
    """h = a gives 0, h = -a gives 2, h = 2a gives 1, h = 0 gives 1, exactly."""
    torch, cdt = gpu
    S, C, T, H = 4, 3, 33, 72
    announce("drift exact cases")
    a16 = inputs.fp16_bits(inputs.ref_normal((1, C, T, H), seed=1))
    a = a16.view(np.float16).astype(np.float32)
    ref = np.concatenate([a] * S)
    h = np.concatenate([a16, inputs.fp16_bits(-a), inputs.fp16_bits(2 * a),
                        np.zeros_like(a16)])
    sc = cdt.drift_score(to_dev(torch, h).view(torch.float16), to_dev(torch, ref))
    torch.cuda.synchronize()
    got = sc.cpu().numpy()
    np.testing.assert_array_equal(got, np.tile(np.array([0.0, 2.0, 1.0, 1.0], np.float32), (C, 1)))


def test_drift_degenerate_and_empty(gpu):
    torch, cdt = gpu
    announce("drift degenerate")
    # all-zero reference blocks: 0 when h = 0 too, +inf otherwise
    ref = np.zeros((2, 2, 1, 8), np.float32)
    h = np.zeros((2, 2, 1, 8), np.uint16)
    h[1, 0, 0, 3] = inputs.fp16_bits(np.float32(0.5))
    sc = cdt.drift_score(to_dev(torch, h).view(torch.float16), to_dev(torch, ref))
    torch.cuda.synchronize()
    got = sc.cpu().numpy()
    assert got[0, 1] == np.inf and got[0, 0] == 0 and got[1, 0] == 0 and got[1, 1] == 0
    # empty blocks (T = 0) score 0; empty shard/canary sets write nothing
    sc = cdt.drift_score(torch.empty((3, 2, 0, 16), dtype=torch.float16, device="cuda"),
                         torch.empty((3, 2, 0, 16), dtype=torch.float32, device="cuda"))
    torch.cuda.synchronize()
    np.testing.assert_array_equal(sc.cpu().numpy(), np.zeros((2, 3), np.float32))
    sc = cdt.drift_score(torch.empty((0, 2, 4, 16), dtype=torch.float16, device="cuda"),
                         torch.empty((0, 2, 4, 16), dtype=torch.float32, device="cuda"))
    torch.cuda.synchronize()
    assert sc.shape == (2, 0)


def test_drift_special_values(gpu):
    """Non-finite and extreme operands, against the oracle: fp16 infinities
    and NaNs in h, an infinite reference element, fp16 subnormals (tiny
    activations, widened exactly), and values at the fp16 limit.  Scores
    agree bit for bit in class (inf, NaN) and within the drift tolerance
    otherwise."""
    torch, cdt = gpu
    S, C, T, H = 6, 2, 5, 40
    announce("drift special values")
    a = inputs.ref_normal((S, C, T, H), seed=21)
    a[3] *= np.float32(1e-6)                 # tiny: h in the fp16 subnormal range
    a[4] *= np.float32(6e4 / np.abs(a[4]).max())  # near the fp16 limit
    h = inputs.live_near(a, seed=22, rel=1e-2)
    h[0, 0, 1, 3] = 0x7C00                   # +inf
    h[0, 1, 2, 5] = 0xFC00                   # -inf
    h[1, 0, 0, 0] = 0x7E00                   # NaN
    h[2, 1, 4, 39] = 0x7C00
    a[2, 1, 4, 39] = np.inf                  # inf - inf = NaN
    a[5, 0, 0, 0] = np.inf                   # infinite reference element
    sc = cdt.drift_score(to_dev(torch, h).view(torch.float16), to_dev(torch, a))
    torch.cuda.synchronize()
    got = sc.cpu().numpy().astype(np.float64)
    want, _, _ = oracle.drift_score(h, a)
    np.testing.assert_array_equal(np.isnan(got), np.isnan(want))
    np.testing.assert_array_equal(np.isposinf(got), np.isposinf(want))
    fin = np.isfinite(want)
    assert np.all(np.abs(got[fin] - want[fin]) <= DRIFT_RTOL * np.abs(want[fin]))
    # the planted cases ([C][S]): +inf and -inf in h give +inf; NaN in h,
    # inf - inf, and an infinite reference (D and R both infinite) give NaN
    assert np.isposinf(want[0, 0]) and np.isposinf(want[1, 0])
    assert np.isnan(want[0, 1]) and np.isnan(want[1, 2]) and np.isnan(want[0, 5])
    assert np.all(np.isfinite(want[:, 3:5]))  # subnormal and near-limit blocks


def test_nan_element_ranks_most_suspicious(gpu):
    """A malicious stage that returns benign-looking activations except for a
    single NaN element per block: its mismatch is NaN, which ranks above
    every number, so Eq. 5 counts it above every benign stage (AUROC 1.0;
    ranking NaN lowest would give 0.0 and let the stage escape).  Scores,
    detector, control and pooled counts against the oracle on the same h."""
    torch, cdt = gpu
    S, C, T, H = 8, 16, 16, 256
    mal = 5
    announce("NaN element in the malicious stage")
    ref = inputs.ref_normal((S, C, T, H), seed=41)
    h = inputs.live_near(ref, seed=42, rel=1e-3)  # every stage benign-looking
    for c in range(C):
        h[mal, c, c % T, (7 * c) % H] = 0x7E00  # one NaN element per canary
    sc = cdt.drift_score(to_dev(torch, h).view(torch.float16), to_dev(torch, ref))
    counts, pooled, _ = cdt.auroc([(S, C, 0, 1 << mal, 9)], sc.view(-1), seed=2, flags=3)
    torch.cuda.synchronize()
    want64, want32, _ = oracle.drift_score(h, ref)
    got = sc.cpu().numpy()
    assert np.isnan(got[:, mal]).all() and np.isnan(want64[:, mal]).all()
    ben = [s for s in range(S) if s != mal]
    assert rel_err(got[:, ben], want64[:, ben]) < DRIFT_RTOL
    want_c, want_p = oracle.auroc_config(want32, 1 << mal, seed=2, cfg_id=9, flags=3)
    np.testing.assert_array_equal(cdt.u64(counts)[0], want_c)
    np.testing.assert_array_equal(cdt.u64(pooled)[0], want_p)
    c = cdt.u64(counts)[0]
    assert int(c[0]) == int(c[2]) == C * (S - 1) and int(c[1]) == 0
    p = cdt.u64(pooled)[0]
    assert int(p[0]) == int(p[2])


@pytest.mark.parametrize("kw", [dict(sigma_b=1e-2), dict(benign_mode=1, sigma_b=1e-2),
                                dict(sigma_b=1e-2, tamper=7, eps=0.05, flip_p=0.5, scale=1.5)],
                         ids=["elementwise", "block", "mixed_tamper"])
def test_canary_sim_special_references(gpu, kw):
    """References holding infinities, NaNs, values beyond the fp16 range and
    fp32 subnormals go through the live pass as the oracle takes them: every
    output that is a number or an infinity matches bit for bit, NaNs match
    as NaNs."""
    torch, cdt = gpu
    S, C, T, H = 4, 2, 3, 64
    announce(f"canary_sim special references {kw}")
    kw = dict(kw)
    eps = kw.pop("eps", 0.0)
    ref = inputs.ref_normal((S, C, T, H), seed=31)
    flat = ref.reshape(-1)
    specials = [np.inf, -np.inf, np.nan, 1e30, -7e4, 65519.0, 1e-40, -1e-45, 0.0, -0.0]
    flat[:: 97][: len(specials)] = np.array(specials, np.float32)
    ref[S // 2, 1, 2, :8] = np.float32(1e6)     # a whole row beyond fp16 on the tampered shard
    q, m = oracle.ref_stats(ref)
    ts, bs = oracle.block_scales(T, H, q, m, eps, kw.get("sigma_b", 0.0))
    mal = 1 << (S // 2)
    h = cdt.canary_sim(to_dev(torch, ref), seed=4, cfg_id=2, mal_mask=mal,
                       bscale=to_dev(torch, bs), tscale=to_dev(torch, ts), **kw)
    torch.cuda.synchronize()
    got = h_bits(h)
    want = oracle.canary_sim(ref, seed=4, cfg_id=2, mal_mask=mal, bscale=bs, tscale=ts, **kw)
    nan_g = (got & 0x7C00) == 0x7C00
    nan_g &= (got & 0x3FF) != 0
    nan_w = ((want & 0x7C00) == 0x7C00) & ((want & 0x3FF) != 0)
    np.testing.assert_array_equal(nan_g, nan_w)
    np.testing.assert_array_equal(got[~nan_w], want[~nan_w])
    assert nan_w.any() and np.any(want == 0x7C00)  # the specials reached the output


def test_drift_deterministic(gpu):
    """No atomics: two runs give bitwise-equal scores and sums."""
    torch, cdt = gpu
    announce("drift determinism")
    shape = (8, 16, 64, 4096)
    a = to_dev(torch, inputs.ref_normal(shape, seed=3, outlier_frac=0.01))
    h = to_dev(torch, inputs.live_near(a.cpu().numpy(), seed=4)).view(torch.float16)
    nd1 = torch.empty((16, 8, 2), dtype=torch.float64, device="cuda")
    nd2 = torch.empty_like(nd1)
    s1 = cdt.drift_score(h, a, num_den=nd1)
    s2 = cdt.drift_score(h, a, num_den=nd2)
    torch.cuda.synchronize()
    assert torch.equal(s1, s2) and torch.equal(nd1, nd2)


# ----------------------------------------------------------------------------
# Eqs. 5-6
# ----------------------------------------------------------------------------
def _auroc_batch():
    """A batch of score tables: ties, NaNs, S = 1 and 64, colluders, C = 0."""
    cases = [
        (8, 32, (4,), dict(gap=0.3)),
        (16, 64, (8,), dict(gap=0.0, tie_levels=6)),
        (64, 256, (3, 17, 40, 63), dict(gap=0.05, nan_frac=0.02)),
        (32, 32, (16,), dict(gap=1.0)),
        (1, 5, (0,), dict()),
        (5, 0, (2,), dict()),
        (12, 100, (5,), dict(gap=-0.2, tie_levels=3)),
        (4, 7, (), dict()),
        (64, 16, tuple(range(64)), dict()),
    ]
    tables, cfgs, off = [], [], 0
    for k, (S, C, pos, kw) in enumerate(cases):
        t = inputs.scores(C, S, seed=100 + k, mal=pos, **kw)
        mask = 0
        for s in pos:
            mask |= 1 << s
        tables.append(t)
        cfgs.append((S, C, off, mask, 1000 + k))
        off += t.size
    return tables, cfgs


@pytest.mark.parametrize("flags", [0, 1, 3, 7])
def test_auroc_counts(gpu, flags):
    torch, cdt = gpu
    announce(f"auroc flags={flags}")
    tables, cfgs = _auroc_batch()
    flat = np.concatenate([t.ravel() for t in tables]).astype(np.float32)
    counts, pooled, _ = cdt.auroc(cfgs, to_dev(torch, flat), seed=42, flags=flags)
    torch.cuda.synchronize()
    got = cdt.u64(counts)
    got_p = cdt.u64(pooled) if pooled is not None else None
    for g, (t, (S, C, off, mask, cid)) in enumerate(zip(tables, cfgs)):
        want, want_p = oracle.auroc_config(t, mask, seed=42, cfg_id=cid, flags=flags)
        np.testing.assert_array_equal(got[g], want, err_msg=f"cfg {g} S={S} C={C}")
        if flags & 2:
            np.testing.assert_array_equal(got_p[g], want_p, err_msg=f"pooled cfg {g}")


@pytest.mark.parametrize("flags,base", [(1 | 8, 0), (0, 0), (1 | 4 | 8, 0), (1 | 8, 4000)])
def test_auroc_canaries(gpu, flags, base):
    """Eq. 5 per canary, bit for bit against the oracle on every canary of
    the batch (ties, NaNs, S = 1 and 64, colluders, C = 0, every stage
    positive, canary_base > 0), and summed over canaries equal to
    cdt_auroc's counts."""
    torch, cdt = gpu
    announce(f"auroc per canary flags={flags} base={base}")
    tables, cfgs = _auroc_batch()
    cfgs = [c + (base,) for c in cfgs]
    flat = to_dev(torch, np.concatenate([t.ravel() for t in tables]).astype(np.float32))
    per = cdt.auroc_canaries(cfgs, flat, seed=42, flags=flags)
    counts, _, rb = cdt.auroc(cfgs, flat, seed=42, flags=flags)
    torch.cuda.synchronize()
    got = per.cpu().numpy().view(np.uint32)
    assert got.shape == (sum(c[1] for c in cfgs), 6)
    tot, tot_b = cdt.u64(counts), cdt.u64(rb) if rb is not None else None
    o = 0
    for g, (t, (S, C, off, mask, cid, cb)) in enumerate(zip(tables, cfgs)):
        want = oracle.auroc_canaries(t, mask, seed=42, cfg_id=cid, canary_base=cb, flags=flags)
        np.testing.assert_array_equal(got[o:o + C], want, err_msg=f"cfg {g} S={S} C={C}")
        s = got[o:o + C].astype(np.uint64).sum(axis=0)
        assert s[0] == tot[g][0] and s[1] == tot[g][1], g
        assert s[2] == tot[g][3] and s[3] == tot[g][4], g
        if flags & 8:
            assert s[4] == tot_b[g][0] and s[5] == tot_b[g][1], g
        o += C


# Pooled sizes C*S padded to P2 = 64 .. 16384: every width of the pooled
# sort (1, 2, 4, 8 and 16 elements per thread), lengths just off a power of
# two, many positives, ties and NaNs.
POOLED_CASES = [(7, 9, (3,), dict(tie_levels=4)), (3, 43, (1,), dict(nan_frac=0.05)),
                (33, 31, (0, 16, 32), dict(gap=0.1)), (5, 205, (2,), dict(tie_levels=7)),
                (16, 150, (8,), dict(gap=0.02, nan_frac=0.01)),
                (48, 120, tuple(range(0, 48, 5)), dict(tie_levels=40)),
                (64, 200, tuple(range(1, 64, 3)), dict(gap=-0.05, tie_levels=100, nan_frac=0.01))]


@pytest.mark.parametrize("case", range(len(POOLED_CASES)))
def test_auroc_pooled_widths(gpu, case):
    torch, cdt = gpu
    S, C, pos, kw = POOLED_CASES[case]
    announce(f"auroc pooled {S}x{C}")
    t = inputs.scores(C, S, seed=500 + case, mal=pos, **kw)
    mask = 0
    for s_ in pos:
        mask |= 1 << s_
    counts, pooled, _ = cdt.auroc([(S, C, 0, mask, 7 + case)], to_dev(torch, t.ravel()),
                                  seed=5, flags=3)
    torch.cuda.synchronize()
    want, want_p = oracle.auroc_config(t, mask, seed=5, cfg_id=7 + case, flags=3)
    np.testing.assert_array_equal(cdt.u64(counts)[0], want)
    np.testing.assert_array_equal(cdt.u64(pooled)[0], want_p)


def test_auroc_pooled_at_capacity(gpu):
    torch, cdt = gpu
    announce("auroc pooled 64x256")
    S, C = 64, 256
    t = inputs.scores(C, S, seed=9, mal=(10, 20), gap=0.01, tie_levels=50)
    counts, pooled, _ = cdt.auroc([(S, C, 0, (1 << 10) | (1 << 20), 3)], to_dev(torch, t.ravel()),
                               seed=1, flags=3)
    torch.cuda.synchronize()
    want, want_p = oracle.auroc_config(t, (1 << 10) | (1 << 20), seed=1, cfg_id=3, flags=3)
    np.testing.assert_array_equal(cdt.u64(counts)[0], want)
    np.testing.assert_array_equal(cdt.u64(pooled)[0], want_p)


@pytest.mark.parametrize("kw", [dict(sigma_b=1e-3), dict(benign_dist=1, sigma_b=2e-2),
                                dict(benign_mode=1, sigma_b=2e-3), dict(sigma_b=0.1, tamper_base=1),
                                dict(sigma_b=1e-2, redraw=True)],
                         ids=["gauss", "t3", "block", "clean", "redraw"])
@pytest.mark.parametrize("shape", SHAPES[:3] + [(1, 1, 130, 8192)])
def test_tamper_scale_exact(gpu, kw, shape):
    """Exact-norm Gaussian tamper scale (Section 3.2): the two fp64 norms
    within the bound of n-term fp64 sums, the fp32 scale within one ulp."""
    torch, cdt = gpu
    S, C, T, H = shape
    announce(f"tamper_scale_exact {kw} {shape}")
    ref = oracle.ref_synth(S, C, T, H, 6, 0, oracle.outlier_gain(H, 1, 20.0, 6, 0))
    q, m = oracle.ref_stats(ref)
    _, bs = oracle.block_scales(T, H, q, m, 0.0, kw.get("sigma_b", 0.0))
    norms = torch.empty((S, C, 2), dtype=torch.float64, device="cuda")
    ts = cdt.tamper_scale_exact(to_dev(torch, ref), 0.05, norms=norms, bscale=to_dev(torch, bs),
                                seed=8, cfg_id=21, **kw)
    torch.cuda.synchronize()
    ts_o, norms_o = oracle.tamper_scale_exact(ref, 0.05, seed=8, cfg_id=21, bscale=bs, **kw)
    assert rel_err(norms.cpu().numpy(), norms_o) < max(1e-14, 2 * T * H * 2.0**-53)
    d = ulp_diff_f32(ts.cpu().numpy(), ts_o)
    assert d.max() <= 1 and (d == 0).mean() > 0.9
