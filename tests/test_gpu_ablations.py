"""GPU parity of the reference conditions and ablations (Sections 4.4-4.5)
against the CPU oracle, through the C ABI: the independent benign redraw
(bit-exact), Eq. 4 against an fp16 reference (1e-5), the cosine mismatch
(1e-5 plus the fp64 rounding bound of its sums), and the random-baseline
counts (bit-exact)."""

import numpy as np
import pytest

import oracle
from paper_2607_19490_amd import inputs
from tests.gpu_util import announce, h_bits, rel_err, require_gpu, to_dev

pytestmark = pytest.mark.gpu

SHAPES = [(4, 8, 16, 256), (3, 5, 7, 264), (2, 3, 41, 1000), (5, 2, 1, 8), (1, 1, 130, 8192),
          (2, 3, 5, 4800)]
DRIFT_RTOL = 1e-5


@pytest.fixture(scope="module")
def gpu():
    return require_gpu()


def _f16(x):
    return np.asarray(x, np.float32).astype(np.float16).view(np.uint16)


def _h(bits):
    return np.asarray(bits, np.uint16).view(np.float16).astype(np.float64)


@pytest.mark.parametrize("kw", [dict(sigma_b=1e-3), dict(benign_dist=1, sigma_b=2e-2),
                                dict(benign_mode=1, sigma_b=2e-3),
                                dict(sigma_b=1e-3, tamper=7, eps=0.05, flip_p=0.1, scale=1.1)],
                         ids=["gauss", "t3", "block", "mixed"])
@pytest.mark.parametrize("shape", SHAPES[:3])
def test_canary_sim_redraw(gpu, kw, shape):
    torch, cdt = gpu
    S, C, T, H = shape
    kw = dict(kw)
    eps = kw.pop("eps", 0.0)
    announce(f"canary_sim redraw {kw} {shape}")
    ref = oracle.ref_synth(S, C, T, H, 4, 1, oracle.outlier_gain(H, 2, 20.0, 4, 1))
    q, m = oracle.ref_stats(ref)
    ts, bs = oracle.block_scales(T, H, q, m, eps, kw.get("sigma_b", 0.0))
    h = cdt.canary_sim(to_dev(torch, ref), seed=12, cfg_id=5, mal_mask=1 << (S // 2),
                       bscale=to_dev(torch, bs), tscale=to_dev(torch, ts), redraw=True, **kw)
    torch.cuda.synchronize()
    want = oracle.canary_sim(ref, seed=12, cfg_id=5, mal_mask=1 << (S // 2), bscale=bs,
                             tscale=ts, redraw=True, **kw)
    assert int((h_bits(h) != want).sum()) == 0
    prim = oracle.canary_sim(ref, seed=12, cfg_id=5, mal_mask=1 << (S // 2), bscale=bs,
                             tscale=ts, **kw)
    assert not np.array_equal(prim, want)


@pytest.mark.parametrize("shape", SHAPES)
def test_drift_score_f16ref(gpu, shape):
    torch, cdt = gpu
    S, C, T, H = shape
    announce(f"drift f16ref {shape}")
    r = _f16(inputs.ref_normal(shape, seed=S + H, outlier_frac=0.01))
    h = inputs.live_near(_h(r).astype(np.float32), seed=3, rel=2e-3, flip_frac=0.001)
    nd = torch.empty((C, S, 2), dtype=torch.float64, device="cuda")
    sc = cdt.drift_score_f16ref(to_dev(torch, h).view(torch.float16),
                                to_dev(torch, r).view(torch.float16), num_den=nd)
    torch.cuda.synchronize()
    s64, _ = oracle.drift_score_f16ref(h, r)
    assert rel_err(sc.cpu().numpy(), s64) < DRIFT_RTOL


def _cos_tol(m_l2, n):
    """Absolute error bound of 1 - cos from fp64 sums of n terms on both
    sides: about 2 n 2^-53 m^2 each (m the relative-L2 mismatch)."""
    return 8.0 * n * 2.0**-53 * m_l2 * m_l2 + 1e-300


@pytest.mark.parametrize("shape", SHAPES)
@pytest.mark.parametrize("kind", ["noise", "rescale", "flip"])
def test_cosine_score(gpu, shape, kind):
    torch, cdt = gpu
    S, C, T, H = shape
    announce(f"cosine {kind} {shape}")
    a = inputs.ref_normal(shape, seed=S * 7 + H, outlier_frac=0.01)
    if kind == "noise":
        h = inputs.live_near(a, seed=5, rel=1e-3)
    elif kind == "rescale":
        h = _f16(1.1 * a)  # the angle is unchanged: cosine ~ 0
    else:
        h = inputs.live_near(a, seed=6, rel=1e-3, flip_frac=0.05)
    sums = torch.empty((C, S, 3), dtype=torch.float64, device="cuda")
    sc = cdt.cosine_score(to_dev(torch, h).view(torch.float16), to_dev(torch, a), sums=sums)
    torch.cuda.synchronize()
    got = sc.cpu().numpy().astype(np.float64)
    want, _ = oracle.cosine_score(h, a)
    l2, _, _ = oracle.drift_score(h, a)
    n = T * H
    for c in range(C):
        for s in range(S):
            tol = DRIFT_RTOL * abs(want[c, s]) + _cos_tol(l2[c, s], n) + 2.0**-24 * abs(want[c, s])
            assert abs(got[c, s] - want[c, s]) <= tol, (c, s, got[c, s], want[c, s])


def test_cosine_exact_cases(gpu):
    torch, cdt = gpu
    announce("cosine exact cases")
    C, T, H = 3, 17, 64
    a16 = _f16(inputs.ref_normal((1, C, T, H), seed=2))
    a = _h(a16).astype(np.float32)
    ref = np.concatenate([a] * 4)
    h = np.concatenate([a16, _f16(2 * a), a16 ^ np.uint16(0x8000), np.zeros_like(a16)])
    sc = cdt.cosine_score(to_dev(torch, h).view(torch.float16), to_dev(torch, ref))
    torch.cuda.synchronize()
    got = sc.cpu().numpy()
    assert np.all(got[:, 0] == 0.0) and np.all(got[:, 1] == 0.0)  # h = a, h = 2a
    assert np.all(np.abs(got[:, 2] - 2.0) <= 2**-22)                # h = -a
    assert np.all(got[:, 3] == 1.0)                                 # h = 0


@pytest.mark.parametrize("shape", SHAPES[:3])
def test_cosine_score_f16ref(gpu, shape):
    torch, cdt = gpu
    S, C, T, H = shape
    announce(f"cosine f16ref {shape}")
    r = _f16(inputs.ref_normal(shape, seed=9))
    h = inputs.live_near(_h(r).astype(np.float32), seed=10, rel=1e-2)
    sc = cdt.cosine_score_f16ref(to_dev(torch, h).view(torch.float16),
                                 to_dev(torch, r).view(torch.float16))
    torch.cuda.synchronize()
    want = oracle.cosine_score_f16ref(h, r)
    l2, _ = oracle.drift_score_f16ref(h, r)
    got = sc.cpu().numpy().astype(np.float64)
    tol = DRIFT_RTOL * np.abs(want) + _cos_tol(l2, T * H) + 2.0**-24 * np.abs(want)
    assert np.all(np.abs(got - want) <= tol)


def test_auroc_random_baseline(gpu):
    torch, cdt = gpu
    announce("auroc random baseline")
    cases = [(8, 32, 1 << 4, 0), (64, 100, (1 << 3) | (1 << 40), 7), (1, 5, 1, 2), (5, 0, 1, 3),
             (16, 256, 1 << 8, 4), (12, 10, 0, 5)]
    cfgs, off, tables = [], 0, []
    for S, C, mask, cid in cases:
        t = inputs.scores(C, S, seed=cid)
        tables.append(t)
        cfgs.append((S, C, off, mask, cid))
        off += t.size
    flat = to_dev(torch, np.concatenate([t.ravel() for t in tables]).astype(np.float32))
    counts, _, base = cdt.auroc(cfgs, flat, seed=77, flags=cdt.AUROC_RANDOM | cdt.AUROC_CONTROL)
    torch.cuda.synchronize()
    got = cdt.u64(base)
    got_c = cdt.u64(counts)
    for g, (S, C, off_g, mask, cid) in enumerate(cfgs):
        np.testing.assert_array_equal(got[g], oracle.random_baseline(C, S, mask, seed=77,
                                                                     cfg_id=cid))
        want_c, _ = oracle.auroc_config(tables[g], mask, seed=77, cfg_id=cid, flags=1)
        np.testing.assert_array_equal(got_c[g], want_c)
