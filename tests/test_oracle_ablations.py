"""Pins of the oracle's reference conditions and detector ablations (CPU only).

Section 4.5 brackets the detector with a random baseline (scores replaced by
Uniform(0,1), E[A] = 0.50) and a redundant-recompute ceiling (the live
output against an independent benign recompute); Section 4.4 ablates the
stored reference (a separately drawn benign pass instead) and the metric
(cosine distance, blind to a pure rescale by construction).  Checked here:
numpy's Frobenius norm (library), 60-digit decimal arithmetic, closed forms,
brute force, and the statistics each construction fixes.
"""
import json
import math
import os
from decimal import Decimal, getcontext

import numpy as np

from paper_2607_19490_amd import inputs

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _h(bits):
    return np.asarray(bits, np.uint16).view(np.float16).astype(np.float64)


def _f16(x):
    return np.asarray(x, np.float32).astype(np.float16).view(np.uint16)


# ----------------------------------------------------------------------------
# Eq. 4 against an fp16 reference
# ----------------------------------------------------------------------------
def test_f16ref_drift_matches_numpy_norm(orc):
    r = _f16(inputs.ref_normal((3, 2, 9, 40), seed=1))
    h = inputs.live_near(_h(r).astype(np.float32), seed=2, rel=1e-2)
    s64, s32 = orc.drift_score_f16ref(h, r)
    for s in range(3):
        for c in range(2):
            want = np.linalg.norm(_h(h[s, c]) - _h(r[s, c])) / np.linalg.norm(_h(r[s, c]))
            assert abs(s64[c, s] - want) <= 1e-13 * want
    assert s32.dtype == np.float32


def test_f16ref_drift_closed_forms(orc):
    r = _f16(inputs.ref_normal((50,), seed=3))
    assert orc.drift_block_f16ref(r, r)[0] == 0.0
    assert orc.drift_block_f16ref(r ^ np.uint16(0x8000), r)[0] == 2.0
    z = np.zeros(8, np.uint16)
    assert orc.drift_block_f16ref(z, z)[0] == 0.0
    assert orc.drift_block_f16ref(_f16(np.ones(8)), z)[0] == math.inf


# ----------------------------------------------------------------------------
# cosine mismatch
# ----------------------------------------------------------------------------
def _cos_decimal(hb, a):
    getcontext().prec = 60
    hv = [Decimal(float(x)) for x in _h(hb)]
    av = [Decimal(float(x)) for x in a]
    hh = sum(x * x for x in hv)
    aa = sum(x * x for x in av)
    ha = sum(x * y for x, y in zip(hv, av))
    return 1 - ha / (hh * aa).sqrt()


def test_cosine_against_60_digit_arithmetic(orc):
    g = np.random.default_rng(4)
    for trial in range(12):
        n = int(g.integers(2, 60))
        a = g.standard_normal(n).astype(np.float32)
        rel = [1e-1, 1e-2, 1e-3, 3e-4][trial % 4]  # down to near-parallel vectors
        h = inputs.live_near(a, seed=trial, rel=rel)
        want = _cos_decimal(h, a)
        got = orc.cosine_block(h, a)
        assert abs(Decimal(got) - want) <= abs(want) * Decimal(1e-9) + Decimal(1e-18)


def test_cosine_closed_forms(orc):
    a16 = _f16(inputs.ref_normal((200,), seed=5))
    a = _h(a16).astype(np.float32)
    # a positive rescale leaves the angle unchanged: the tampered stage of the
    # rescale attack has cosine mismatch 0 (Section 4.4)
    assert abs(orc.cosine_block(_f16(2 * a), a)) < 1e-15
    assert abs(orc.cosine_block(_f16(0.5 * a), a)) < 1e-15
    assert abs(orc.cosine_block(a16, a)) < 1e-15
    assert abs(orc.cosine_block(a16 ^ np.uint16(0x8000), a) - 2.0) < 1e-15  # opposite: 2
    e1 = np.array([1, 0, 0, 0, 0, 0, 0, 0], np.float32)
    e2 = np.array([0, 1, 0, 0, 0, 0, 0, 0], np.float32)
    assert orc.cosine_block(_f16(e2), e1) == 1.0  # orthogonal
    z = np.zeros(8, np.float32)
    assert orc.cosine_block(_f16(z), z) == 0.0
    assert orc.cosine_block(_f16(z), e1) == 1.0
    assert orc.cosine_block(_f16(e1), z) == 1.0


def test_cosine_f16ref_matches_fp32_path_and_decimal(orc):
    """Against an fp16 reference the cosine equals the fp32-reference cosine
    of the same (exactly widened) values, and the 60-digit value."""
    g = np.random.default_rng(8)
    for trial in range(8):
        r = _f16(g.standard_normal(int(g.integers(2, 50))).astype(np.float32))
        h = inputs.live_near(_h(r).astype(np.float32), seed=trial, rel=[1e-1, 1e-3][trial % 2])
        got = orc.cosine_block_f16ref(h, r)
        assert got == orc.cosine_block(h, _h(r).astype(np.float32))
        want = _cos_decimal(h, _h(r))
        assert abs(Decimal(got) - want) <= abs(want) * Decimal(1e-9) + Decimal(1e-18)
    r = _f16(inputs.ref_normal((100,), seed=9))
    assert abs(orc.cosine_block_f16ref(_f16(2 * _h(r)), r)) < 1e-15


def test_cosine_small_angle_law(orc):
    """For h = a + d with d independent of a, 1 - cos ~ |d|^2 / (2 |a|^2)
    = m^2 / 2 (m the relative-L2 mismatch)."""
    a = inputs.ref_normal((64, 256), seed=6)
    h = inputs.live_near(a, seed=7, rel=1e-2)
    m, _, _ = orc.drift_block(h, a)
    c = orc.cosine_block(h, a)
    assert abs(c / (m * m / 2) - 1.0) < 0.02


# ----------------------------------------------------------------------------
# random baseline
# ----------------------------------------------------------------------------
def test_random_scores_uniform(orc):
    u = np.array([orc.random_score(3, 5, t, s) for t in range(400) for s in range(25)])
    assert u.min() >= 0.0 and u.max() < 1.0
    assert abs(u.mean() - 0.5) < 5 * math.sqrt(1 / 12 / u.size)
    assert abs(u.var() - 1 / 12) < 0.005
    assert np.all((u * 2**24) == np.floor(u * 2**24))  # 24 random bits, exact in fp32


def test_random_baseline_counts_follow_definition(orc):
    C, S, pos = 30, 7, (2, 5)
    mask = (1 << 2) | (1 << 5)
    base = orc.random_baseline(C, S, mask, seed=9, cfg_id=4)
    G = E = N = 0
    for t in range(C):
        u = [orc.random_score(9, 4, t, s) for s in range(S)]
        for i in pos:
            for j in range(S):
                if j in pos:
                    continue
                G += u[i] > u[j]
                E += u[i] == u[j]
                N += 1
    assert tuple(int(x) for x in base) == (G, E, N)


def test_random_baseline_is_chance(orc):
    """Section 4.5: scores replaced by Uniform(0,1) give E[A] = 0.50."""
    with open(os.path.join(GOLDEN, "paper_outcomes.json")) as f:
        gold = json.load(f)
    C, S = 5000, 12
    base = orc.random_baseline(C, S, 1 << 5, seed=0, cfg_id=2)
    a = int(base[0]) / int(base[2])
    # per canary A is uniform on {0, 1/11, ..., 1}: sd 0.316 / sqrt(C)
    sd = math.sqrt((S - 1) * (S + 1) / 12.0) / (S - 1) / math.sqrt(C)
    assert abs(a - gold["random_baseline_mean"]["value"]) < 5 * sd


# ----------------------------------------------------------------------------
# independent benign redraw (recompute ceiling, noisy reference)
# ----------------------------------------------------------------------------
def test_redraw_is_an_independent_benign_pass(orc):
    a = orc.ref_block(0, 0, 256, 512, 3, 0, np.ones(512, np.float32))
    h = orc.sim_block(0, 0, a, seed=1, cfg_id=0, sigma_b=1e-2)
    r = orc.sim_block(0, 0, a, seed=1, cfg_id=0, sigma_b=1e-2, redraw=True)
    assert not np.array_equal(h, r)
    # same law: m(r, a) = sigma; independent noise: m(h, r) = sqrt(2) sigma
    m_r, _, _ = orc.drift_block(r, a)
    assert abs(m_r / 1e-2 - 1.0) < 0.01
    m_hr = orc.drift_block_f16ref(h, r)[0]
    assert abs(m_hr / (math.sqrt(2) * 1e-2) - 1.0) < 0.01
    # the two noise draws are uncorrelated
    dh = _h(h) - a
    dr = _h(r) - a
    rho = (dh * dr).sum() / math.sqrt((dh * dh).sum() * (dr * dr).sum())
    assert abs(rho) < 5 / math.sqrt(a.size)


def test_redraw_changes_only_the_benign_noise(orc):
    a = orc.ref_block(0, 0, 16, 64, 3, 0, np.ones(64, np.float32))
    kw = dict(seed=1, cfg_id=0, sigma_b=0.0)
    np.testing.assert_array_equal(orc.sim_block(0, 0, a, **kw),
                                  orc.sim_block(0, 0, a, redraw=True, **kw))
    kw = dict(seed=1, cfg_id=0, sigma_b=0.3, malicious=True, tamper=1 | 2, tscale=0.5,
              flip_p=0.5, tamper_base=1)
    np.testing.assert_array_equal(orc.sim_block(0, 0, a, **kw),
                                  orc.sim_block(0, 0, a, redraw=True, **kw))
    # Student-t redraw also leaves the primary streams alone
    kw = dict(seed=1, cfg_id=0, sigma_b=0.1, benign_dist=1)
    assert not np.array_equal(orc.sim_block(0, 0, a, **kw),
                              orc.sim_block(0, 0, a, redraw=True, **kw))
