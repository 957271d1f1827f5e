"""Pins of the oracle's relative-L2 mismatch, Eq. 4 (CPU only).

m = ||h - a||_F / ||a||_F over a T x d block.  Checked against exact
rational arithmetic on tiny blocks, numpy's Frobenius norm (a library
routine), closed forms (h = a, -a, 2a, 0, a constant offset) and the scale
invariance of a ratio of norms.
"""
import math
from fractions import Fraction

import numpy as np

from paper_2607_19490_amd import inputs


def _h(bits):
    return np.asarray(bits, np.uint16).view(np.float16).astype(np.float64)


def test_exact_rational_on_tiny_blocks(orc):
    g = np.random.default_rng(0)
    for trial in range(20):
        n = int(g.integers(1, 40))
        a = g.standard_normal(n).astype(np.float32)
        h = inputs.live_near(a, seed=trial, rel=0.05)
        m, D, R = orc.drift_block(h, a)
        Dq = sum((Fraction(float(x)) - Fraction(float(y))) ** 2 for x, y in zip(_h(h), a))
        Rq = sum(Fraction(float(y)) ** 2 for y in a)
        assert abs(Fraction(D) - Dq) <= Dq * Fraction(1, 2**50)
        assert abs(Fraction(R) - Rq) <= Rq * Fraction(1, 2**50)
        exact = math.sqrt(Dq / Rq)
        assert abs(m - exact) <= 1e-14 * exact


def test_matches_numpy_frobenius_norm(orc):
    a = inputs.ref_normal((4, 3, 17, 40), seed=1, outlier_frac=0.05)
    h = inputs.live_near(a, seed=2, rel=1e-3)
    s64, s32, nd = orc.drift_score(h, a)
    S, C = a.shape[:2]
    for s in range(S):
        for c in range(C):
            d = _h(h[s, c]) - a[s, c].astype(np.float64)
            want = np.linalg.norm(d) / np.linalg.norm(a[s, c].astype(np.float64))
            assert abs(s64[c, s] - want) <= 1e-13 * want
            assert s32[c, s] == np.float32(s64[c, s])
            assert nd[c, s, 1] > 0


def test_closed_forms(orc):
    # a exactly representable in fp16, so h can equal it
    a = inputs.fp16_bits(inputs.ref_normal((64, 64), seed=3)).view(np.float16).astype(np.float32)
    f16 = lambda x: np.asarray(x, np.float32).astype(np.float16).view(np.uint16)
    assert orc.drift_block(f16(a), a)[0] == 0.0        # h = a
    assert orc.drift_block(f16(-a), a)[0] == 2.0       # sign flip: m = 2
    assert orc.drift_block(f16(2 * a), a)[0] == 1.0    # doubling: m = 1
    assert orc.drift_block(np.zeros(a.shape, np.uint16), a)[0] == 1.0  # h = 0
    # a constant block plus a constant offset: m = |offset| / |a|
    a = np.full(100, 4.0, np.float32)
    assert orc.drift_block(f16(np.full(100, 4.5)), a)[0] == 0.125


def test_scale_invariance(orc):
    """m is a ratio of norms: scaling h and a by 2^k leaves it bit-identical."""
    a = inputs.ref_normal((32, 48), seed=4)
    h = inputs.live_near(a, seed=5, rel=1e-2)
    m0 = orc.drift_block(h, a)[0]
    for k in (-3, 2, 5):
        a2 = (a * np.float32(2.0**k)).astype(np.float32)
        h2 = (_h(h) * 2.0**k).astype(np.float16).view(np.uint16)
        assert orc.drift_block(h2, a2)[0] == m0


def test_degenerate_blocks(orc):
    z = np.zeros(16, np.float32)
    assert orc.drift_block(np.zeros(16, np.uint16), z)[0] == 0.0
    assert orc.drift_block(inputs.fp16_bits(np.ones(16)), z)[0] == math.inf
    m, D, R = orc.drift_block(np.zeros(0, np.uint16), np.zeros(0, np.float32))
    assert (m, D, R) == (0.0, 0.0, 0.0)


def test_score_layout_is_canary_major(orc):
    S, C, T, H = 3, 5, 2, 8
    a = inputs.ref_normal((S, C, T, H), seed=6)
    h = inputs.live_near(a, seed=7, rel=1e-2)
    s64, _, nd = orc.drift_score(h, a)
    assert s64.shape == (C, S)
    for s in range(S):
        for c in range(C):
            m, D, R = orc.drift_block(h[s, c], a[s, c])
            assert s64[c, s] == m and nd[c, s, 0] == D and nd[c, s, 1] == R
