"""Pins of the oracle's random and rounding primitives (CPU only).

Philox4x32-10 (Salmon et al., SC'11) is checked against the authors'
published known-answer vectors and rocRAND's independent header
implementation; the Irwin-Hall normal against its closed-form moments,
symmetry and distribution; fp32 -> fp16 rounding against numpy's float16
conversion (a library routine) on every rounding boundary.
"""
import math
import warnings

import numpy as np
import pytest


def test_philox_known_answers(orc):
    """The generator authors' published known-answer vectors
    (tests/golden/philox4x32_10_kat.json)."""
    import json
    import os
    path = os.path.join(os.path.dirname(__file__), "golden", "philox4x32_10_kat.json")
    for v in json.load(open(path))["vectors"]:
        ctr = np.array([int(x, 16) for x in v["counter"]], np.uint64).astype(np.uint32)
        key = np.array([int(x, 16) for x in v["key"]], np.uint64).astype(np.uint32)
        want = np.array([int(x, 16) for x in v["output"]], np.uint64).astype(np.uint32)
        np.testing.assert_array_equal(orc.philox(ctr, key), want)


def test_philox_matches_rocrand(orc, philox_pin):
    g = np.random.default_rng(1234)
    ctr = g.integers(0, 2**32, size=(2000, 4), dtype=np.uint64).astype(np.uint32)
    key = g.integers(0, 2**32, size=(2000, 2), dtype=np.uint64).astype(np.uint32)
    # structured corner cases: zero, all-ones, counter words used by the streams
    ctr[0] = 0
    key[0] = 0
    ctr[1] = 0xFFFFFFFF
    key[1] = 0xFFFFFFFF
    ctr[2] = [7, 3, 5, (4 << 24) | 17]
    key[2] = [0, 0]
    want = philox_pin(ctr, key)
    got = np.stack([orc.philox(c, k) for c, k in zip(ctr, key)])
    np.testing.assert_array_equal(got, want)


def test_philox_avalanche(orc):
    """A one-bit counter change flips about half of the 128 output bits."""
    g = np.random.default_rng(5)
    flips = []
    for _ in range(200):
        c = g.integers(0, 2**32, size=4, dtype=np.uint64).astype(np.uint32)
        k = g.integers(0, 2**32, size=2, dtype=np.uint64).astype(np.uint32)
        c2 = c.copy()
        bit = int(g.integers(0, 128))
        c2[bit // 32] ^= np.uint32(1 << (bit % 32))
        x = orc.philox(c, k) ^ orc.philox(c2, k)
        flips.append(sum(bin(int(w)).count("1") for w in x))
    assert abs(np.mean(flips) - 64.0) < 2.0


def test_k16_unit_variance_constant(orc):
    """K16^2 * (2^32 - 1) / 3 is 1 up to fp32 rounding of K16."""
    k = float(orc.k16())
    assert abs(k * k * (2**32 - 1) / 3.0 - 1.0) < 2.0**-22


def test_z16_extremes_and_zero(orc):
    k = float(orc.k16())
    assert float(orc.z16(0, 0)) == float(np.float32(-131070.0 * k))
    assert float(orc.z16(0xFFFFFFFF, 0xFFFFFFFF)) == float(np.float32(131070.0 * k))
    # 0x8000 + 0x7FFF in each word: the centred sum is exactly zero
    assert float(orc.z16(0x7FFF8000, 0x80007FFF)) == 0.0
    assert abs(float(orc.z16(0xFFFFFFFF, 0xFFFFFFFF)) - math.sqrt(12.0)) < 1e-4


def test_z16_antisymmetric(orc):
    """Complementing every 16-bit lane negates the centred sum exactly."""
    g = np.random.default_rng(7)
    for w0, w1 in g.integers(0, 2**32, size=(500, 2), dtype=np.uint64):
        w0, w1 = int(w0), int(w1)
        assert float(orc.z16(w0 ^ 0xFFFFFFFF, w1 ^ 0xFFFFFFFF)) == -float(orc.z16(w0, w1))


def _irwin_hall4_cdf(x):
    """CDF of the sum of 4 independent U(0,1) (closed form)."""
    x = np.asarray(x, np.float64)
    out = np.zeros_like(x)
    for k in range(5):
        term = (-1) ** k * math.comb(4, k) * np.clip(x - k, 0, None) ** 4
        out += term
    return np.clip(out / 24.0, 0, 1)


def test_normal_stream_moments_and_shape(orc):
    """1M normals of one stream: mean 0, variance 1, excess kurtosis -0.3,
    support +-sqrt(12), and the Irwin-Hall(4) distribution (chi-square)."""
    z = orc.ref_block(0, 0, 1024, 1024, 99, 3, np.ones(1024, np.float32)).ravel().astype(np.float64)
    n = z.size
    assert abs(z.mean()) < 5 / math.sqrt(n)
    var = z.var()
    assert abs(var - 1.0) < 0.006
    kurt = ((z - z.mean()) ** 4).mean() / var**2
    assert abs(kurt - 2.7) < 0.03
    assert np.abs(z).max() <= math.sqrt(12.0) + 1e-6
    # chi-square against the Irwin-Hall(4) CDF on 40 equiprobable-ish bins
    u = z / math.sqrt(12.0) * 2.0 + 2.0  # back to the sum of four U(0,1)
    edges = np.linspace(0.0, 4.0, 41)
    obs, _ = np.histogram(u, bins=edges)
    p = np.diff(_irwin_hall4_cdf(edges))
    exp = p * n
    keep = exp > 50
    chi2 = (((obs - exp) ** 2) / exp)[keep].sum()
    dof = keep.sum() - 1
    # mean dof, sd sqrt(2 dof); 6 sd is far beyond sampling noise
    assert chi2 < dof + 6 * math.sqrt(2 * dof), (chi2, dof)


def _np_f16(x):
    with warnings.catch_warnings():
        warnings.simplefilter("ignore")
        return np.asarray(x, np.float32).astype(np.float16).view(np.uint16)


def _check_f16(orc, x):
    x = np.asarray(x, np.float32)
    got = orc.f16_rne(x)
    want = _np_f16(x)
    nan = np.isnan(x)
    np.testing.assert_array_equal(got[~nan], want[~nan])
    # NaN stays NaN (payload not specified)
    assert np.all((got[nan] & 0x7C00) == 0x7C00) and np.all((got[nan] & 0x3FF) != 0)


def test_f16_every_rounding_boundary(orc):
    """Every fp16 value, every midpoint between neighbours, and the fp32
    values one ulp either side of each midpoint (where RNE decides)."""
    halves = np.arange(0, 0x7C00, dtype=np.uint16).view(np.float16).astype(np.float64)
    nxt = np.append(halves[1:], 65536.0)
    mid = ((halves + nxt) / 2.0).astype(np.float32)  # exact in fp32
    assert np.all(mid.astype(np.float64) == (halves + nxt) / 2.0)
    vals = np.concatenate([halves.astype(np.float32), mid,
                           np.nextafter(mid, np.float32(np.inf)),
                           np.nextafter(mid, np.float32(0))])
    vals = np.concatenate([vals, -vals])
    _check_f16(orc, vals)


def test_f16_specials_and_random(orc):
    specials = np.array([0.0, -0.0, np.inf, -np.inf, np.nan, 65504, 65519.996, 65520, 1e30,
                         2**-24, 2**-25, 2**-25 * 1.0000001, 3 * 2**-26, 2**-14, 2**-14 * 0.999],
                        np.float32)
    _check_f16(orc, specials)
    g = np.random.default_rng(11)
    bits = g.integers(0, 2**32, size=1 << 22, dtype=np.uint64).astype(np.uint32)
    _check_f16(orc, bits.view(np.float32))


@pytest.mark.slow
def test_f16_exhaustive(orc):
    """All 2^32 fp32 inputs (opt-in: about ten minutes)."""
    step = 1 << 26
    for start in range(0, 1 << 32, step):
        bits = np.arange(start, start + step, dtype=np.uint64).astype(np.uint32)
        x = bits.view(np.float32)
        got = orc.f16_rne_range(start, step)
        want = _np_f16(x)
        nan = np.isnan(x)
        assert np.array_equal(got[~nan], want[~nan]), hex(start)


def test_f16_value_roundtrip(orc):
    for b in [0, 1, 0x3FF, 0x400, 0x3C00, 0x7BFF, 0x8001, 0xFBFF, 0x7C00, 0xFC00]:
        want = float(np.array([b], np.uint16).view(np.float16)[0])
        assert orc.f16_value(b) == want
