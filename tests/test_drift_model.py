"""Checks of the statistical model in tests/drift_model.py against closed
forms and brute force, so the statistical tests rest on a model that obeys
the laws it claims: the Irwin-Hall normal's moments, the chi-square laws its
quadrature must reproduce for a true normal, the Student-t energy against a
sum drawn element by element, the carry law, Eq. 4 on an exact-norm
attack, Eq. 6's chance level."""
import math

import numpy as np
import pytest
from scipy import special

from tests import drift_model as M

pytestmark = pytest.mark.statistical


def test_benign_floor_follows_the_carry_law():
    """m_s^2 = beta^2 (1 + g^2 + ... + g^(2s)), beta^2 = sigma^2 E[(U/n)^2 / (A/n)]
    + rho^2: with sigma^2 dominant, its mean per stage against the sum."""
    S, g, sigma, T, H = 8, 0.7, 0.05, 48, 768
    l2, _, _ = M.simulate(S, 50, T, H, (), sigma=sigma, carry=g, reps=200, seed=3)
    n_out = int(0.01 * H + 0.5)
    mean_abs = M.IH_ABS * (H - n_out + 20.0 * n_out) / H
    mean_sq = (H - n_out + 400.0 * n_out) / H
    beta2 = sigma ** 2 * mean_abs ** 2 / mean_sq
    got = (l2 ** 2).mean(axis=(0, 1))
    for s in range(S):
        want = beta2 * sum(g ** (2 * j) for j in range(s + 1))
        # E[U^2 / A] exceeds E[U]^2 / E[A] by the relative variance of A
        assert abs(got[s] / want - 1.0) < 0.02, (s, got[s], want)
    assert np.all(np.diff(got) > 0)


def test_exact_norm_attack_adds_eps_squared():
    """With no noise the attacker's m is eps (its tamper has norm eps ||v||,
    v = a) up to fp16 rounding."""
    l2, _, im = M.simulate(4, 20, 16, 256, (2,), sigma=0.0, attack="gauss", eps=0.05, reps=5)
    assert np.allclose(l2[..., im], 0.05, rtol=1e-3)
    assert (l2[..., ~im] < 1e-3).all()


def test_exchangeable_stages_give_chance():
    """A rescale seen by the angle only, with independent stages: every stage
    is alike, so the AUROC averages 1/2 (Eq. 6's chance level)."""
    _, cos, im = M.simulate(12, 100, 48, 768, (5,), sigma=0.002, attack="rescale", scale=1.1,
                            reps=400, seed=5)
    a = M.auroc_strict(cos, im)
    assert abs(a.mean() - 0.5) < 0.01


def test_irwin_hall_moments():
    """The generator's normal is (sum of four U(0, 1) - 2) sqrt 3: unit
    variance, E|z| = sqrt(3) E|s - 2| = 7 sqrt(3) / 15 (integrating the
    Irwin-Hall density piece by piece), E z^4 = 3 - 6 / (5 * 4) (the
    Irwin-Hall excess kurtosis -6 / (5n), n = 4); the model's draws agree."""
    assert M.ih_moment(lambda x: np.ones_like(x)) == pytest.approx(1.0, abs=1e-14)
    assert M.ih_moment(lambda x: x * x) == pytest.approx(1.0, abs=1e-14)
    assert M.IH_ABS == pytest.approx(7.0 * math.sqrt(3.0) / 15.0, abs=1e-14)
    assert M.IH_K4 == pytest.approx(2.7, abs=1e-13)
    z = M.ih_draw(np.random.default_rng(1), 1 << 22)
    assert abs(z.max()) <= 2.0 * math.sqrt(3.0) and abs(z.min()) <= 2.0 * math.sqrt(3.0)
    se = 1.0 / math.sqrt(z.size)
    assert abs((z * z).mean() - 1.0) < 6 * math.sqrt(1.7) * se
    assert abs(np.abs(z).mean() - M.IH_ABS) < 6 * se
    assert abs((z ** 4).mean() - 2.7) < 6 * 3.5 * se
    # the gamma law of a sum of squares: its mean and variance
    q = M.ih_sq_sum(np.random.default_rng(2), 384, 200000)
    assert abs(q.mean() / 384 - 1.0) < 1e-3
    assert abs(q.var() / (384 * 1.7) - 1.0) < 0.02


@pytest.mark.parametrize("q0", [0.002, 0.05])
def test_cut_moments_reproduce_chi_square(q0):
    """With the normal density, q = z1^2 + z2^2 + z3^2 is chi-square(3):
    P(q < q0) = P(3/2, q0/2) (regularised incomplete gamma), E[1/q; q >= q0]
    = Q(1/2, q0/2) and E[1/q^2; q >= q0] = e^-x / sqrt(pi x) - erfc(sqrt x),
    x = q0 / 2.  The same quadrature gives the Irwin-Hall values."""
    p0, m1, m2 = M.t3_cut_moments(q0, M.normal_density, 14.0)
    x = q0 / 2
    assert p0 == pytest.approx(special.gammainc(1.5, x), rel=1e-10)
    assert m1 == pytest.approx(special.gammaincc(0.5, x), rel=1e-10)
    assert m2 == pytest.approx(math.exp(-x) / math.sqrt(math.pi * x) - special.erfc(math.sqrt(x)),
                               rel=1e-10)


def test_irwin_hall_cut_moments_match_draws():
    """The Irwin-Hall quadrature against q drawn from the model's own normals
    (2^22 triplets): the mass below the cut and the truncated moments agree
    within their sampling errors; the Irwin-Hall Student-t has E[1/q] < 1 (a
    true one has exactly 1) and less mass near q = 0."""
    q0 = 0.05
    p0, m1, m2 = M.t3_cut_moments(q0)
    rng = np.random.default_rng(3)
    q = np.zeros(1 << 22)
    for _ in range(3):
        q += M.ih_draw(rng, q.size) ** 2
    n = q.size
    keep = q >= q0
    inv = np.where(keep, 1.0 / q, 0.0)
    assert abs((~keep).mean() - p0) < 5 * math.sqrt(p0 / n)
    assert abs(inv.mean() - m1) < 5 * inv.std() / math.sqrt(n)
    assert abs((inv * inv).mean() - m2) < 5 * (inv * inv).std() / math.sqrt(n)
    whole = M.radial_integral(M.ih_density, lambda r: np.ones_like(r), 0.0, 6.0)
    assert 0.93 < whole < 0.95
    assert p0 < special.gammainc(1.5, q0 / 2)


def test_student_t_energy_against_brute_force():
    """W = sum a^2 z^2 / sum a^2 for Student-t noise on blocks of the SNR
    study's size (128 x 4096 elements, 41 outlier channels at gain 20): the
    model's split (tail drawn element by element below the cut, the rest
    through the normal limit) against W summed over every element of 120
    blocks, z = z0 / sqrt(z1^2 + z2^2 + z3^2) of Irwin-Hall draws.  The two
    distributions agree (two-sample Kolmogorov-Smirnov, medians within 3%)
    whichever cut splits the tail off."""
    from scipy import stats
    T, H, n_out, G = 128, 4096, 41, 20.0
    rng = np.random.default_rng(4)
    gain = np.where(np.arange(H) < n_out, G, 1.0).astype(np.float32)

    def ih32(shape):
        return (rng.random(shape + (4,), dtype=np.float32).sum(-1) - 2.0) * np.float32(M.SQ3)

    brute = np.empty(120)
    for b in range(brute.size):
        a2 = ((ih32((T, H)) * gain) ** 2).astype(np.float64)
        u = ih32((3, T, H))
        z0 = ih32((T, H))
        brute[b] = (a2 * (z0 * z0 / (u * u).sum(0))).sum() / a2.sum()
    for seed, cuts in ((5, M.T3_CUTS), (6, (0.005, 0.2))):
        model = M.elementwise_energy(np.random.default_rng(seed), (20, 50, 10), T, H, n_out, G,
                                     "t3", cuts=cuts).ravel()
        assert stats.ks_2samp(brute, model).pvalue > 1e-3, cuts
        assert np.median(model) == pytest.approx(np.median(brute), rel=0.03), cuts
