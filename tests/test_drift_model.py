"""Checks of the statistical model in tests/drift_model.py against closed
forms, so the statistical tests rest on a model that obeys the laws it
claims (carry law, Eq. 4 on an exact-norm attack, Eq. 6's chance level)."""
import math

import numpy as np
import pytest

from tests import drift_model as M

pytestmark = pytest.mark.statistical


def test_benign_floor_follows_the_carry_law():
    """m_s^2 = beta^2 (1 + g^2 + ... + g^(2s)), beta^2 = sigma^2 E[(U/n)^2 / (A/n)]
    + rho^2: with sigma^2 dominant, its mean per stage against the sum."""
    S, g, sigma, T, H = 8, 0.7, 0.05, 48, 768
    l2, _, _ = M.simulate(S, 50, T, H, (), sigma=sigma, carry=g, reps=200, seed=3)
    n_out = int(0.01 * H + 0.5)
    mean_abs = math.sqrt(2 / math.pi) * (H - n_out + 20.0 * n_out) / H
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
