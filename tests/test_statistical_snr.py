"""Statistical expectation (not parity) for the raised-noise-floor study
(Section 5.4; 16 x 128 x 128 x 4096, Gaussian tamper 0.02 per element,
benign noise sigma |a| z raised from 1e-4 to 1e-1): the oracle's detection
AUROC at each of its 40 runs (20 noise levels, Gaussian and Student-t
noise), counted by brute force from its stored per-block scores
(tests/golden/fullsize_snr.npz), lies inside the central 99.8% of the
independent Monte Carlo model of tests/drift_model.py.  The model knows only
the generator's laws (Eqs. 2-4, the reference distribution and the
Irwin-Hall normals everything is drawn from), so this pins the oracle's
statistics, not its arithmetic.

The Student-t noise is the generator's z0 / sqrt(z1^2 + z2^2 + z3^2) of four
Irwin-Hall normals, whose tail is lighter than a true Student-t's (less
mass near q = 0, E[1/q] = 0.941 instead of 1): the model draws that law,
not the textbook one, which would put the curve's knee too low.
"""
import os

import numpy as np
import pytest

from paper_2607_19490_amd import workloads as W
from tests import drift_model as M

pytestmark = pytest.mark.statistical

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "fullsize_snr.npz")


def strict_auroc(sc, is_mal):
    """Eq. 6 (strict) by brute force over (attacker, benign) pairs per canary."""
    return float((sc[:, is_mal][:, :, None] > sc[:, ~is_mal][:, None, :]).mean())


def test_gaussian_snr_curve_follows_the_model():
    wl = W.snr()
    rs = wl.ref_sets[0]
    S, C = rs.S, rs.C
    s64 = np.load(GOLDEN)["score64"]
    is_mal = np.zeros(S, bool)
    is_mal[list(rs.mal_shards)] = True
    seen = []
    for r, run in enumerate(rs.runs):
        if run.benign_dist != W.DIST_GAUSS:
            continue
        got = strict_auroc(s64[r * S * C:(r + 1) * S * C].reshape(C, S), is_mal)
        l2, im = M.simulate_elementwise(S, C, rs.T, rs.H, rs.mal_shards, sigma=run.sigma_b,
                                        eps=run.eps, reps=1000, seed=r)
        lo, hi = M.interval(M.auroc_strict(l2, im))
        assert lo <= got <= hi, (run.label, got, lo, hi)
        seen.append((run.sigma_b, got, lo, hi))
    assert len(seen) == 20
    # the curve falls off where the noise floor reaches the tamper: the model
    # puts the last level's AUROC well below 1, and the oracle agrees
    assert seen[-1][3] < 0.95 and seen[-1][1] < 0.95


def test_student_t_snr_curve_follows_the_model():
    """The Student-t half: one draw of the benign energy W per block (it
    does not depend on sigma) serves all 20 levels, each with its own
    tamper draws."""
    wl = W.snr()
    rs = wl.ref_sets[0]
    S, C = rs.S, rs.C
    s64 = np.load(GOLDEN)["score64"]
    is_mal = np.zeros(S, bool)
    is_mal[list(rs.mal_shards)] = True
    n_out = W.n_outliers(rs.H)
    w = M.elementwise_energy(np.random.default_rng(2024), (1000, C, S), rs.T, rs.H, n_out, 20.0,
                             "t3")
    seen = []
    for r, run in enumerate(rs.runs):
        if run.benign_dist != W.DIST_T3:
            continue
        got = strict_auroc(s64[r * S * C:(r + 1) * S * C].reshape(C, S), is_mal)
        l2, im = M.simulate_elementwise(S, C, rs.T, rs.H, rs.mal_shards, sigma=run.sigma_b,
                                        eps=run.eps, dist="t3", seed=r, w=w)
        lo, hi = M.interval(M.auroc_strict(l2, im))
        assert lo <= got <= hi, (run.label, got, lo, hi)
        seen.append((run.sigma_b, got, lo, hi))
    assert len(seen) == 20
    # heavy tails break detection sooner than Gaussian noise of the same
    # scale: the model and the oracle both put sigma_b = 0.07 below 0.82
    knee = [x for x in seen if 0.06 < x[0] < 0.08][0]
    assert knee[3] < 0.82 and knee[1] < 0.82
