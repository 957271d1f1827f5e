"""Statistical expectation (not parity) for the raised-noise-floor study
(Section 5.4; 16 x 128 x 128 x 4096, Gaussian tamper 0.02 per element,
benign noise sigma |a| z raised from 1e-4 to 1e-1): the oracle's detection
AUROC over the Gaussian half of its 20 noise levels, counted by brute force
from its stored per-block scores (tests/golden/fullsize_snr.npz), lies inside
the central 99.8% of the independent Monte Carlo model of tests/drift_model.py.
The model knows only the generator's laws (Eqs. 2-4 and the reference
distribution), so this pins the oracle's statistics, not its arithmetic.

The Student-t half has no such model here: its noise has no fourth moment,
so the block statistic is not close to normal and the cheap model does not
apply; the full-size parity tests compare that half with the oracle exactly.
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
