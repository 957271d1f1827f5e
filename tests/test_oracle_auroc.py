"""Pins of the oracle's detection AUROC, Eqs. 5-6 (CPU only).

Per canary t, A(t) counts benign stages j whose mismatch the malicious stage
exceeds (Eq. 5); the aggregate is the mean over canaries (Eq. 6), which the
paper equates with the normalised Mann-Whitney U.  Checked against
scikit-learn's roc_auc_score and scipy's mannwhitneyu (library routines), a
pure-Python brute force on tiny inputs exhaustive over label sets, closed
forms (perfect separation, reversal, all ties) and the scrambled-label
control's exchangeability (Section 4.5).
"""
import itertools
import json
import math
import os

import numpy as np
import pytest
from scipy import stats
from sklearn.metrics import roc_auc_score

from paper_2607_19490_amd import inputs

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _mask(shards):
    m = 0
    for s in shards:
        m |= 1 << s
    return m


def _key(x):
    # numeric order (-0 == +0), NaN above every number, NaN == NaN
    return (1, 0.0) if math.isnan(x) else (0, float(x))


def _brute(scores, pos):
    """Pure-Python counts of Eq. 5 summed over canaries."""
    G = E = N = 0
    C, S = scores.shape
    for t in range(C):
        for i in pos:
            for j in range(S):
                if j in pos:
                    continue
                ki, kj = _key(scores[t, i]), _key(scores[t, j])
                G += ki > kj
                E += ki == kj
                N += 1
    return G, E, N


def test_perfect_separation_reversal_and_ties(orc):
    C, S = 7, 6
    sc = inputs.scores(C, S, seed=0, mal=(3,), gap=2.0)
    counts, pooled = orc.auroc_config(sc, _mask([3]))
    assert counts[0] == counts[2] == C * 5 and counts[1] == 0
    assert orc.auroc_strict(counts) == 1.0 and pooled[0] == pooled[2]
    sc = inputs.scores(C, S, seed=0, mal=(3,), gap=-2.0)
    counts, pooled = orc.auroc_config(sc, _mask([3]))
    assert counts[0] == 0 and counts[1] == 0 and pooled[0] == 0
    sc = np.full((C, S), 0.25, np.float32)
    counts, pooled = orc.auroc_config(sc, _mask([3]))
    assert orc.auroc_strict(counts) == 0.0 and orc.auroc_mw(counts) == 0.5
    assert pooled[1] == pooled[2]


def test_matches_sklearn_per_canary(orc):
    """Eq. 6 with ties counted one half is the mean of per-canary ROC AUCs."""
    C, S = 40, 9
    pos = (2, 6)
    sc = inputs.scores(C, S, seed=1, mal=pos, gap=0.3, tie_levels=12)
    counts, _ = orc.auroc_config(sc, _mask(pos))
    labels = np.zeros(S, int)
    labels[list(pos)] = 1
    want = np.mean([roc_auc_score(labels, sc[t]) for t in range(C)])
    assert abs(orc.auroc_mw(counts) - want) < 1e-12


def test_pooled_matches_scipy_mannwhitneyu(orc):
    C, S = 30, 8
    pos = (4,)
    sc = inputs.scores(C, S, seed=2, mal=pos, gap=0.1, tie_levels=20)
    _, pooled = orc.auroc_config(sc, _mask(pos))
    x = sc[:, list(pos)].ravel()
    y = np.delete(sc, list(pos), axis=1).ravel()
    U = stats.mannwhitneyu(x, y, alternative="two-sided", method="asymptotic").statistic
    assert pooled[0] + pooled[1] / 2 == U
    assert pooled[2] == x.size * y.size


def test_exhaustive_label_sets_with_ties(orc):
    """Every non-trivial malicious set for k <= 6, forced ties and NaNs."""
    for S in (2, 3, 4, 6):
        sc = inputs.scores(5, S, seed=S, tie_levels=3, nan_frac=0.1)
        for r in range(1, S):
            for pos in itertools.combinations(range(S), r):
                counts, pooled = orc.auroc_config(sc, _mask(pos), flags=2)
                assert tuple(int(x) for x in counts[:3]) == _brute(sc, set(pos))
                # pooled: every positive against every negative, across canaries
                flat_p = [sc[t, i] for t in range(sc.shape[0]) for i in pos]
                flat_n = [sc[t, j] for t in range(sc.shape[0]) for j in range(S) if j not in pos]
                G = sum(_key(p) > _key(n) for p in flat_p for n in flat_n)
                E = sum(_key(p) == _key(n) for p in flat_p for n in flat_n)
                assert (int(pooled[0]), int(pooled[1]), int(pooled[2])) == \
                    (G, E, len(flat_p) * len(flat_n))


def test_nan_and_signed_zero_order(orc):
    assert orc.score_cmp(float("nan"), math.inf) == 1
    assert orc.score_cmp(-math.inf, float("nan")) == -1
    assert orc.score_cmp(float("nan"), float("nan")) == 0
    assert orc.score_cmp(-0.0, 0.0) == 0
    assert orc.score_cmp(math.inf, 1e30) == 1


def test_scramble_draws_only_benign_stages_uniformly(orc):
    S, pos = 8, (4,)
    draws = [orc.scramble_jstar(S, _mask(pos), 0, 3, t) for t in range(7000)]
    assert 4 not in draws
    counts = np.bincount(draws, minlength=S)
    benign = [j for j in range(S) if j not in pos]
    chi2 = stats.chisquare(counts[benign]).pvalue
    assert chi2 > 1e-4
    # collusion: j* is never a colluder
    draws = [orc.scramble_jstar(S, _mask((1, 5)), 0, 3, t) for t in range(500)]
    assert not ({1, 5} & set(draws))
    assert orc.scramble_jstar(3, _mask((0, 1, 2)), 0, 0, 0) == -1


def test_control_counts_follow_definition(orc):
    C, S, pos = 25, 6, (3,)
    sc = inputs.scores(C, S, seed=4, tie_levels=5)
    for include_true in (False, True):
        flags = 1 | (4 if include_true else 0)
        counts, _ = orc.auroc_config(sc, _mask(pos), seed=11, cfg_id=7, flags=flags)
        G = E = N = 0
        for t in range(C):
            js = orc.scramble_jstar(S, _mask(pos), 11, 7, t)
            for j in range(S):
                if j == js or (j in pos and not include_true):
                    continue
                G += _key(sc[t, js]) > _key(sc[t, j])
                E += _key(sc[t, js]) == _key(sc[t, j])
                N += 1
        assert tuple(int(x) for x in counts[3:]) == (G, E, N)


def test_control_is_chance_on_the_true_scores(orc):
    """Scrambling the label on scores where the malicious stage stands out
    gives E[A] = 0.5 when the true stage is left out of the negatives, and
    (k - 2) / (2 (k - 1)) when it is kept in."""
    with open(os.path.join(GOLDEN, "paper_outcomes.json")) as f:
        gold = json.load(f)
    lo, hi = gold["control_window"]["value"]
    C, S, pos = 4000, 8, (4,)
    sc = inputs.scores(C, S, seed=5, mal=pos, gap=5.0)
    counts, _ = orc.auroc_config(sc, _mask(pos), seed=0, cfg_id=1, flags=1)
    a_ctrl = counts[3] / counts[5]
    assert lo <= a_ctrl <= hi and abs(a_ctrl - 0.5) < 0.02
    assert orc.auroc_strict(counts) >= gold["success_auroc"]["value"]
    counts, _ = orc.auroc_config(sc, _mask(pos), seed=0, cfg_id=1, flags=1 | 4)
    assert abs(counts[3] / counts[5] - (S - 2) / (2 * (S - 1))) < 0.02


def test_degenerate_label_sets(orc):
    sc = inputs.scores(3, 4, seed=6)
    counts, pooled = orc.auroc_config(sc, 0)  # nobody malicious
    assert counts[2] == 0 and pooled[2] == 0 and math.isnan(orc.auroc_strict(counts))
    counts, pooled = orc.auroc_config(sc, 0b1111)  # everybody malicious
    assert counts[2] == 0 and counts[5] == 0
    counts, _ = orc.auroc_config(inputs.scores(3, 1, seed=7), 0b1)  # a single stage
    assert counts[2] == 0
    with pytest.raises(ValueError):
        orc.auroc_config(inputs.scores(2, 65, seed=8), 1)


@pytest.mark.parametrize("flags,base", [(1 | 8, 0), (1 | 4 | 8, 0), (1 | 8, 1000), (0, 7)])
def test_per_canary_counts_brute_force(orc, flags, base):
    """Eq. 5 per canary (A^(t) = G_t / (|M| |N|)): every canary's detector,
    control and random-baseline counts equal a pure-Python count over that
    canary's pairs, with ties and NaNs, the control's chosen stage and the
    baseline's uniforms taken from the oracle's draws for the canary's
    global index; summed over canaries they give the configuration totals."""
    C, S = 9, 7
    pos = (1, 4)
    sc = inputs.scores(C, S, seed=5, mal=pos, gap=0.1, tie_levels=5)
    sc[2, 3] = np.nan
    sc[5, 1] = np.nan
    sc[6, :] = -0.0
    sc[6, 2] = 0.0
    mask = _mask(pos)
    got = orc.auroc_canaries(sc, mask, seed=3, cfg_id=11, canary_base=base, flags=flags)
    assert got.shape == (C, 6) and got.dtype == np.uint32
    neg = [j for j in range(S) if j not in pos]
    for t in range(C):
        G, E, _ = _brute(sc[t:t + 1], pos)
        want = [G, E, 0, 0, 0, 0]
        if flags & 1:
            js = orc.scramble_jstar(S, mask, 3, 11, base + t)
            others = [j for j in range(S) if j != js and (flags & 4 or j not in pos)]
            kj = _key(sc[t, js])
            want[2] = sum(kj > _key(sc[t, j]) for j in others)
            want[3] = sum(kj == _key(sc[t, j]) for j in others)
        if flags & 8:
            u = [orc.random_score(3, 11, base + t, s) for s in range(S)]
            want[4] = sum(u[i] > u[j] for i in pos for j in neg)
            want[5] = sum(u[i] == u[j] for i in pos for j in neg)
        np.testing.assert_array_equal(got[t], want, err_msg=f"canary {t}")
    if base == 0:
        counts, _ = orc.auroc_config(sc, mask, seed=3, cfg_id=11, flags=flags & 5)
        tot = got.astype(np.uint64).sum(axis=0)
        assert tot[0] == counts[0] and tot[1] == counts[1]
        if flags & 1:
            assert tot[2] == counts[3] and tot[3] == counts[4]
        if flags & 8:
            b = orc.random_baseline(C, S, mask, seed=3, cfg_id=11)
            assert tot[4] == b[0] and tot[5] == b[1]


def test_per_canary_rejects_more_than_64_stages(orc):
    with pytest.raises(ValueError):
        orc.auroc_canaries(np.zeros((2, 65), np.float32), 1)


def test_per_canary_sums_are_the_totals_on_random_tables(orc):
    """Property over random tables (S 1..12, C 0..9, any positive set, ties,
    NaNs, both control variants): the per-canary counts of Eq. 5 add up to
    the configuration's totals, and each canary's detector counts never
    exceed its number of pairs."""
    from hypothesis import given, settings, strategies as st

    @settings(max_examples=150, deadline=None, derandomize=True)
    @given(S=st.integers(1, 12), C=st.integers(0, 9), mask_bits=st.integers(0, (1 << 12) - 1),
           levels=st.integers(1, 6), nan_frac=st.sampled_from([0.0, 0.1]),
           include_true=st.booleans(), seed=st.integers(0, 2**31))
    def check(S, C, mask_bits, levels, nan_frac, include_true, seed):
        rng = np.random.default_rng(seed)
        sc = (rng.integers(0, levels, (C, S)) / levels).astype(np.float32)
        sc[rng.random((C, S)) < nan_frac] = np.nan
        mask = mask_bits & ((1 << S) - 1)
        flags = 1 | 8 | (4 if include_true else 0)
        per = orc.auroc_canaries(sc, mask, seed=seed, cfg_id=3, flags=flags)
        counts, _ = orc.auroc_config(sc, mask, seed=seed, cfg_id=3, flags=flags & 5)
        n_pos = bin(mask).count("1")
        tot = per.astype(np.uint64).sum(axis=0) if C else np.zeros(6, np.uint64)
        assert tot[0] == counts[0] and tot[1] == counts[1]
        assert tot[2] == counts[3] and tot[3] == counts[4]
        base = orc.random_baseline(C, S, mask, seed=seed, cfg_id=3)
        assert tot[4] == base[0] and tot[5] == base[1]
        if C:
            assert np.all(per[:, 0] + per[:, 1] <= n_pos * (S - n_pos))

    check()
