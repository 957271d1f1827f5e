"""Statistical expectations (not parity) for the outcomes the device reports
on the paper's shape (12 stages x 100 canaries x 48 tokens x d = 768, block
noise): the depth, position, collusion, frontier and SNR substudies under
the propagation model (Sections 4.4, 5.3-5.5), the raised-noise-floor
curve of Section 5.4 at two further seeds (on its own 16 x 128 x 128 x 4096
shape, elementwise noise, 500 model replicates) and the cosine metric's AUROC
on the pure rescale in Table 1 (Section 5.2), each against the central
99.8% of the seeded Monte Carlo model in tests/drift_model.py (1000
replicates; the model uses neither the oracle nor the device).

AUROCs must fall inside the model's interval (an interval of [1, 1] asks for
exactly 1).  The score summaries (median attacker score, largest benign
score) may stray 0.5% past it: the model's expansions drop terms of relative
order 1/n and of the squared relative error, and the benchmark rounds them
to four digits.  The whole-configuration parity of these runs with the
oracle is in tests/test_gpu_chain.py and tests/test_gpu_workloads.py."""
import pytest

from paper_2607_19490_amd import workloads as W
from tests import drift_model as M
from tests.gpu_util import announce, require_gpu

pytestmark = [pytest.mark.gpu, pytest.mark.statistical]

REPS = 1000
SLACK = 0.005


@pytest.fixture(scope="module")
def gpu():
    return require_gpu()


def inside(x, lo, hi, slack=0.0):
    return lo * (1 - slack) <= x <= hi * (1 + slack)


def test_substudies_follow_the_model(gpu):
    torch, cdt = gpu
    import bench
    announce("substudies against the model")
    res = bench.substudies(torch, cdt, W)["studies"]
    wl = W.substudies()
    misses = []
    for k, rs in enumerate(wl.ref_sets):
        run = rs.runs[0]
        study, name = run.label.split(":")
        row = res[study][name]
        l2, _, im = M.simulate(rs.S, rs.C, rs.T, rs.H, rs.mal_shards, sigma=run.sigma_b,
                               carry=run.carry, attack="gauss", eps=run.eps, reps=REPS, seed=k)
        a_lo, a_hi = M.interval(M.auroc_strict(l2, im))
        med, mx = M.summaries(l2, im)
        checks = (("auroc", row["auroc"], (a_lo, a_hi), 0.0),
                  ("median_m_malicious", row["median_m_malicious"], M.interval(med), SLACK),
                  ("max_m_benign", row["max_m_benign"], M.interval(mx), SLACK))
        for key, got, (lo, hi), slack in checks:
            if not inside(got, lo, hi, slack):
                misses.append((run.label, key, got, lo, hi))
    assert not misses, misses


def test_table1_cosine_on_the_rescale_follows_the_model(gpu):
    """The cosine metric is blind to a pure rescale: with independent stages
    the rescaled stage's angular error is a benign one (AUROC near 0.5);
    with the live error carried between stages the stages after it inherit
    its (k - 1) a and rank above it, the ones before it have less carried
    error and rank below it, so the AUROC sits well under 0.5 (the paper's
    0.194 is on real models).  Eq. 4 sees the rescale in both."""
    torch, cdt = gpu
    import bench
    announce("table 1 cosine rescale against the model")
    t = bench.table1(torch, cdt, W)
    rs = W.paper().ref_sets[0]
    run = [r for r in rs.runs if r.label.startswith("rescale")][0]
    got = {0.0: t["per_attack"]["cosine_metric"][run.label]["auroc"],
           W.SUBSTUDY_CARRY: t["with_propagation"]["per_attack"][run.label]["auroc_cosine"]}
    for seed, carry in enumerate(sorted(got)):
        l2, cos, im = M.simulate(rs.S, rs.C, rs.T, rs.H, rs.mal_shards, sigma=run.sigma_b,
                                 carry=carry, attack="rescale", scale=run.scale, reps=REPS,
                                 seed=100 + seed)
        lo, hi = M.interval(M.auroc_strict(cos, im))
        assert lo <= got[carry] <= hi, (carry, got[carry], lo, hi)
        assert M.interval(M.auroc_strict(l2, im)) == (1.0, 1.0)
    assert t["with_propagation"]["per_attack"][run.label]["auroc_l2"] == 1.0


def test_snr_curve_of_further_seeds_follows_the_model(gpu):
    """The SNR study's 40 runs with seeds 1 and 2 (their own references and
    noise; seed 0 is the oracle's, tests/test_statistical_snr.py): the
    device's detection AUROCs lie inside the model's central 99.8%,
    Gaussian and Student-t noise alike.  Of the 80 checks at 0.2% each, 0.16
    miss by chance on average, so one miss is allowed; two or more have a
    chance of about 1.2% under the model."""
    import numpy as np
    torch, cdt = gpu
    import bench
    announce("snr curve, seeds 1 and 2, against the model")
    got = bench.snr_seeds(torch, cdt, W, seeds=(1, 2))["curve"]
    rs = W.snr().ref_sets[0]
    n_out = W.n_outliers(rs.H)
    w = M.elementwise_energy(np.random.default_rng(77), (500, rs.C, rs.S), rs.T, rs.H, n_out,
                             20.0, "t3")
    misses = []
    for r, run in enumerate(rs.runs):
        if run.benign_dist == W.DIST_T3:
            l2, im = M.simulate_elementwise(rs.S, rs.C, rs.T, rs.H, rs.mal_shards,
                                            sigma=run.sigma_b, eps=run.eps, dist="t3",
                                            seed=300 + r, w=w)
        else:
            l2, im = M.simulate_elementwise(rs.S, rs.C, rs.T, rs.H, rs.mal_shards,
                                            sigma=run.sigma_b, eps=run.eps, reps=500,
                                            seed=300 + r)
        lo, hi = M.interval(M.auroc_strict(l2, im))
        for a in got[run.label]["auroc"]:
            if not lo <= a <= hi:
                misses.append((run.label, a, lo, hi))
    assert len(misses) <= 1, misses
