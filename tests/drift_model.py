"""A scalar Monte Carlo model of the detector's outcomes, for the statistical
tests of the substudies and of Table 1 (Sections 3.1-3.4, 4.4, 5.2-5.5).

Neither the oracle nor the device path is used: the model draws, per
(replicate, canary, stage), the few block-level quantities the drift scores
depend on and combines them with the laws the generator obeys, and from
them the detection AUROC (Eqs. 5-6) and the score summaries the benchmark
reports.  What it encodes:

* references a = gain_j z (z ~ N(0, 1)), n_out outlier channels at gain G
  and the rest at 1; per block the energy A = sum a^2 and the absolute sum
  U = sum |a| are drawn: the outlier elements' energy exactly (chi-square),
  everything else through the normal limit with the exact means, variances
  and covariance of (z^2, |z|);
* block-scaled benign noise (Eq. 2, block mode): scale sigma U / n, energy
  scale^2 chi2_n;
* fp16 rounding of the stage output: energy rho^2 A, rho^2 the relative
  mean squared RNE error of the reference distribution (measured on a
  numpy float16 cast of a sample of it);
* the propagation model: the error energy of stage s is g^2 times the
  previous stage's plus the stage's own (the carry law e_s = delta_s +
  g e_{s-1}), with the cross term of the carried error and the new noise
  drawn from its normal law; the carried error is orthogonal to the stage's
  own reference (independent draws), so all of it is angular error;
* the attacks (Eq. 3): the exact-norm Gaussian eps ||v|| U/||U|| (energy
  eps^2 ||v||^2, all of it angular), the full sign flip h = -v and the
  rescale h = k v (error (k - 1) a + k (carried + noise), whose angular
  part relative to h is that of v);
* the scores: Eq. 4, m = sqrt(E / A); the cosine mismatch, monotone in the
  angular energy over A (its AUROC is what the model predicts).

The small-error expansions hold while the relative errors stay well below
1, which covers every configuration tested.  Every draw is seeded."""
import math

import numpy as np

SQ2PI = math.sqrt(2.0 / math.pi)


def fp16_rel_mse(H, n_out, gain_big, rng, n=1 << 20):
    """rho^2: E[(fl16(a) - a)^2] / E[a^2] for the reference distribution."""
    j = rng.integers(0, H, n)
    a = rng.standard_normal(n) * np.where(j < n_out, gain_big, 1.0)
    r = a.astype(np.float16).astype(np.float64) - a
    return float((r * r).sum() / (a * a).sum())


def block_stats(rng, shape, T, H, n_out, gain_big):
    """(A, U) per block: energy and absolute sum of T x H references.  The
    outlier elements' sum of squares is drawn exactly (chi-square) and their
    absolute sum from its normal law given that sum (slope and residual
    variance of the joint limit of (z^2, |z|))."""
    n1 = T * (H - n_out)
    m1 = np.array([n1, n1 * SQ2PI])
    cov = np.array([[2.0 * n1, n1 * SQ2PI], [n1 * SQ2PI, n1 * (1.0 - 2.0 / math.pi)]])
    x = rng.multivariate_normal(m1, cov, size=shape)
    A, U = x[..., 0], x[..., 1]
    n2 = T * n_out
    if n2:
        q = rng.chisquare(n2, size=shape)
        r = n2 * SQ2PI + 0.5 * SQ2PI * (q - n2) + \
            math.sqrt(n2 * (1.0 - 3.0 / math.pi)) * rng.standard_normal(shape)
        A = A + gain_big ** 2 * q
        U = U + gain_big * r
    return A, U


def simulate(S, C, T, H, mal, *, sigma, carry=0.0, attack="gauss", eps=0.0, scale=1.0,
             n_out=None, gain_big=20.0, reps=200, seed=0):
    """Scores of `reps` replicates of one configuration.

    Returns (l2, cos, mal_mask): arrays [reps, C, S] of the Eq. 4 score m and
    of the angular error energy over A (the cosine mismatch's order), and the
    boolean stage mask of the attackers."""
    rng = np.random.default_rng(seed)
    n_out = int(0.01 * H + 0.5) if n_out is None else n_out
    n = T * H
    rho2 = fp16_rel_mse(H, n_out, gain_big, rng)
    shape = (reps, C, S)
    A, U = block_stats(rng, shape, T, H, n_out, gain_big)
    bsc = sigma * U / n
    noise = bsc ** 2 * rng.chisquare(n, size=shape)
    is_mal = np.zeros(S, bool)
    is_mal[list(mal)] = True
    E = np.zeros(shape)  # error energy of each stage's output
    P = np.zeros(shape)  # its angular part
    prev = np.zeros((reps, C))
    for s in range(S):
        carried = carry * carry * prev
        # cross term of the carried error and this stage's noise
        cross = 2.0 * carry * np.sqrt(prev) * bsc[..., s] * rng.standard_normal((reps, C))
        pre = carried + noise[..., s] + cross  # v - a before rounding
        rnd = rho2 * A[..., s]
        if not is_mal[s]:
            E[..., s] = pre + rnd
            P[..., s] = pre + rnd
        elif attack == "gauss":
            v2 = A[..., s] + pre
            t2 = eps * eps * v2
            cross_t = 2.0 * np.sqrt(np.maximum(pre, 0) * t2 / n) * rng.standard_normal((reps, C))
            E[..., s] = pre + t2 + cross_t + rnd
            P[..., s] = E[..., s]
        elif attack == "rescale":
            k = scale
            par = (k - 1.0) ** 2 * A[..., s]
            cross_a = 2.0 * (k - 1.0) * k * np.sqrt(A[..., s] * pre / n) * \
                rng.standard_normal((reps, C))
            E[..., s] = par + k * k * pre + cross_a + k * k * rnd
            P[..., s] = pre + rnd  # the angle of v: a rescale keeps it
        elif attack == "signflip":
            E[..., s] = 4.0 * A[..., s] + pre + rnd
            P[..., s] = 4.0 * A[..., s]  # cos = -1: the largest mismatch there is
        else:
            raise ValueError(attack)
        prev = E[..., s]
    l2 = np.sqrt(np.maximum(E, 0) / A)
    cos = P / A
    return l2, cos, is_mal


def auroc_strict(scores, is_mal):
    """Eq. 6 (strict) per replicate: the share of (attacker, benign) pairs of
    one canary in which the attacker's score is the larger."""
    m = scores[..., is_mal]          # [reps, C, n_mal]
    b = scores[..., ~is_mal]         # [reps, C, n_ben]
    g = (m[..., :, None] > b[..., None, :]).sum(axis=(1, 2, 3))
    return g / (scores.shape[1] * m.shape[-1] * b.shape[-1])


def summaries(l2, is_mal):
    """Per replicate: the median attacker score and the largest benign one."""
    return (np.median(l2[..., is_mal].reshape(l2.shape[0], -1), axis=1),
            l2[..., ~is_mal].reshape(l2.shape[0], -1).max(axis=1))


def interval(x, lo=0.001, hi=0.999):
    return float(np.quantile(x, lo)), float(np.quantile(x, hi))


def simulate_elementwise(S, C, T, H, mal, *, sigma, eps, n_out=None, gain_big=20.0, reps=200,
                         seed=0):
    """Eq. 4 scores of independent stages with Gaussian elementwise benign
    noise sigma |a| z (Eq. 2) and the additive tamper eps rms(a) z' of the
    attackers (Eq. 3): m^2 = sigma^2 W + rho^2 (+ eps^2 chi2_n / n + cross),
    with W = sum a^2 z^2 / sum a^2 drawn per channel class from the normal
    limit of (z'^2, z'^2 z^2) (means 1 and 1, variances 2 and 8, covariance
    2; a = gain z').  Returns (l2, mal_mask) as simulate() does."""
    rng = np.random.default_rng(seed)
    n_out = int(0.01 * H + 0.5) if n_out is None else n_out
    n = T * H
    rho2 = fp16_rel_mse(H, n_out, gain_big, rng)
    shape = (reps, C, S)
    cov = np.array([[2.0, 2.0], [2.0, 8.0]])

    def sums(k):
        if k == 0:
            return np.zeros(shape), np.zeros(shape)
        x = rng.multivariate_normal(np.array([k, k], float), cov * k, size=shape)
        return x[..., 0], x[..., 1]

    A1, N1 = sums(T * (H - n_out))
    A2, N2 = sums(T * n_out)
    A = A1 + gain_big ** 2 * A2
    Wn = (N1 + gain_big ** 2 * N2) / A
    m2 = sigma * sigma * Wn + rho2
    is_mal = np.zeros(S, bool)
    is_mal[list(mal)] = True
    k = int(is_mal.sum())
    t2 = eps * eps * rng.chisquare(n, size=(reps, C, k)) / n
    cross = 2.0 * sigma * eps * np.sqrt(Wn[..., is_mal] / n) * rng.standard_normal((reps, C, k))
    m2[..., is_mal] += t2 + cross
    return np.sqrt(m2), is_mal
