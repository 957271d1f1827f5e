"""A scalar Monte Carlo model of the detector's outcomes, for the statistical
tests of the substudies, of the SNR curve and of Table 1 (Sections 3.1-3.4,
4.4, 5.2-5.5).

Neither the oracle nor the device path is used: the model draws, per
(replicate, canary, stage), the few block-level quantities the drift scores
depend on and combines them with the laws the generator obeys, and from
them the detection AUROC (Eqs. 5-6) and the score summaries the benchmark
reports.  What it encodes:

* the generator's unit normal z: the Irwin-Hall sum of four uniforms,
  centred and scaled to unit variance (bounded at +-2 sqrt 3; E|z| =
  7 sqrt(3) / 15 and E z^4 = 2.7, against sqrt(2 / pi) and 3 for a normal),
  used for the references, the noise and the tamper alike;
* references a = gain_j z, n_out outlier channels at gain G and the rest at
  1; per block the energy A = sum a^2 and the absolute sum U = sum |a| are
  drawn: the outlier elements' energy from a gamma law with the exact mean
  and variance, everything else through the normal limit with the exact
  means, variances and covariance of (z^2, |z|);
* block-scaled benign noise (Eq. 2, block mode): scale sigma U / n, energy
  scale^2 sum z^2;
* elementwise benign noise sigma |a| z (Eq. 2): W = sum a^2 z^2 / sum a^2
  through its normal limit; with Student-t noise (nu = 3, the generator's
  z0 / sqrt(z1^2 + z2^2 + z3^2) of four of its normals) the elements whose
  denominator q falls below a cut q0 are drawn one by one (they carry the
  heavy tail) and the rest through the normal limit of the truncated
  moments, which a quadrature of the Irwin-Hall density gives exactly;
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
  part relative to h is that of v), and the per-element Gaussian tamper
  eps rms(a) z';
* the scores: Eq. 4, m = sqrt(E / A); the cosine mismatch, monotone in the
  angular energy over A (its AUROC is what the model predicts).

The small-error expansions hold while the relative errors stay well below
1, which covers every configuration tested.  Every draw is seeded."""
import functools
import math

import numpy as np

SQ3 = math.sqrt(3.0)
_GL_X, _GL_W = np.polynomial.legendre.leggauss(24)


def ih_density(x):
    """Density of the generator's unit normal: s = 2 + x / sqrt(3) is the
    sum of four U(0, 1), with the Irwin-Hall density
    (1/6) sum_k (-1)^k C(4, k) (s - k)_+^3 on [0, 4]."""
    s = 2.0 + np.asarray(x, float) / SQ3
    f = np.zeros_like(s)
    for k, c in enumerate((1, -4, 6, -4, 1)):
        f += c * np.maximum(s - k, 0.0) ** 3
    return np.where((s > 0) & (s < 4), f / 6.0, 0.0) / SQ3


def normal_density(x):
    return np.exp(-0.5 * np.asarray(x, float) ** 2) / math.sqrt(2.0 * math.pi)


def ih_moment(g):
    """E g(z) for the Irwin-Hall normal: Gauss-Legendre on each cubic piece
    of its density (exact for polynomial g up to degree 43)."""
    tot = 0.0
    for k in range(4):
        lo, hi = (k - 2) * SQ3, (k - 1) * SQ3
        x = lo + (hi - lo) * (_GL_X + 1) / 2
        tot += ((hi - lo) / 2 * _GL_W * g(x) * ih_density(x)).sum()
    return float(tot)


IH_ABS = ih_moment(np.abs)                      # E|z| = 7 sqrt(3) / 15
IH_ABS3 = ih_moment(lambda x: np.abs(x) ** 3)   # E|z|^3
IH_K4 = ih_moment(lambda x: x ** 4)             # E z^4 = 2.7


def ih_draw(rng, size):
    """Irwin-Hall normals (the continuous limit of the generator's 16-bit
    lattice, whose spacing is 2.6e-5)."""
    size = (size,) if isinstance(size, int) else tuple(size)
    return (rng.random(size + (4,)).sum(-1) - 2.0) * SQ3


def ih_sq_sum(rng, n, size):
    """sum of n squared Irwin-Hall normals: a gamma law with their mean n and
    variance (E z^4 - 1) n."""
    v = IH_K4 - 1.0
    return rng.gamma(n / v, v, size=size)


def shell_density(p, r, n_ang=40):
    """F(r) = integral over the unit sphere of p(r u1) p(r u2) p(r u3): the
    density of |z| for three independent draws of density p is r^2 F(r)."""
    c, wc = np.polynomial.legendre.leggauss(n_ang)
    c, wc = (c + 1) / 2, wc / 2                      # cos(theta) in [0, 1]
    ph, wp = np.polynomial.legendre.leggauss(n_ang)
    ph, wp = (ph + 1) * math.pi / 4, wp * math.pi / 4  # phi in [0, pi/2]
    st = np.sqrt(1 - c * c)
    u1 = (st[:, None] * np.cos(ph)[None, :]).ravel()
    u2 = (st[:, None] * np.sin(ph)[None, :]).ravel()
    u3 = np.repeat(c, n_ang)
    w = 8.0 * (wc[:, None] * wp[None, :]).ravel()  # the eight octants (p even)
    r = np.asarray(r, float)[:, None]
    return (p(r * u1) * p(r * u2) * p(r * u3) * w).sum(axis=1)


def radial_integral(p, g, a, b, panels=48):
    """int_a^b g(r) F(r) dr, Gauss-Legendre on panels (geometric from a > 0)."""
    edges = np.geomspace(a, b, panels + 1) if a > 0 else np.linspace(a, b, panels + 1)
    tot = 0.0
    for lo, hi in zip(edges[:-1], edges[1:]):
        r = lo + (hi - lo) * (_GL_X + 1) / 2
        tot += ((hi - lo) / 2 * _GL_W * g(r) * shell_density(p, r)).sum()
    return float(tot)


@functools.lru_cache(maxsize=None)
def t3_cut_moments(q0, p=ih_density, rmax=6.0):
    """For q = z1^2 + z2^2 + z3^2 of three independent draws of density p:
    (P(q < q0), E[1/q; q >= q0], E[1/q^2; q >= q0]).  With the normal density
    these are the chi-square(3) values; rmax = 6 covers the Irwin-Hall
    support (|z_i| <= 2 sqrt 3)."""
    r0 = math.sqrt(q0)
    return (radial_integral(p, lambda r: r * r, 0.0, r0),
            radial_integral(p, lambda r: np.ones_like(r), r0, rmax),
            radial_integral(p, lambda r: r ** -2.0, r0, rmax))


def fp16_rel_mse(H, n_out, gain_big, rng, n=1 << 20):
    """rho^2: E[(fl16(a) - a)^2] / E[a^2] for the reference distribution."""
    j = rng.integers(0, H, n)
    a = ih_draw(rng, n) * np.where(j < n_out, gain_big, 1.0)
    r = a.astype(np.float16).astype(np.float64) - a
    return float((r * r).sum() / (a * a).sum())


def block_stats(rng, shape, T, H, n_out, gain_big):
    """(A, U) per block: energy and absolute sum of T x H references.  The
    outlier elements' sum of squares is drawn from its gamma law and their
    absolute sum from its normal law given that sum (slope and residual
    variance of the joint limit of (z^2, |z|))."""
    var_sq, cov_sa, var_abs = IH_K4 - 1.0, IH_ABS3 - IH_ABS, 1.0 - IH_ABS ** 2
    n1 = T * (H - n_out)
    m1 = np.array([n1, n1 * IH_ABS])
    cov = n1 * np.array([[var_sq, cov_sa], [cov_sa, var_abs]])
    x = rng.multivariate_normal(m1, cov, size=shape)
    A, U = x[..., 0], x[..., 1]
    n2 = T * n_out
    if n2:
        q = ih_sq_sum(rng, n2, shape)
        slope = cov_sa / var_sq
        r = n2 * IH_ABS + slope * (q - n2) + \
            math.sqrt(n2 * (var_abs - slope * cov_sa)) * rng.standard_normal(shape)
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
    noise = bsc ** 2 * ih_sq_sum(rng, n, shape)
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


T3_CUTS = (0.002, 0.05)  # q0 of the Student-t tail: normal channels, outlier channels


def elementwise_energy(rng, shape, T, H, n_out, gain_big, dist="gauss", cuts=T3_CUTS):
    """W = sum a^2 z^2 / sum a^2 per block, z the elementwise benign noise
    draw (Gaussian, or Student-t with nu = 3).  Per channel class (count k,
    gain g) the pair (sum a^2, sum a^2 z^2) is drawn from its normal limit:
    means k g^2 (1, mu1), covariance k g^4 [[K4 - 1, (K4 - 1) mu1],
    [(K4 - 1) mu1, K4 m4 - mu1^2]], with mu1 = E z^2 = 1 and m4 = E z^4 =
    K4 for Gaussian noise.  For Student-t noise z = z0 / sqrt(q) and the
    truncated moments mu1 = E[1/q; q >= q0], m4 = K4 E[1/q^2; q >= q0];
    the elements with q < q0 (a Poisson count at rate k P(q < q0)) are drawn
    one by one: a and z0 from the Irwin-Hall law and q from its law near
    zero, density proportional to sqrt(q) (the density of the three
    normals is flat to within q0 there)."""
    A = np.zeros(shape)
    N = np.zeros(shape)
    for k, g, cut in ((T * (H - n_out), 1.0, cuts[0]), (T * n_out, gain_big, cuts[1])):
        if k == 0:
            continue
        if dist == "gauss":
            p0, mu1, m4 = 0.0, 1.0, IH_K4
        elif dist == "t3":
            p0, mu1, inv2 = t3_cut_moments(cut)
            m4 = IH_K4 * inv2
        else:
            raise ValueError(dist)
        v = IH_K4 - 1.0
        cov = k * g ** 4 * np.array([[v, v * mu1], [v * mu1, IH_K4 * m4 - mu1 * mu1]])
        x = rng.multivariate_normal(np.array([k * g * g, k * g * g * mu1]), cov, size=shape)
        A += x[..., 0]
        N += x[..., 1]
        if p0 > 0.0:
            cnt = rng.poisson(k * p0, size=shape)
            flat = N.reshape(-1)
            per = cnt.reshape(-1)
            step = max(1, (1 << 23) // max(1, int(per.mean() + 1)))
            for b0 in range(0, per.size, step):
                c = per[b0:b0 + step]
                m = int(c.sum())
                z0, za = ih_draw(rng, m), ih_draw(rng, m)
                q = cut * rng.random(m) ** (2.0 / 3.0)
                idx = np.repeat(np.arange(c.size), c)
                flat[b0:b0 + step] += np.bincount(idx, weights=g * g * za * za * z0 * z0 / q,
                                                  minlength=c.size)
    return N / A


def simulate_elementwise(S, C, T, H, mal, *, sigma, eps, dist="gauss", n_out=None,
                         gain_big=20.0, reps=200, seed=0, w=None):
    """Eq. 4 scores of independent stages with elementwise benign noise
    sigma |a| z (Eq. 2; z Gaussian or Student-t) and the additive tamper
    eps rms(a) z' of the attackers (Eq. 3): m^2 = sigma^2 W + rho^2
    (+ eps^2 sum z'^2 / n + cross), W from elementwise_energy (or given:
    W does not depend on sigma, so one draw can serve a whole noise sweep).
    Returns (l2, mal_mask) as simulate() does."""
    rng = np.random.default_rng(seed)
    n_out = int(0.01 * H + 0.5) if n_out is None else n_out
    n = T * H
    rho2 = fp16_rel_mse(H, n_out, gain_big, rng)
    shape = (reps, C, S)
    Wn = elementwise_energy(rng, shape, T, H, n_out, gain_big, dist) if w is None else w
    m2 = sigma * sigma * Wn + rho2
    is_mal = np.zeros(S, bool)
    is_mal[list(mal)] = True
    k = int(is_mal.sum())
    t2 = eps * eps * ih_sq_sum(rng, n, (Wn.shape[0], C, k)) / n
    cross = 2.0 * sigma * eps * np.sqrt(Wn[..., is_mal] / n) * \
        rng.standard_normal((Wn.shape[0], C, k))
    m2[..., is_mal] += t2 + cross
    return np.sqrt(m2), is_mal
