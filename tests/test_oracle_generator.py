"""Pins of the oracle's synthetic generator (CPU only).

The references stand in for the fp32 activations of Eq. 1 and the live pass
follows Eqs. 2-3.  What the paper and the mathematics fix, checked here:
  * special cases that reduce to numpy's fp16 conversion (sigma = 0, clean
    base, full sign flip, power-of-two rescale);
  * the noise scale of Eq. 2 (elementwise and block-scaled), the Student-t
    tails, the Gaussian tamper magnitude m ~ eps, the flip fraction and
    m ~ 2 sqrt(p), the rescale m ~ alpha;
  * the outlier channel choice against an independent sort.
"""
import math
import warnings

import numpy as np
import pytest
from scipy import stats

NOISE_ELEMENTWISE, NOISE_BLOCK = 0, 1
DIST_GAUSS, DIST_T3 = 0, 1
T_ADD, T_FLIP, T_SCALE = 1, 2, 4
BASE_BENIGN, BASE_CLEAN = 0, 1


def _f16(x):
    with warnings.catch_warnings():
        warnings.simplefilter("ignore")
        return np.asarray(x, np.float32).astype(np.float16).view(np.uint16)


def _h(bits):
    return np.asarray(bits, np.uint16).view(np.float16).astype(np.float64)


def _ref(orc, T=64, H=512, s=0, c=0, seed=3, gain=None):
    if gain is None:
        gain = np.ones(H, np.float32)
    return orc.ref_block(s, c, T, H, seed, 0, gain)


def _rel(h_bits, a):
    d = _h(h_bits) - a.astype(np.float64)
    return math.sqrt((d * d).sum() / (a.astype(np.float64) ** 2).sum())


# ----------------------------------------------------------------------------
# references and outlier channels
# ----------------------------------------------------------------------------
def test_outlier_channels_are_the_smallest_words(orc, philox_pin):
    H, n_out = 4096, 41
    g = orc.outlier_gain(H, n_out, 20.0, 5, 2)
    ctr = np.zeros((H, 4), np.uint32)
    ctr[:, 0] = np.arange(H)
    ctr[:, 3] = (8 << 24) | 2
    words = philox_pin(ctr, np.tile(np.array([5, 0], np.uint32), (H, 1)))[:, 0].astype(np.uint64)
    order = np.lexsort((np.arange(H), words))  # by word, then channel
    want = np.ones(H, np.float32)
    want[order[:n_out]] = 20.0
    np.testing.assert_array_equal(g, want)
    assert (g == 20.0).sum() == n_out


def test_outlier_zero_and_all(orc):
    assert np.all(orc.outlier_gain(256, 0, 20.0, 0, 0) == 1.0)
    assert np.all(orc.outlier_gain(256, 256, 20.0, 0, 0) == 20.0)
    with pytest.raises(ValueError):
        orc.outlier_gain(8, 9, 20.0, 0, 0)


def test_reference_gain_and_variance(orc):
    H = 1024
    gain = orc.outlier_gain(H, 10, 20.0, 0, 0)
    a = _ref(orc, T=256, H=H, gain=gain)
    out = gain == 20.0
    # each channel holds z * gain: outlier channels have variance 400
    v_in = a[:, ~out].astype(np.float64).var()
    v_out = a[:, out].astype(np.float64).var()
    assert abs(v_in - 1.0) < 0.02
    assert abs(v_out / 400.0 - 1.0) < 0.1
    # gain 20 multiplies exactly the unit-gain draw of the same element, rounded
    z = _ref(orc, T=256, H=H)
    np.testing.assert_array_equal(a[:, out], (z[:, out].astype(np.float64) * 20.0).astype(np.float32))
    np.testing.assert_array_equal(a[:, ~out], z[:, ~out])


def test_reference_blocks_are_distinct_and_deterministic(orc):
    a00 = _ref(orc, T=8, H=64, s=0, c=0)
    a01 = _ref(orc, T=8, H=64, s=0, c=1)
    a10 = _ref(orc, T=8, H=64, s=1, c=0)
    assert not np.array_equal(a00, a01) and not np.array_equal(a00, a10)
    np.testing.assert_array_equal(a00, _ref(orc, T=8, H=64, s=0, c=0))
    # whole-array generator lays blocks out as [S][C][T][H]
    full = orc.ref_synth(2, 2, 8, 64, 3, 0, np.ones(64, np.float32))
    np.testing.assert_array_equal(full[0, 1], a01)
    np.testing.assert_array_equal(full[1, 0], a10)


# ----------------------------------------------------------------------------
# counter layout of every stream, against rocRAND's Philox4x32-10
# ----------------------------------------------------------------------------
K16 = np.float32(math.sqrt(3.0 / (2.0**32 - 1.0)))


def _ih(w0, w1):
    """Irwin-Hall normal from two words (its moments are pinned above)."""
    w0 = w0.astype(np.int64)
    w1 = w1.astype(np.int64)
    n = (w0 & 0xFFFF) + (w0 >> 16) + (w1 & 0xFFFF) + (w1 >> 16) - 131070
    return n.astype(np.float32) * K16


def _words(philox_pin, q, c, s, stream, cid, seed):
    q = np.asarray(q, np.uint64)
    ctr = np.zeros((q.size, 4), np.uint32)
    ctr[:, 0] = q
    ctr[:, 1] = c
    ctr[:, 2] = s
    ctr[:, 3] = (stream << 24) | cid
    key = np.tile(np.array([seed & 0xFFFFFFFF, seed >> 32], np.uint32), (q.size, 1))
    return philox_pin(ctr, key)


def _one_normal(philox_pin, e, c, s, stream, cid, seed):
    """Element e draws call q = e / 2: words 0-1 for even e, 2-3 for odd e."""
    w = _words(philox_pin, e // 2, c, s, stream, cid, seed)
    odd = (e % 2) == 1
    return np.where(odd, _ih(w[:, 2], w[:, 3]), _ih(w[:, 0], w[:, 1]))


@pytest.mark.parametrize("s,c", [(0, 0), (3, 1), (1, 6)])
def test_stream_counters_against_rocrand(orc, philox_pin, s, c):
    """Each stream's draw for element e of block (s, c) is the Philox call
    with counter (q, c, s, stream << 24 | id) under key (lo32 seed, hi32
    seed), with q and the words used as the generator's spec states.
    rocRAND's Philox (an independent library routine) supplies the words;
    each stream is made visible through a case where it alone sets the
    output."""
    T, H, seed, cid = 4, 64, (7 << 32) | 11, 5
    e = np.arange(T * H)
    zero = np.zeros((T, H), np.float32)
    # REF: with unit gains the reference is the normal itself
    a = orc.ref_block(s, c, T, H, seed, cid, np.ones(H, np.float32))
    np.testing.assert_array_equal(a.ravel(), _one_normal(philox_pin, e, c, s, 0, cid, seed))
    # BENIGN: a = 0 and block scale 1 give h = fp16(z_BENIGN)
    h = orc.sim_block(s, c, zero, seed=seed, cfg_id=cid, benign_mode=NOISE_BLOCK, bscale=1.0)
    np.testing.assert_array_equal(h.ravel(), _f16(_one_normal(philox_pin, e, c, s, 1, cid, seed)))
    # ALT (independent recompute): the same with stream 9
    h = orc.sim_block(s, c, zero, seed=seed, cfg_id=cid, benign_mode=NOISE_BLOCK, bscale=1.0,
                      redraw=True)
    np.testing.assert_array_equal(h.ravel(), _f16(_one_normal(philox_pin, e, c, s, 9, cid, seed)))
    # TAMPER_ADD: clean base a = 0 and scale 1 give h = fp16(z_TADD)
    h = orc.sim_block(s, c, zero, seed=seed, cfg_id=cid, sigma_b=0.0, malicious=True,
                      tamper=T_ADD, tscale=1.0, tamper_base=BASE_CLEAN)
    np.testing.assert_array_equal(h.ravel(), _f16(_one_normal(philox_pin, e, c, s, 4, cid, seed)))
    # TAMPER_FLIP: element e uses word e % 4 of call e / 4; p = 1/2 flips u < 2^31
    one = np.ones((T, H), np.float32)
    h = orc.sim_block(s, c, one, seed=seed, cfg_id=cid, sigma_b=0.0, malicious=True,
                      tamper=T_FLIP, flip_p=0.5)
    w = _words(philox_pin, e // 4, c, s, 5, cid, seed)
    u = w[np.arange(e.size), e % 4]
    np.testing.assert_array_equal(h.ravel(), _f16(np.where(u < 2**31, -1.0, 1.0)))
    # Student-t: T12 call q = e (words 0-1, 2-3), T3 one normal per element
    h = orc.sim_block(s, c, zero, seed=seed, cfg_id=cid, benign_mode=NOISE_BLOCK, bscale=1.0,
                      benign_dist=DIST_T3)
    z0 = _one_normal(philox_pin, e, c, s, 1, cid, seed)
    w12 = _words(philox_pin, e, c, s, 2, cid, seed)
    z1, z2 = _ih(w12[:, 0], w12[:, 1]), _ih(w12[:, 2], w12[:, 3])
    z3 = _one_normal(philox_pin, e, c, s, 3, cid, seed)
    q = (z1 * z1 + z2 * z2) + z3 * z3
    with np.errstate(divide="ignore", invalid="ignore"):
        t = np.where(q == 0, np.float32(0), z0 / np.sqrt(q))
    np.testing.assert_array_equal(h.ravel(), _f16(t))


def test_control_and_random_counters_against_rocrand(orc, philox_pin):
    """Scrambled stage j* of canary t: word 0 of (t, 0, 0, SCRAMBLE<<24|id)
    modulo the number of benign stages; random-baseline score of (t, s):
    (word 0 of (t, s, 0, RANDOM<<24|id) >> 8) 2^-24."""
    seed, cid, S, pos = 9, 3, 7, (1 << 2) | (1 << 5)
    benign = [j for j in range(S) if not (pos >> j) & 1]
    for t in range(50):
        w = _words(philox_pin, [t], 0, 0, 6, cid, seed)[0]
        assert orc.scramble_jstar(S, pos, seed, cid, t) == benign[int(w[0]) % len(benign)]
        for s in range(S):
            w = _words(philox_pin, [t], s, 0, 7, cid, seed)[0]
            assert orc.random_score(seed, cid, t, s) == np.float32((int(w[0]) >> 8) * 2.0**-24)


# ----------------------------------------------------------------------------
# live pass: exact special cases
# ----------------------------------------------------------------------------
def test_zero_noise_benign_is_fp16_of_reference(orc):
    a = _ref(orc)
    h = orc.sim_block(0, 0, a, seed=1, cfg_id=0, sigma_b=0.0)
    np.testing.assert_array_equal(h, _f16(a))
    h = orc.sim_block(0, 0, a, seed=1, cfg_id=0, benign_mode=NOISE_BLOCK, bscale=0.0)
    np.testing.assert_array_equal(h, _f16(a))


def test_full_sign_flip_is_negated_reference(orc):
    a = _ref(orc)
    h = orc.sim_block(0, 0, a, seed=1, cfg_id=0, sigma_b=0.0, malicious=True, tamper=T_FLIP,
                      flip_p=1.0)
    np.testing.assert_array_equal(h, _f16(-a))
    assert abs(_rel(h, a) - 2.0) < 1e-3  # tau(v) = -v gives m = 2


def test_power_of_two_rescale(orc):
    a = _ref(orc)
    h = orc.sim_block(0, 0, a, seed=1, cfg_id=0, sigma_b=0.0, malicious=True, tamper=T_SCALE,
                      scale=2.0)
    np.testing.assert_array_equal(h, _f16(2.0 * a))


def test_clean_base_ignores_benign_noise(orc):
    a = _ref(orc)
    h = orc.sim_block(0, 0, a, seed=1, cfg_id=0, sigma_b=0.5, malicious=True, tamper=T_SCALE,
                      scale=1.0, tamper_base=BASE_CLEAN)
    np.testing.assert_array_equal(h, _f16(a))
    # ... while a benign shard in the same call is noisy
    hb = orc.sim_block(0, 0, a, seed=1, cfg_id=0, sigma_b=0.5)
    assert not np.array_equal(hb, _f16(a))


def test_benign_shard_ignores_tamper_settings(orc):
    a = _ref(orc)
    kw = dict(seed=1, cfg_id=4, sigma_b=1e-3)
    h0 = orc.sim_block(0, 0, a, **kw)
    h1 = orc.sim_block(0, 0, a, malicious=False, tamper=T_ADD | T_FLIP | T_SCALE, tscale=5.0,
                       flip_p=1.0, scale=3.0, **kw)
    np.testing.assert_array_equal(h0, h1)


def test_noise_is_keyed_by_config_block_and_seed(orc):
    a = _ref(orc, T=8, H=64)
    base = orc.sim_block(0, 0, a, seed=1, cfg_id=0, sigma_b=1e-2)
    np.testing.assert_array_equal(base, orc.sim_block(0, 0, a, seed=1, cfg_id=0, sigma_b=1e-2))
    for kw in (dict(seed=2, cfg_id=0), dict(seed=1, cfg_id=1)):
        assert not np.array_equal(base, orc.sim_block(0, 0, a, sigma_b=1e-2, **kw))
    assert not np.array_equal(base, orc.sim_block(1, 0, a, seed=1, cfg_id=0, sigma_b=1e-2))
    assert not np.array_equal(base, orc.sim_block(0, 1, a, seed=1, cfg_id=0, sigma_b=1e-2))


# ----------------------------------------------------------------------------
# live pass: magnitudes fixed by Eqs. 2-4
# ----------------------------------------------------------------------------
def test_elementwise_benign_noise_scale(orc):
    """delta ~ N(0, (sigma |a|)^2): m^2 = sigma^2 E[a^2 z^2]/E[a^2] = sigma^2
    (plus the fp16 rounding floor, negligible at sigma = 1e-2)."""
    a = _ref(orc, T=256, H=512)
    h = orc.sim_block(0, 0, a, seed=1, cfg_id=0, sigma_b=1e-2)
    m = _rel(h, a)
    assert abs(m / 1e-2 - 1.0) < 0.01
    # the relative displacement has unit variance and no bias
    ok = np.abs(a) > 1.0  # fp16 rounding is small against the noise there
    r = (_h(h)[ok] - a[ok]) / (1e-2 * np.abs(a[ok].astype(np.float64)))
    assert abs(r.mean()) < 0.01 and abs(r.std() - 1.0) < 0.02


def test_block_benign_noise_scale(orc):
    """Eq. 2 proper: delta ~ N(0, sigma^2 mu^2), mu the mean |a| of the block,
    so m = sigma mu / rms(a) (about sigma sqrt(2/pi) for normal activations)."""
    a = _ref(orc, T=256, H=512)
    q, mu_sum = orc.ref_stats_block(a)
    n = a.size
    _, bs = orc.block_scales(256, 512, np.array([q]), np.array([mu_sum]), 0.0, 1e-2)
    assert bs[0] == np.float32(1e-2 * (mu_sum / n))
    h = orc.sim_block(0, 0, a, seed=1, cfg_id=0, benign_mode=NOISE_BLOCK, bscale=bs[0])
    m = _rel(h, a)
    rms = math.sqrt(q / n)
    assert abs(m / (1e-2 * (mu_sum / n) / rms) - 1.0) < 0.01
    assert abs((mu_sum / n) / rms - math.sqrt(2 / math.pi)) < 0.02
    # additive noise of constant scale: (h - a) / bscale has unit variance
    r = (_h(h) - a) / float(bs[0])
    assert abs(r.std() - 1.0) < 0.02


def test_student_t_noise(orc):
    """Heavy-tailed benign noise: unit-variance Student-t with 3 degrees of
    freedom.  Its median |t| and tail mass match the t(3) law / sqrt(3)."""
    T, H = 512, 512
    a = np.full((T, H), 1.0, np.float32)  # |a| = 1: the noise is read off directly
    h = orc.sim_block(0, 0, a, seed=2, cfg_id=0, benign_dist=DIST_T3, sigma_b=0.25)
    # fp16 spacing near 1 is 2^-10 (2^-11 just below 1): small against 0.25
    t = (_h(h) - 1.0) / 0.25 * math.sqrt(3.0)
    med = np.median(np.abs(t))
    assert abs(med - stats.t(3).ppf(0.75)) < 0.02
    tail = (np.abs(t) > stats.t(3).ppf(0.995)).mean()
    assert 0.007 < tail < 0.013
    # Gaussian noise on the same input has a much lighter tail
    hg = orc.sim_block(0, 0, a, seed=2, cfg_id=0, sigma_b=0.25)
    tg = (_h(hg) - 1.0) / 0.25 * math.sqrt(3.0)
    assert (np.abs(tg) > stats.t(3).ppf(0.995)).mean() < 0.002


def test_gaussian_tamper_magnitude(orc):
    """m = ||eps rms(a) z|| / ||a|| = eps (the paper: m ~ eps)."""
    a = _ref(orc, T=256, H=512)
    q, s = orc.ref_stats_block(a)
    ts, _ = orc.block_scales(256, 512, np.array([q]), np.array([s]), 0.05, 0.0)
    assert ts[0] == np.float32(0.05 * math.sqrt(q / a.size))
    h = orc.sim_block(0, 0, a, seed=1, cfg_id=0, sigma_b=0.0, malicious=True, tamper=T_ADD,
                      tscale=ts[0])
    assert abs(_rel(h, a) / 0.05 - 1.0) < 0.01
    # with benign noise underneath: m^2 = eps^2 + sigma^2
    h = orc.sim_block(0, 0, a, seed=1, cfg_id=0, sigma_b=0.02, malicious=True, tamper=T_ADD,
                      tscale=ts[0])
    assert abs(_rel(h, a) / math.sqrt(0.05**2 + 0.02**2) - 1.0) < 0.01


@pytest.mark.parametrize("p", [0.001, 0.01, 0.25])
def test_partial_sign_flip(orc, p):
    """Each element flips with probability p; m = 2 sqrt(p)."""
    a = _ref(orc, T=512, H=512)
    h = orc.sim_block(0, 0, a, seed=1, cfg_id=0, sigma_b=0.0, malicious=True, tamper=T_FLIP,
                      flip_p=p, tamper_base=BASE_CLEAN)
    flipped = ((h ^ _f16(a)) & 0x8000) != 0  # sign bit differs from fp16(a)
    n = a.size
    frac = flipped.mean()
    assert abs(frac - p) < 6 * math.sqrt(p * (1 - p) / n)
    # unflipped elements are exactly fp16(a), flipped ones exactly fp16(-a)
    np.testing.assert_array_equal(h[~flipped], _f16(a)[~flipped])
    np.testing.assert_array_equal(h[flipped], _f16(-a)[flipped])
    assert abs(_rel(h, a) / (2 * math.sqrt(p)) - 1.0) < 0.1


def test_flip_probability_zero(orc):
    a = _ref(orc)
    h = orc.sim_block(0, 0, a, seed=1, cfg_id=0, sigma_b=0.0, malicious=True, tamper=T_FLIP,
                      flip_p=0.0)
    np.testing.assert_array_equal(h, _f16(a))


def test_rescale_magnitude(orc):
    """tau(v) = (1 + alpha) v gives m = alpha (Section 4.4 rescale)."""
    a = _ref(orc, T=128, H=512)
    h = orc.sim_block(0, 0, a, seed=1, cfg_id=0, sigma_b=0.0, malicious=True, tamper=T_SCALE,
                      scale=1.10)
    assert abs(_rel(h, a) - 0.10) < 5e-4


def test_mixed_tamper_order(orc):
    """Mixed = Gaussian, then sign flip, then rescale.  A full flip after the
    Gaussian step gives exactly -(a + tscale z) (the other order would give
    -a + tscale z); a power-of-two rescale after both doubles that (exact in
    fp16 away from the subnormal range)."""
    a = _ref(orc)
    add_only = orc.sim_block(0, 0, a, seed=1, cfg_id=0, sigma_b=0.0, malicious=True,
                             tamper=T_ADD, tscale=0.1)
    flip_after = orc.sim_block(0, 0, a, seed=1, cfg_id=0, sigma_b=0.0, malicious=True,
                               tamper=T_ADD | T_FLIP | T_SCALE, tscale=0.1, flip_p=1.0,
                               scale=1.0)
    np.testing.assert_array_equal(flip_after, add_only ^ np.uint16(0x8000))
    mixed = orc.sim_block(0, 0, a, seed=1, cfg_id=0, sigma_b=0.0, malicious=True,
                          tamper=T_ADD | T_FLIP | T_SCALE, tscale=0.1, flip_p=1.0, scale=2.0)
    normal = np.abs(_h(add_only)) >= 2.0**-13
    assert normal.mean() > 0.99
    np.testing.assert_array_equal(_h(mixed)[normal], -2.0 * _h(add_only)[normal])


def test_canary_sim_array_layout(orc):
    S, C, T, H = 3, 2, 4, 16
    ref = orc.ref_synth(S, C, T, H, 9, 1, np.ones(H, np.float32))
    ts = np.full((S, C), 0.07, np.float32)
    h = orc.canary_sim(ref, seed=9, cfg_id=5, sigma_b=1e-3, mal_mask=0b010, tamper=T_ADD,
                       tscale=ts)
    for s in range(S):
        for c in range(C):
            want = orc.sim_block(s, c, ref[s, c], seed=9, cfg_id=5, sigma_b=1e-3,
                                 malicious=(s == 1), tamper=T_ADD, tscale=0.07)
            np.testing.assert_array_equal(h[s, c], want)


def test_block_scales_closed_form(orc):
    """A block of constant magnitude c has rms = mu = c."""
    T, H = 4, 8
    a = np.full(T * H, -3.0, np.float32)
    q, s = orc.ref_stats_block(a)
    assert q == 9.0 * T * H and s == 3.0 * T * H
    ts, bs = orc.block_scales(T, H, np.array([q]), np.array([s]), 0.5, 0.25)
    assert ts[0] == 1.5 and bs[0] == 0.75


# ----------------------------------------------------------------------------
# exact-norm Gaussian tamper (Section 3.2: v + eps ||v|| N / ||N||)
# ----------------------------------------------------------------------------
def test_exact_norm_tamper_has_norm_eps_times_v(orc):
    """On the clean base the added perturbation has norm eps ||a|| exactly
    (up to rounding), where the per-element form only matches it on average."""
    a = _ref(orc, T=16, H=256)  # a small block: per-element fluctuation is visible
    eps = 0.05
    ts, vv, zz = orc.tamper_scale_exact_block(0, 0, a, eps, seed=1, cfg_id=3, sigma_b=0.0,
                                              tamper_base=BASE_CLEAN)
    q, _ = orc.ref_stats_block(a)
    assert vv == q  # clean base: sum v^2 is sum a^2
    h = orc.sim_block(0, 0, a, seed=1, cfg_id=3, sigma_b=0.0, malicious=True, tamper=T_ADD,
                      tscale=ts, tamper_base=BASE_CLEAN)
    m = _rel(h, a)
    assert abs(m / eps - 1.0) < 2e-4
    # the per-element form at the same eps misses eps by the sampling error of ||N||
    ts_el, _ = orc.block_scales(16, 256, np.array([q]), np.array([0.0]), eps, 0.0)
    h_el = orc.sim_block(0, 0, a, seed=1, cfg_id=3, sigma_b=0.0, malicious=True, tamper=T_ADD,
                         tscale=ts_el[0], tamper_base=BASE_CLEAN)
    assert abs(_rel(h_el, a) / eps - 1.0) > 10 * abs(m / eps - 1.0)


def test_exact_norm_tamper_on_benign_output(orc):
    """On the benign base the perturbation is eps ||a + delta||: m^2 = eps^2
    ||v||^2 / ||a||^2 + sigma^2, with ||v|| = ||a|| (1 + O(sigma^2))."""
    a = _ref(orc, T=64, H=512)
    eps, sigma = 0.05, 0.01
    ts, vv, zz = orc.tamper_scale_exact_block(0, 0, a, eps, seed=2, cfg_id=1, sigma_b=sigma)
    q, _ = orc.ref_stats_block(a)
    assert abs(vv / q - 1.0) < 5 * sigma**2
    # sum v^2 is the norm of the benign output itself: at a large noise level
    # it differs from sum a^2 by ~sigma^2 and matches the stored fp16 output
    # to within fp16 rounding
    big = 0.3
    _, vv_big, _ = orc.tamper_scale_exact_block(0, 0, a, eps, seed=2, cfg_id=1, sigma_b=big)
    v16 = _h(orc.sim_block(0, 0, a, seed=2, cfg_id=1, sigma_b=big))
    assert abs(vv_big / (v16 * v16).sum() - 1.0) < 2.0**-10
    assert abs(vv_big / q - (1.0 + big**2)) < 0.02
    assert abs(zz / a.size - 1.0) < 0.05  # unit-variance normals
    h = orc.sim_block(0, 0, a, seed=2, cfg_id=1, sigma_b=sigma, malicious=True, tamper=T_ADD,
                      tscale=ts)
    assert abs(_rel(h, a) / math.sqrt(eps**2 + sigma**2) - 1.0) < 0.01


# ----------------------------------------------------------------------------
# propagation model (Eq. 2 with the live input h_{i-1}; Sections 5.3-5.5)
# ----------------------------------------------------------------------------
def _chain(orc, ref, carry, **kw):
    import ctypes
    ref = np.ascontiguousarray(ref, np.float32)
    S, C, T, H = ref.shape
    h = np.empty(ref.shape, np.uint16)
    args = dict(seed=4, cfg_id=2, benign_mode=0, benign_dist=0, sigma_b=0.0, mal_mask=0,
                tamper=0, tamper_base=0, flip_p=0.0, scale=1.0, redraw=0)
    args.update(kw)
    ts = args.pop("tscale", None)
    ts = None if ts is None else np.ascontiguousarray(ts, np.float32)
    bs = args.pop("bscale", None)
    bs = None if bs is None else np.ascontiguousarray(bs, np.float32)
    orc.lib().orc_canary_sim_chain(
        S, C, T, H, args["seed"], args["cfg_id"], args["benign_mode"], args["benign_dist"],
        args["sigma_b"], None if bs is None else bs.ctypes.data_as(ctypes.POINTER(ctypes.c_float)),
        args["mal_mask"], args["tamper"], args["tamper_base"],
        None if ts is None else ts.ctypes.data_as(ctypes.POINTER(ctypes.c_float)),
        args["flip_p"], args["scale"], args["redraw"], carry,
        ref.ctypes.data_as(ctypes.POINTER(ctypes.c_float)),
        h.ctypes.data_as(ctypes.POINTER(ctypes.c_uint16)))
    return h


def test_chain_without_carry_is_the_independent_pass(orc):
    ref = orc.ref_synth(5, 3, 8, 64, 4, 0, np.ones(64, np.float32))
    ts = np.full((5, 3), 0.05, np.float32)
    kw = dict(sigma_b=1e-2, mal_mask=1 << 2, tamper=1 | 2, tscale=ts, flip_p=0.1)
    want = orc.canary_sim(ref, seed=4, cfg_id=2, **kw)
    np.testing.assert_array_equal(_chain(orc, ref, 0.0, **kw), want)


def test_chain_benign_error_law(orc):
    """e_s = delta_s + g e_{s-1} with independent deltas: m_s^2 = sigma^2
    (1 + g^2 + ... + g^(2s))."""
    S, g, sigma = 6, 0.8, 1e-2
    ref = orc.ref_synth(S, 1, 128, 512, 5, 0, np.ones(512, np.float32))
    h = _chain(orc, ref, g, sigma_b=sigma)
    for s in range(S):
        m = _rel(h[s, 0], ref[s, 0])
        want = sigma * math.sqrt(sum(g ** (2 * j) for j in range(s + 1)))
        assert abs(m / want - 1.0) < 0.02, (s, m, want)


def test_chain_carry_has_the_sign_of_the_previous_error(orc):
    """With noise at stage 0 only, stage 1's live error is g times stage 0's
    (e_1 = delta_1 + g e_0 with delta_1 = 0), up to fp16 rounding: a
    regression of e_1 on e_0 has slope g, not -g."""
    S, g = 3, 0.6
    ref = orc.ref_synth(S, 1, 64, 512, 8, 0, np.ones(512, np.float32))
    bscale = np.zeros((S, 1), np.float32)
    bscale[0, 0] = 0.05
    h = _chain(orc, ref, g, benign_mode=1, bscale=bscale)
    e0 = _h(h[0, 0]) - ref[0, 0].astype(np.float64)
    e1 = _h(h[1, 0]) - ref[1, 0].astype(np.float64)
    slope = (e0 * e1).sum() / (e0 * e0).sum()
    assert abs(slope / g - 1.0) < 0.01, slope


def test_chain_carries_the_tamper_downstream(orc):
    """A Gaussian tamper eps at stage 2 reaches stage 2 + k scaled by g^k; with
    g = 1 and no noise it propagates undiminished (relative to equal-scale
    references)."""
    S, eps = 6, 0.05
    ref = orc.ref_synth(S, 1, 128, 512, 6, 0, np.ones(512, np.float32))
    q, _ = orc.ref_stats(ref)
    ts, _ = orc.block_scales(128, 512, q, q, eps, 0.0)
    for g in (0.5, 1.0):
        h = _chain(orc, ref, g, mal_mask=1 << 2, tamper=1, tscale=ts, tamper_base=1)
        for s in range(S):
            m = _rel(h[s, 0], ref[s, 0])
            want = 0.0 if s < 2 else eps * g ** (s - 2)
            assert abs(m - want) < 0.02 * eps + 3e-4, (g, s, m, want)


def test_chain_canary_base_picks_the_run_canaries(orc):
    """The propagation model on a slice of canaries with canary_base c0
    reproduces those canaries of the whole run; without the offset it repeats
    canary 0's noise instead."""
    S, C, T, H = 4, 5, 3, 16
    ref = orc.ref_synth(S, C, T, H, 11, 0, np.ones(H, np.float32))
    ts = np.full((S, C), 0.04, np.float32)
    kw = dict(seed=11, cfg_id=4, sigma_b=2e-2, mal_mask=1 << 2, tamper=3, flip_p=0.2,
              carry=0.7)
    whole = orc.canary_sim(ref, tscale=ts, **kw)
    part = orc.canary_sim(np.ascontiguousarray(ref[:, 2:4]), tscale=np.ascontiguousarray(ts[:, 2:4]),
                          canary_base=2, **kw)
    np.testing.assert_array_equal(part, whole[:, 2:4])
    unshifted = orc.canary_sim(np.ascontiguousarray(ref[:, 2:4]),
                               tscale=np.ascontiguousarray(ts[:, 2:4]), **kw)
    assert not np.array_equal(unshifted, whole[:, 2:4])


# ----------------------------------------------------------------------------
# exact-norm Gaussian tamper under the propagation model
# ----------------------------------------------------------------------------
def _tamper_normals_sumsq(orc, seed, cfg_id, s, c, n):
    """Sum of squares of the TAMPER_ADD normals of block (s, c), element by
    element from the Philox words (call e/2, words 0-1 even / 2-3 odd) and
    the Irwin-Hall rule, in fp64 in index order."""
    tot = 0.0
    key = np.array([seed & 0xFFFFFFFF, seed >> 32], np.uint32)
    for e in range(n):
        w = orc.philox(np.array([e >> 1, c, s, (4 << 24) | cfg_id], np.uint32), key)
        z = float(orc.z16(w[0], w[1]) if e % 2 == 0 else orc.z16(w[2], w[3]))
        tot += z * z
    return tot


def test_exact_norm_chain_first_stage_is_the_independent_form(orc):
    """An attacker at stage 0 has no upstream: its exact-norm scale under the
    propagation model equals the independent-stage one bit for bit."""
    S, C, T, H = 5, 3, 6, 64
    ref = orc.ref_synth(S, C, T, H, 9, 0, np.ones(H, np.float32))
    q, m = orc.ref_stats(ref)
    _, bs = orc.block_scales(T, H, q, m, 0.0, 0.01)
    kw = dict(seed=9, cfg_id=5, benign_mode=NOISE_BLOCK, sigma_b=0.01, bscale=bs)
    ts, nm = orc.tamper_scale_exact(ref, 0.05, carry=0.7, mal_mask=1, tamper=T_ADD, **kw)
    ts_i, nm_i = orc.tamper_scale_exact(ref, 0.05, **kw)
    np.testing.assert_array_equal(ts[0], ts_i[0])
    np.testing.assert_array_equal(nm[0], nm_i[0])
    assert (ts[1:] == 0).all() and (nm[1:] == 0).all()  # benign stages: no scale


def test_exact_norm_chain_uses_the_untampered_live_output(orc):
    """For an attacker at stage 3 of a carried pipeline, sum v^2 is the norm
    of the stage's own benign output given the live error carried in: the
    all-benign chain's stage-3 fp16 output reproduces it to fp16 rounding,
    while the reference block alone does not; sum N^2 is the TAMPER_ADD
    normals' of that block, recomputed from the Philox words."""
    S, C, T, H, g, m = 6, 2, 8, 64, 0.7, 3
    ref = orc.ref_synth(S, C, T, H, 4, 0, np.ones(H, np.float32))
    kw = dict(seed=4, cfg_id=2, sigma_b=0.05)
    ts, nm = orc.tamper_scale_exact(ref, 0.05, carry=g, mal_mask=1 << m, tamper=T_ADD, **kw)
    h = _chain(orc, ref, g, **kw)
    for c in range(C):
        v16 = _h(h[m, c])
        assert abs(nm[m, c, 0] / (v16 * v16).sum() - 1.0) < 2.0**-10
        a2 = (ref[m, c].astype(np.float64) ** 2).sum()
        assert abs(nm[m, c, 0] / a2 - 1.0) > 4 * 2.0**-10  # not the reference's norm
        assert nm[m, c, 1] == _tamper_normals_sumsq(orc, 4, 2, m, c, T * H)


def test_exact_norm_chain_colluders_in_pipeline_order(orc):
    """Two colluders at stages 1 and 3: the second one's v carries the
    first one's tamper (taken with its own exact scale; g^2 eps = 0.25 of
    the reference norm reaches stage 3), and each added perturbation has
    norm eps ||v|| (Section 3.2), measured as the change of the stage's fp16
    output when it tampers."""
    S, C, T, H, g, eps = 5, 2, 16, 128, 0.7, 0.5
    ref = orc.ref_synth(S, C, T, H, 6, 0, np.ones(H, np.float32))
    mal = (1 << 1) | (1 << 3)
    kw = dict(seed=6, cfg_id=3, sigma_b=0.01)
    ts, nm = orc.tamper_scale_exact(ref, eps, carry=g, mal_mask=mal, tamper=T_ADD, **kw)
    only1 = _chain(orc, ref, g, mal_mask=1 << 1, tamper=T_ADD, tscale=ts, **kw)
    benign = _chain(orc, ref, g, **kw)
    both = _chain(orc, ref, g, mal_mask=mal, tamper=T_ADD, tscale=ts, **kw)
    for c in range(C):
        v3 = _h(only1[3, c])  # stage 3 untampered, downstream of the tampered stage 1
        assert abs(nm[3, c, 0] / (v3 * v3).sum() - 1.0) < 2.0**-10
        w3 = _h(benign[3, c])
        assert abs(nm[3, c, 0] / (w3 * w3).sum() - 1.0) > 0.02
        for s, base in ((1, benign), (3, only1)):
            d = _h(both[s, c]) - _h(base[s, c])
            assert abs(math.sqrt((d * d).sum()) / (eps * math.sqrt(nm[s, c, 0])) - 1.0) < 2e-3
