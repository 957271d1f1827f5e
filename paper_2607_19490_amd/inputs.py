"""Seeded synthetic inputs shared by the tests, the smoke check and the bench.

Holds none of the detector's arithmetic: only numpy random draws of arrays
with the shapes and value ranges the detector sees (fp32 references, fp16
live activations near them, score tables with ties and NaNs).
"""
import numpy as np


def rng(seed):
    return np.random.default_rng(seed)


def ref_normal(shape, seed, outlier_frac=0.0, outlier_gain=20.0):
    """fp32 array ~ N(0, 1), with a random set of last-axis channels scaled."""
    g = rng(seed)
    a = g.standard_normal(shape, dtype=np.float32)
    if outlier_frac > 0:
        H = shape[-1]
        n = max(1, int(outlier_frac * H))
        ch = g.choice(H, size=n, replace=False)
        a[..., ch] *= np.float32(outlier_gain)
    return a


def live_near(ref, seed, rel=1e-3, flip_frac=0.0):
    """fp16 array near ref: ref * (1 + rel * N(0,1)), optional random sign flips.
    Returned as uint16 bit patterns (the way fp16 travels through the C ABI)."""
    g = rng(seed)
    x = ref.astype(np.float64) * (1.0 + rel * g.standard_normal(ref.shape))
    if flip_frac > 0:
        x = np.where(g.random(ref.shape) < flip_frac, -x, x)
    return x.astype(np.float16).view(np.uint16)


def fp16_bits(x):
    return np.asarray(x, np.float32).astype(np.float16).view(np.uint16)


def scores(C, S, seed, mal=(), gap=0.0, tie_levels=0, nan_frac=0.0):
    """[C][S] fp32 score table.  Malicious columns are shifted up by `gap`;
    tie_levels > 0 quantises every score to that many levels (forcing ties);
    nan_frac plants NaNs."""
    g = rng(seed)
    sc = g.random((C, S))
    if tie_levels:
        sc = np.floor(sc * tie_levels) / tie_levels
    for s in mal:
        sc[:, s] += gap
    sc = sc.astype(np.float32)
    if nan_frac > 0:
        sc[g.random((C, S)) < nan_frac] = np.nan
    return sc
