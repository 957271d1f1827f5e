"""CPU oracle for the canary-versus-reference drift detector (numpy front end).

TEST INFRASTRUCTURE ONLY: the tests, the smoke check and the benchmark's
CPU-baseline leg may import this package; the product path never does.  It
imports nothing from the GPU package and the GPU package imports nothing
from it.

Every function wraps one routine of ``oracle.c`` (plain C, fp64), which
states the passage of the paper it follows:
  * ``drift_score``  -- Eq. 4, relative-L2 mismatch per (stage, canary);
  * ``auroc_config`` -- Eqs. 5-6 and the Mann-Whitney form, brute-force pair
    counts, plus the scrambled-label control of Section 4.5;
  * ``ref_synth`` / ``canary_sim`` -- the synthetic stand-ins for the fp32
    references of Eq. 1 and the live pass of Eqs. 2-3.
"""
import ctypes
import os

import numpy as np

from . import build as _build

_LIB = None

NOISE_ELEMENTWISE = 0
NOISE_BLOCK = 1
DIST_GAUSS = 0
DIST_T3 = 1
T_ADD = 1
T_FLIP = 2
T_SCALE = 4
BASE_BENIGN = 0
BASE_CLEAN = 1
AUROC_CONTROL = 1
AUROC_POOLED = 2
CTRL_INCLUDE_TRUE = 4
AUROC_RANDOM = 8

_u16p = ctypes.POINTER(ctypes.c_uint16)
_u32p = ctypes.POINTER(ctypes.c_uint32)
_u64p = ctypes.POINTER(ctypes.c_uint64)
_f32p = ctypes.POINTER(ctypes.c_float)
_f64p = ctypes.POINTER(ctypes.c_double)
_u32 = ctypes.c_uint32
_u64 = ctypes.c_uint64
_i = ctypes.c_int
_f = ctypes.c_float
_d = ctypes.c_double

_SIGS = {
    "orc_version": ([], _i),
    "orc_philox": ([_u32p, _u32p, _u32p], None),
    "orc_z16": ([_u32, _u32], _f),
    "orc_k16": ([], _f),
    "orc_f16_rne": ([_f], ctypes.c_uint16),
    "orc_f16_value": ([ctypes.c_uint16], _d),
    "orc_f16_rne_range": ([_u64, _u64, _u16p], None),
    "orc_f16_rne_array": ([_u64, _f32p, _u16p], None),
    "orc_outlier_gain": ([_u32, _u32, _f, _u64, _u32, _f32p], _i),
    "orc_ref_range": ([_u32, _u32, _u32, _u64, _u64, _u64, _u32, _f32p, _f32p], None),
    "orc_sim_range": ([_u32, _u32, _u64, _u64, _u64, _u32, _i, _i, _d, _f, _i, _u32, _i, _f,
                       _d, _d, _f32p, _u16p], _i),
    "orc_sim_range_ex": ([_u32, _u32, _u64, _u64, _u64, _u32, _i, _i, _d, _f, _i, _u32, _i, _f,
                          _d, _d, _i, _f32p, _u16p], _i),
    "orc_canary_sim_chain": ([_u32, _u32, _u32, _u32, _u64, _u32, _i, _i, _d, _f32p, _u64, _u32,
                              _i, _f32p, _d, _d, _i, _d, _f32p, _u16p], _i),
    "orc_canary_sim_chain_at": ([_u32, _u32, _u32, _u32, _u32, _u64, _u32, _i, _i, _d, _f32p,
                                 _u64, _u32, _i, _f32p, _d, _d, _i, _d, _f32p, _u16p], _i),
    "orc_tamper_scale_exact_block": ([_u32, _u32, _u32, _u32, _u64, _u32, _i, _i, _d, _f, _i, _i,
                                      _d, _f32p, _f64p, _f64p], _f),
    "orc_tamper_scale_exact_chain_at": ([_u32, _u32, _u32, _u32, _u32, _u64, _u32, _i, _i, _d,
                                         _f32p, _u64, _u32, _i, _d, _d, _i, _d, _d, _f32p, _f32p,
                                         _f64p], _i),
    "orc_drift_block_f16ref": ([_u64, _u16p, _u16p, _f64p, _f64p], _d),
    "orc_drift_score_f16ref": ([_u32, _u32, _u32, _u32, _u16p, _u16p, _f64p, _f32p], None),
    "orc_cosine_block": ([_u64, _u16p, _f32p], _d),
    "orc_cosine_block_f16ref": ([_u64, _u16p, _u16p], _d),
    "orc_cosine_score": ([_u32, _u32, _u32, _u32, _u16p, _f32p, _f64p, _f32p], None),
    "orc_random_score": ([_u64, _u32, _u32, _u32], _f),
    "orc_ref_block": ([_u32, _u32, _u32, _u32, _u64, _u32, _f32p, _f32p], None),
    "orc_ref_synth": ([_u32, _u32, _u32, _u32, _u64, _u32, _f32p, _f32p], None),
    "orc_ref_stats_block": ([_u64, _f32p, _f64p, _f64p], None),
    "orc_ref_stats": ([_u32, _u32, _u32, _u32, _f32p, _f64p, _f64p], None),
    "orc_block_scales": ([_u64, _u32, _u32, _f64p, _f64p, _d, _d, _f32p, _f32p], None),
    "orc_sim_block": ([_u32, _u32, _u32, _u32, _u64, _u32, _i, _i, _d, _f, _i, _u32, _i, _f,
                       _d, _d, _f32p, _u16p], _i),
    "orc_canary_sim": ([_u32, _u32, _u32, _u32, _u64, _u32, _i, _i, _d, _f32p, _u64, _u32, _i,
                        _f32p, _d, _d, _i, _f32p, _u16p], _i),
    "orc_drift_block": ([_u64, _u16p, _f32p, _f64p, _f64p], _d),
    "orc_drift_score": ([_u32, _u32, _u32, _u32, _u16p, _f32p, _f64p, _f32p, _f64p], None),
    "orc_score_cmp": ([_f, _f], _i),
    "orc_scramble_jstar": ([_u32, _u64, _u64, _u32, _u32], _i),
    "orc_auroc_config": ([_u32, _u32, _f32p, _u64, _u64, _u32, _u32, _u64p, _u64p, _u64p], _i),
    "orc_auroc_canaries": ([_u32, _u32, _f32p, _u64, _u64, _u32, _u32, _u32, _u32p], _i),
}


def lib():
    """Load liboracle.so, compiling it first if it has not been built.
    CDT_ORACLE_LIB names another build of oracle.c to load instead: the test
    that plants mistakes in copies of the oracle runs the pins against them."""
    global _LIB
    if _LIB is None:
        path = os.environ.get("CDT_ORACLE_LIB", _build.LIB)
        if path == _build.LIB and not os.path.exists(path):
            _build.build()
        L = ctypes.CDLL(path)
        for name, (args, res) in _SIGS.items():
            fn = getattr(L, name)
            fn.argtypes = args
            fn.restype = res
        _LIB = L
    return _LIB


def _p(a, ctype):
    return None if a is None else a.ctypes.data_as(ctypes.POINTER(ctype))


def _c(a, dtype):
    a = np.ascontiguousarray(a, dtype=dtype)
    return a


# ---------------------------------------------------------------------------
# primitives
# ---------------------------------------------------------------------------
def philox(ctr, key):
    """Philox4x32-10 of one 4-word counter and a 2-word key -> 4 uint32 words."""
    c = _c(ctr, np.uint32)
    k = _c(key, np.uint32)
    out = np.zeros(4, np.uint32)
    lib().orc_philox(_p(c, ctypes.c_uint32), _p(k, ctypes.c_uint32), _p(out, ctypes.c_uint32))
    return out


def z16(w0, w1):
    return np.float32(lib().orc_z16(int(w0), int(w1)))


def k16():
    return np.float32(lib().orc_k16())


def f16_rne(x):
    """fp32 array -> fp16 bit patterns (uint16), round to nearest even."""
    x = _c(x, np.float32)
    out = np.empty(x.shape, np.uint16)
    lib().orc_f16_rne_array(x.size, _p(x, ctypes.c_float), _p(out, ctypes.c_uint16))
    return out


def f16_rne_range(start, count):
    out = np.empty(count, np.uint16)
    lib().orc_f16_rne_range(start, count, _p(out, ctypes.c_uint16))
    return out


def f16_value(bits):
    return lib().orc_f16_value(int(bits))


# ---------------------------------------------------------------------------
# generator (stand-in for Eqs. 1-3)
# ---------------------------------------------------------------------------
def outlier_gain(H, n_out, big, seed, ref_set_id):
    g = np.empty(H, np.float32)
    rc = lib().orc_outlier_gain(H, n_out, big, seed, ref_set_id, _p(g, ctypes.c_float))
    if rc:
        raise ValueError(f"orc_outlier_gain failed ({rc})")
    return g


def ref_block(s, c, T, H, seed, ref_set_id, gain):
    gain = _c(gain, np.float32)
    out = np.empty(T * H, np.float32)
    lib().orc_ref_block(s, c, T, H, seed, ref_set_id, _p(gain, ctypes.c_float),
                        _p(out, ctypes.c_float))
    return out.reshape(T, H)


def ref_range(s, c, H, e0, count, seed, ref_set_id, gain):
    """Elements [e0, e0 + count) of reference block (s, c) (flat, e = t*H + j)."""
    gain = _c(gain, np.float32)
    out = np.empty(count, np.float32)
    lib().orc_ref_range(s, c, H, e0, count, seed, ref_set_id, _p(gain, ctypes.c_float),
                        _p(out, ctypes.c_float))
    return out


def ref_synth(S, C, T, H, seed, ref_set_id, gain):
    gain = _c(gain, np.float32)
    out = np.empty((S, C, T, H), np.float32)
    lib().orc_ref_synth(S, C, T, H, seed, ref_set_id, _p(gain, ctypes.c_float),
                        _p(out, ctypes.c_float))
    return out


def ref_stats(ref):
    """ref [S][C][T][H] -> (sumsq [S][C], sumabs [S][C]) in fp64."""
    ref = _c(ref, np.float32)
    S, C, T, H = ref.shape
    q = np.empty((S, C), np.float64)
    m = np.empty((S, C), np.float64)
    lib().orc_ref_stats(S, C, T, H, _p(ref, ctypes.c_float), _p(q, ctypes.c_double),
                        _p(m, ctypes.c_double))
    return q, m


def ref_stats_block(a):
    a = _c(a, np.float32)
    q = ctypes.c_double()
    m = ctypes.c_double()
    lib().orc_ref_stats_block(a.size, _p(a, ctypes.c_float), ctypes.byref(q), ctypes.byref(m))
    return q.value, m.value


def block_scales(T, H, sumsq, sumabs, eps, sigma_b):
    sumsq = _c(sumsq, np.float64)
    sumabs = _c(sumabs, np.float64)
    ts = np.empty(sumsq.shape, np.float32)
    bs = np.empty(sumsq.shape, np.float32)
    lib().orc_block_scales(sumsq.size, T, H, _p(sumsq, ctypes.c_double),
                           _p(sumabs, ctypes.c_double), eps, sigma_b,
                           _p(ts, ctypes.c_float), _p(bs, ctypes.c_float))
    return ts, bs


def sim_block(s, c, ref_block_arr, *, seed, cfg_id, benign_mode=NOISE_ELEMENTWISE,
              benign_dist=DIST_GAUSS, sigma_b=1e-3, bscale=0.0, malicious=False, tamper=0,
              tamper_base=BASE_BENIGN, tscale=0.0, flip_p=0.0, scale=1.0, redraw=False):
    a = _c(ref_block_arr, np.float32)
    T, H = a.shape
    h = np.empty((T, H), np.uint16)
    lib().orc_sim_range_ex(s, c, 0, T * H, seed, cfg_id, benign_mode, benign_dist, sigma_b,
                           float(bscale), int(bool(malicious)), tamper, tamper_base,
                           float(tscale), flip_p, scale, int(bool(redraw)),
                           _p(a, ctypes.c_float), _p(h, ctypes.c_uint16))
    return h


def sim_range(s, c, e0, ref_part, *, seed, cfg_id, benign_mode=NOISE_ELEMENTWISE,
              benign_dist=DIST_GAUSS, sigma_b=1e-3, bscale=0.0, malicious=False, tamper=0,
              tamper_base=BASE_BENIGN, tscale=0.0, flip_p=0.0, scale=1.0):
    """Live fp16 bits of elements [e0, e0 + len(ref_part)) of block (s, c)."""
    a = _c(ref_part, np.float32).ravel()
    h = np.empty(a.size, np.uint16)
    lib().orc_sim_range(s, c, e0, a.size, seed, cfg_id, benign_mode, benign_dist, sigma_b,
                        float(bscale), int(bool(malicious)), tamper, tamper_base, float(tscale),
                        flip_p, scale, _p(a, ctypes.c_float), _p(h, ctypes.c_uint16))
    return h


def tamper_scale_exact_block(s, c, ref_block_arr, eps, *, seed, cfg_id,
                             benign_mode=NOISE_ELEMENTWISE, benign_dist=DIST_GAUSS, sigma_b=1e-3,
                             bscale=0.0, tamper_base=BASE_BENIGN, redraw=False):
    """Exact-norm Gaussian tamper scale of one block: (tscale, sum v^2, sum N^2)."""
    a = _c(ref_block_arr, np.float32)
    T, H = a.shape
    vv = ctypes.c_double()
    zz = ctypes.c_double()
    ts = lib().orc_tamper_scale_exact_block(s, c, T, H, seed, cfg_id, benign_mode, benign_dist,
                                            sigma_b, float(bscale), tamper_base,
                                            int(bool(redraw)), eps, _p(a, ctypes.c_float),
                                            ctypes.byref(vv), ctypes.byref(zz))
    return np.float32(ts), vv.value, zz.value


def tamper_scale_exact(ref, eps, *, seed, cfg_id, benign_mode=NOISE_ELEMENTWISE,
                       benign_dist=DIST_GAUSS, sigma_b=1e-3, bscale=None,
                       tamper_base=BASE_BENIGN, redraw=False, carry=0.0, mal_mask=0, tamper=0,
                       flip_p=0.0, scale=1.0, canary_base=0):
    """[S][C] exact-norm tamper scales (and the [S][C][2] norms) of a whole array.
    carry > 0: the propagation model, malicious stages only (in pipeline
    order, each from its untampered output given everything upstream; the
    tamper settings apply to the earlier malicious stages); benign entries 0."""
    ref = _c(ref, np.float32)
    S, C = ref.shape[:2]
    if carry != 0.0:
        T, H = ref.shape[2:]
        bs = None if bscale is None else _c(bscale, np.float32)
        ts = np.empty((S, C), np.float32)
        norms = np.empty((S, C, 2), np.float64)
        lib().orc_tamper_scale_exact_chain_at(canary_base, S, C, T, H, seed, cfg_id, benign_mode,
                                              benign_dist, sigma_b, _p(bs, ctypes.c_float),
                                              mal_mask, tamper, tamper_base, flip_p, scale,
                                              int(bool(redraw)), carry, eps,
                                              _p(ref, ctypes.c_float), _p(ts, ctypes.c_float),
                                              _p(norms, ctypes.c_double))
        return ts, norms
    assert canary_base == 0, "canary_base is for the propagation model"
    ts = np.empty((S, C), np.float32)
    norms = np.empty((S, C, 2), np.float64)
    for s in range(S):
        for c in range(C):
            t, vv, zz = tamper_scale_exact_block(
                s, c, ref[s, c], eps, seed=seed, cfg_id=cfg_id, benign_mode=benign_mode,
                benign_dist=benign_dist, sigma_b=sigma_b,
                bscale=0.0 if bscale is None else bscale[s, c], tamper_base=tamper_base,
                redraw=redraw)
            ts[s, c] = t
            norms[s, c] = (vv, zz)
    return ts, norms


def canary_sim(ref, *, seed, cfg_id, benign_mode=NOISE_ELEMENTWISE, benign_dist=DIST_GAUSS,
               sigma_b=1e-3, bscale=None, mal_mask=0, tamper=0, tamper_base=BASE_BENIGN,
               tscale=None, flip_p=0.0, scale=1.0, redraw=False, carry=0.0, canary_base=0):
    """ref [S][C][T][H] fp32 -> h [S][C][T][H] fp16 bit patterns (uint16).
    carry > 0 runs the propagation model (stages in order per canary);
    canary_base: the run's index of the arrays' first canary (propagation
    model only)."""
    ref = _c(ref, np.float32)
    S, C, T, H = ref.shape
    bs = None if bscale is None else _c(bscale, np.float32)
    ts = None if tscale is None else _c(tscale, np.float32)
    h = np.empty((S, C, T, H), np.uint16)
    if carry != 0.0:
        lib().orc_canary_sim_chain_at(canary_base, S, C, T, H, seed, cfg_id, benign_mode,
                                      benign_dist, sigma_b, _p(bs, ctypes.c_float), mal_mask,
                                      tamper, tamper_base, _p(ts, ctypes.c_float), flip_p, scale,
                                      int(bool(redraw)), carry, _p(ref, ctypes.c_float),
                                      _p(h, ctypes.c_uint16))
        return h
    assert canary_base == 0, "canary_base is for the propagation model; use sim_block"
    lib().orc_canary_sim(S, C, T, H, seed, cfg_id, benign_mode, benign_dist, sigma_b,
                         _p(bs, ctypes.c_float), mal_mask, tamper, tamper_base,
                         _p(ts, ctypes.c_float), flip_p, scale, int(bool(redraw)),
                         _p(ref, ctypes.c_float), _p(h, ctypes.c_uint16))
    return h


# ---------------------------------------------------------------------------
# Eq. 4
# ---------------------------------------------------------------------------
def drift_block(h_bits, a):
    """One block: returns (m, D, R) in fp64."""
    h = _c(h_bits, np.uint16).ravel()
    a = _c(a, np.float32).ravel()
    assert h.size == a.size
    D = ctypes.c_double()
    R = ctypes.c_double()
    m = lib().orc_drift_block(h.size, _p(h, ctypes.c_uint16), _p(a, ctypes.c_float),
                              ctypes.byref(D), ctypes.byref(R))
    return m, D.value, R.value


def drift_score(h_bits, ref):
    """h [S][C][T][H] (fp16 bits), ref same shape fp32 ->
    (score64 [C][S], score32 [C][S], num_den [C][S][2])."""
    h = _c(h_bits, np.uint16)
    ref = _c(ref, np.float32)
    S, C, T, H = ref.shape
    assert h.shape == ref.shape
    s64 = np.empty((C, S), np.float64)
    s32 = np.empty((C, S), np.float32)
    nd = np.empty((C, S, 2), np.float64)
    lib().orc_drift_score(S, C, T, H, _p(h, ctypes.c_uint16), _p(ref, ctypes.c_float),
                          _p(s64, ctypes.c_double), _p(s32, ctypes.c_float),
                          _p(nd, ctypes.c_double))
    return s64, s32, nd


def drift_block_f16ref(h_bits, r_bits):
    """Eq. 4 against an fp16 reference (second live pass): (m, D, R)."""
    h = _c(h_bits, np.uint16).ravel()
    r = _c(r_bits, np.uint16).ravel()
    assert h.size == r.size
    D = ctypes.c_double()
    R = ctypes.c_double()
    m = lib().orc_drift_block_f16ref(h.size, _p(h, ctypes.c_uint16), _p(r, ctypes.c_uint16),
                                     ctypes.byref(D), ctypes.byref(R))
    return m, D.value, R.value


def drift_score_f16ref(h_bits, r_bits):
    """h, r [S][C][T][H] fp16 bits -> (score64 [C][S], score32 [C][S])."""
    h = _c(h_bits, np.uint16)
    r = _c(r_bits, np.uint16)
    S, C, T, H = h.shape
    assert r.shape == h.shape
    s64 = np.empty((C, S), np.float64)
    s32 = np.empty((C, S), np.float32)
    lib().orc_drift_score_f16ref(S, C, T, H, _p(h, ctypes.c_uint16), _p(r, ctypes.c_uint16),
                                 _p(s64, ctypes.c_double), _p(s32, ctypes.c_float))
    return s64, s32


def cosine_block(h_bits, a):
    """Cosine mismatch 1 - h.a / (|h| |a|) of one block (Section 4.4 ablation)."""
    h = _c(h_bits, np.uint16).ravel()
    a = _c(a, np.float32).ravel()
    assert h.size == a.size
    return lib().orc_cosine_block(h.size, _p(h, ctypes.c_uint16), _p(a, ctypes.c_float))


def cosine_block_f16ref(h_bits, r_bits):
    """Cosine mismatch against an fp16 reference (second live pass)."""
    h = _c(h_bits, np.uint16).ravel()
    r = _c(r_bits, np.uint16).ravel()
    assert h.size == r.size
    return lib().orc_cosine_block_f16ref(h.size, _p(h, ctypes.c_uint16), _p(r, ctypes.c_uint16))


def cosine_score_f16ref(h_bits, r_bits):
    """h, r [S][C][T][H] fp16 bits -> cosine mismatch [C][S] (fp64)."""
    h = _c(h_bits, np.uint16)
    r = _c(r_bits, np.uint16)
    S, C = h.shape[:2]
    out = np.empty((C, S), np.float64)
    for s in range(S):
        for c in range(C):
            out[c, s] = cosine_block_f16ref(h[s, c], r[s, c])
    return out


def cosine_score(h_bits, ref):
    h = _c(h_bits, np.uint16)
    ref = _c(ref, np.float32)
    S, C, T, H = ref.shape
    s64 = np.empty((C, S), np.float64)
    s32 = np.empty((C, S), np.float32)
    lib().orc_cosine_score(S, C, T, H, _p(h, ctypes.c_uint16), _p(ref, ctypes.c_float),
                           _p(s64, ctypes.c_double), _p(s32, ctypes.c_float))
    return s64, s32


# ---------------------------------------------------------------------------
# Eqs. 5-6
# ---------------------------------------------------------------------------
def score_cmp(x, y):
    return lib().orc_score_cmp(float(x), float(y))


def scramble_jstar(S, pos_mask, seed, cfg_id, t):
    return lib().orc_scramble_jstar(S, pos_mask, seed, cfg_id, t)


def auroc_config(scores, pos_mask, *, seed=0, cfg_id=0, flags=AUROC_CONTROL | AUROC_POOLED):
    """scores [C][S] fp32 -> (counts[6], pooled[3]) as uint64 arrays:
    counts = G, E, pairs, G_ctrl, E_ctrl, pairs_ctrl; pooled = G, E, pairs."""
    sc = _c(scores, np.float32)
    C, S = sc.shape
    counts = np.zeros(6, np.uint64)
    pooled = np.zeros(3, np.uint64)
    rc = lib().orc_auroc_config(S, C, _p(sc, ctypes.c_float), pos_mask, seed, cfg_id, flags,
                                _p(counts, ctypes.c_uint64), _p(pooled, ctypes.c_uint64), None)
    if rc:
        raise ValueError(f"orc_auroc_config failed ({rc})")
    return counts, pooled


def auroc_canaries(scores, pos_mask, *, seed=0, cfg_id=0, canary_base=0,
                   flags=AUROC_CONTROL | AUROC_RANDOM):
    """Eq. 5 per canary: scores [C][S] fp32 -> uint32 [C][6] = (G_t, E_t,
    control G_t, E_t, random-baseline G_t, E_t), draws keyed by canary_base + t."""
    sc = _c(scores, np.float32)
    C, S = sc.shape
    out = np.zeros((C, 6), np.uint32)
    rc = lib().orc_auroc_canaries(S, C, _p(sc, ctypes.c_float), pos_mask, seed, cfg_id,
                                  canary_base, flags, _p(out, ctypes.c_uint32))
    if rc:
        raise ValueError(f"orc_auroc_canaries failed ({rc})")
    return out


def random_score(seed, cfg_id, t, s):
    return np.float32(lib().orc_random_score(seed, cfg_id, t, s))


def random_baseline(C, S, pos_mask, *, seed=0, cfg_id=0):
    """Eq. 5 counts (G, E, pairs) with every score replaced by Uniform[0,1)
    (the random baseline of Section 4.5)."""
    counts = np.zeros(6, np.uint64)
    base = np.zeros(3, np.uint64)
    dummy = np.zeros((max(C, 1), max(S, 1)), np.float32)
    rc = lib().orc_auroc_config(S, C, _p(dummy, ctypes.c_float), pos_mask, seed, cfg_id,
                                AUROC_RANDOM, _p(counts, ctypes.c_uint64), None,
                                _p(base, ctypes.c_uint64))
    if rc:
        raise ValueError(f"orc_auroc_config failed ({rc})")
    return base


def auroc_strict(counts):
    """Eq. 6 as printed: ties count zero."""
    G, E, N = (int(x) for x in counts[:3])
    return G / N if N else float("nan")


def auroc_mw(counts):
    """Mann-Whitney normalisation: ties count one half."""
    G, E, N = (int(x) for x in counts[:3])
    return (G + 0.5 * E) / N if N else float("nan")
