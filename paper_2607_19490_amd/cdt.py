"""Thin Python binding of libcdt (declared in include/cdt.h).

Argument marshalling only: every function checks the torch tensors it is
given (device, dtype, contiguity, shape), passes their device pointers and
the current HIP stream to the C ABI, and raises CdtError on a non-zero
return.  Every step of the method, Eq. 6's ratios included
(auroc_values), runs in the HIP kernels.  If libcdt.so has not been
built, loading fails loudly; there is no fallback path.

fp16 activations travel as torch.float16 tensors (their bits are the
uint16 words of the C ABI).
"""
import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libcdt.so")

OK, EINVAL, EALIGN, ELIMIT, EDEVICE = 0, 1, 2, 3, 4
NOISE_ELEMENTWISE, NOISE_BLOCK = 0, 1
DIST_GAUSS, DIST_T3 = 0, 1
T_ADD, T_FLIP, T_SCALE = 1, 2, 4
BASE_BENIGN, BASE_CLEAN = 0, 1
AUROC_CONTROL, AUROC_POOLED, CTRL_INCLUDE_TRUE, AUROC_RANDOM = 1, 2, 4, 8


class CdtError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"[{code}] {msg}")
        self.code = code


class SimParams(ctypes.Structure):
    _fields_ = [
        ("seed", ctypes.c_uint64),
        ("cfg_id", ctypes.c_uint32),
        ("benign_mode", ctypes.c_uint32),
        ("benign_dist", ctypes.c_uint32),
        ("tamper", ctypes.c_uint32),
        ("tamper_base", ctypes.c_uint32),
        ("redraw", ctypes.c_uint32),
        ("mal_mask", ctypes.c_uint64),
        ("sigma_b", ctypes.c_double),
        ("flip_p", ctypes.c_double),
        ("scale", ctypes.c_double),
        ("bscale", ctypes.c_void_p),
        ("tscale", ctypes.c_void_p),
        ("carry", ctypes.c_double),
        ("canary_base", ctypes.c_uint32),
        ("reserved", ctypes.c_uint32),
    ]


class AurocCfg(ctypes.Structure):
    _fields_ = [
        ("S", ctypes.c_uint32),
        ("C", ctypes.c_uint32),
        ("score_off", ctypes.c_uint64),
        ("pos_mask", ctypes.c_uint64),
        ("cfg_id", ctypes.c_uint32),
        ("canary_base", ctypes.c_uint32),
    ]


class DriftJob(ctypes.Structure):
    _fields_ = [
        ("S", ctypes.c_uint32),
        ("C", ctypes.c_uint32),
        ("T", ctypes.c_uint32),
        ("H", ctypes.c_uint32),
        ("h", ctypes.c_void_p),
        ("ref", ctypes.c_void_p),
        ("score", ctypes.c_void_p),
        ("num_den", ctypes.c_void_p),
    ]


class SimJob(ctypes.Structure):
    _fields_ = [
        ("S", ctypes.c_uint32),
        ("C", ctypes.c_uint32),
        ("T", ctypes.c_uint32),
        ("H", ctypes.c_uint32),
        ("p", ctypes.POINTER(SimParams)),
        ("ref", ctypes.c_void_p),
        ("h", ctypes.c_void_p),
    ]


_u32, _u64, _f, _d, _vp, _sz = (ctypes.c_uint32, ctypes.c_uint64, ctypes.c_float, ctypes.c_double,
                                ctypes.c_void_p, ctypes.c_size_t)
_SIGS = {
    "cdt_version": ([], ctypes.c_int),
    "cdt_last_error": ([], ctypes.c_char_p),
    "cdt_outlier_gain": ([_u32, _u32, _f, _u64, _u32, _vp, _vp], ctypes.c_int),
    "cdt_ref_synth": ([_u32, _u32, _u32, _u32, _u64, _u32, _u32, _vp, _vp, _vp], ctypes.c_int),
    "cdt_reduce_workspace_bytes": ([_u32, _u32, _u32, _u32], _sz),
    "cdt_ref_stats": ([_u32, _u32, _u32, _u32, _vp, _vp, _vp, _vp, _sz, _vp], ctypes.c_int),
    "cdt_block_scales": ([_u64, _u32, _u32, _vp, _vp, _d, _d, _vp, _vp, _vp], ctypes.c_int),
    "cdt_canary_sim": ([_u32, _u32, _u32, _u32, ctypes.POINTER(SimParams), _vp, _vp, _vp],
                       ctypes.c_int),
    "cdt_canary_sim_stream": ([_u32, _u32, _u32, _u32, _vp, _vp, _vp], ctypes.c_int),
    "cdt_sim_batch_workspace_bytes": ([_u32], _sz),
    "cdt_canary_sim_batch": ([_u32, ctypes.POINTER(SimJob), _vp, _sz, _vp], ctypes.c_int),
    "cdt_drift_batch_workspace_bytes": ([_u32, ctypes.POINTER(DriftJob)], _sz),
    "cdt_drift_score_batch": ([_u32, ctypes.POINTER(DriftJob), _vp, _sz, _vp], ctypes.c_int),
    "cdt_tamper_scale_exact": ([_u32, _u32, _u32, _u32, ctypes.POINTER(SimParams), _vp, _d, _vp,
                                _vp, _vp, _sz, _vp], ctypes.c_int),
    "cdt_sim_score": ([_u32, _u32, _u32, _u32, ctypes.POINTER(SimParams), _vp, _vp, _vp, _vp, _vp,
                       _sz, _vp], ctypes.c_int),
    "cdt_drift_score": ([_u32, _u32, _u32, _u32, _vp, _vp, _vp, _vp, _vp, _sz, _vp], ctypes.c_int),
    "cdt_drift_score_noalloc": ([_u32, _u32, _u32, _u32, _vp, _vp, _vp, _vp, _vp], ctypes.c_int),
    "cdt_drift_read_stream": ([_u32, _u32, _u32, _u32, _vp, _vp, _vp, _sz, _vp], ctypes.c_int),
    "cdt_drift_score_f16ref": ([_u32, _u32, _u32, _u32, _vp, _vp, _vp, _vp, _vp, _sz, _vp],
                               ctypes.c_int),
    "cdt_cosine_score": ([_u32, _u32, _u32, _u32, _vp, _vp, _vp, _vp, _vp, _sz, _vp], ctypes.c_int),
    "cdt_cosine_score_f16ref": ([_u32, _u32, _u32, _u32, _vp, _vp, _vp, _vp, _vp, _sz, _vp],
                                ctypes.c_int),
    "cdt_auroc_workspace_bytes": ([_u32], _sz),
    "cdt_auroc": ([_u32, ctypes.POINTER(AurocCfg), _vp, _u64, _u64, _u32, _vp, _vp, _vp, _vp, _sz,
                   _vp], ctypes.c_int),
    "cdt_auroc_upload": ([_u32, ctypes.POINTER(AurocCfg), _u64, _u32, _vp, _sz, _vp], ctypes.c_int),
    "cdt_auroc_launch": ([_u32, _vp, _vp, _u64, _u64, _u32, _vp, _vp, _vp, _vp], ctypes.c_int),
    "cdt_auroc_values": ([_u32, _vp, _vp, _vp, _vp, _vp], ctypes.c_int),
    "cdt_drift_read_stream_batch": ([_u32, ctypes.POINTER(DriftJob), _vp, _sz, _vp],
                                    ctypes.c_int),
    "cdt_auroc_canaries_workspace_bytes": ([_u32], _sz),
    "cdt_auroc_canaries": ([_u32, ctypes.POINTER(AurocCfg), _vp, _u64, _u64, _u32, _vp, _vp, _sz,
                            _vp], ctypes.c_int),
}

_LIB = None


# Interface version of include/cdt.h that the structures and signatures
# below mirror (cdt_version()).
ABI_VERSION = 11


def lib():
    """Load libcdt.so (built by paper_2607_19490_amd.build); raises if absent."""
    global _LIB
    if _LIB is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"libcdt.so is not built ({LIB_PATH}); run __graft_entry__.build()")
        L = ctypes.CDLL(LIB_PATH)
        L.cdt_version.argtypes, L.cdt_version.restype = [], ctypes.c_int
        if L.cdt_version() != ABI_VERSION:  # before binding entry points it may lack
            raise RuntimeError(f"libcdt.so has interface version {L.cdt_version()}, this binding "
                               f"expects {ABI_VERSION}; rebuild with __graft_entry__.build()")
        for name, (args, res) in _SIGS.items():
            fn = getattr(L, name)
            fn.argtypes = args
            fn.restype = res
        _LIB = L
    return _LIB


def exported_symbols():
    return list(_SIGS)


def _check(rc):
    if rc != OK:
        raise CdtError(rc, lib().cdt_last_error().decode())


def _torch():
    import torch
    return torch


def _stream():
    torch = _torch()
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _need(t, name, dtype, shape=None):
    torch = _torch()
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch tensor")
    if not t.is_cuda:
        raise ValueError(f"{name} must live on the GPU")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")


def _empty(shape, dtype, like=None):
    torch = _torch()
    dev = like.device if like is not None else torch.device("cuda", torch.cuda.current_device())
    return torch.empty(shape, dtype=dtype, device=dev)


def version():
    return lib().cdt_version()


def last_error():
    return lib().cdt_last_error().decode()


# ---------------------------------------------------------------------------
def outlier_gain(H, n_out, big, seed, ref_set_id, out=None):
    torch = _torch()
    out = _empty((H,), torch.float32) if out is None else out
    _need(out, "gain", torch.float32, (H,))
    _check(lib().cdt_outlier_gain(H, n_out, big, seed, ref_set_id, _ptr(out), _stream()))
    return out


def ref_synth(S, C, T, H, seed, ref_set_id, gain, out=None, canary_base=0):
    """References [S][C][T][H] fp32 of canaries canary_base .. canary_base + C - 1."""
    torch = _torch()
    _need(gain, "gain", torch.float32, (H,))
    out = _empty((S, C, T, H), torch.float32, gain) if out is None else out
    _need(out, "ref", torch.float32, (S, C, T, H))
    _check(lib().cdt_ref_synth(S, C, T, H, seed, ref_set_id, canary_base, _ptr(gain), _ptr(out),
                               _stream()))
    return out


def reduce_workspace_bytes(S, C, T, H):
    return lib().cdt_reduce_workspace_bytes(S, C, T, H)


def workspace(S, C, T, H, like=None):
    torch = _torch()
    n = max(16, reduce_workspace_bytes(S, C, T, H))
    return _empty((n,), torch.uint8, like)


def _ws_arg(ws, S, C, T, H, like):
    if ws is None:
        ws = workspace(S, C, T, H, like)
    _need(ws, "ws", ws.dtype)
    return ws, ctypes.c_size_t(ws.numel() * ws.element_size())


def ref_stats(ref, ws=None):
    torch = _torch()
    _need(ref, "ref", torch.float32)
    S, C, T, H = ref.shape
    sumsq = _empty((S, C), torch.float64, ref)
    sumabs = _empty((S, C), torch.float64, ref)
    ws, nbytes = _ws_arg(ws, S, C, T, H, ref)
    _check(lib().cdt_ref_stats(S, C, T, H, _ptr(ref), _ptr(sumsq), _ptr(sumabs), _ptr(ws), nbytes,
                               _stream()))
    return sumsq, sumabs


def block_scales(sumsq, sumabs, T, H, eps, sigma_b, tscale=None, bscale=None):
    torch = _torch()
    _need(sumsq, "sumsq", torch.float64)
    _need(sumabs, "sumabs", torch.float64, tuple(sumsq.shape))
    tscale = _empty(tuple(sumsq.shape), torch.float32, sumsq) if tscale is None else tscale
    bscale = _empty(tuple(sumsq.shape), torch.float32, sumsq) if bscale is None else bscale
    _need(tscale, "tscale", torch.float32, tuple(sumsq.shape))
    _need(bscale, "bscale", torch.float32, tuple(sumsq.shape))
    _check(lib().cdt_block_scales(sumsq.numel(), T, H, _ptr(sumsq), _ptr(sumabs), eps, sigma_b,
                                  _ptr(tscale), _ptr(bscale), _stream()))
    return tscale, bscale


def sim_params(*, seed, cfg_id, benign_mode=NOISE_ELEMENTWISE, benign_dist=DIST_GAUSS,
               sigma_b=1e-3, mal_mask=0, tamper=0, tamper_base=BASE_BENIGN, flip_p=0.0,
               scale=1.0, bscale=None, tscale=None, redraw=False, carry=0.0, canary_base=0):
    return SimParams(seed, cfg_id, benign_mode, benign_dist, tamper, tamper_base, int(redraw),
                     mal_mask, sigma_b, flip_p, scale,
                     None if bscale is None else bscale.data_ptr(),
                     None if tscale is None else tscale.data_ptr(), carry, canary_base, 0)


def canary_sim(ref, out=None, *, bscale=None, tscale=None, **kw):
    """ref [S][C][T][H] fp32 -> h [S][C][T][H] fp16.  Keywords as sim_params."""
    torch = _torch()
    _need(ref, "ref", torch.float32)
    S, C, T, H = ref.shape
    for name, t in (("bscale", bscale), ("tscale", tscale)):
        if t is not None:
            _need(t, name, torch.float32, (S, C))
    out = _empty((S, C, T, H), torch.float16, ref) if out is None else out
    _need(out, "h", torch.float16, (S, C, T, H))
    p = sim_params(bscale=bscale, tscale=tscale, **kw)
    _check(lib().cdt_canary_sim(S, C, T, H, ctypes.byref(p), _ptr(ref), _ptr(out), _stream()))
    return out


class Batch:
    """A checked ctypes job table (with the tensors and parameter structs it
    points to kept alive) and its device workspace: built once, launched as
    often as needed (the tensors' contents may change between launches,
    not their shapes or storage)."""

    def __init__(self, arr, n, keep, ws):
        self.arr, self.n, self.keep, self.ws = arr, n, keep, ws


def sim_batch(jobs):
    """Prepare a batched live pass.  jobs: list of (ref [S][C][T][H] fp32,
    h [S][C][T][H] fp16 output, keywords as sim_params including bscale /
    tscale tensors).  Every job must use the same benign noise distribution
    and mode, carry 0 (checked by the library when launched).  Jobs in a row
    over one reference tensor share its reads (cdt_canary_sim_batch)."""
    torch = _torch()
    n = len(jobs)
    arr = (SimJob * max(1, n))()
    keep = []
    for i, (ref, h, kw) in enumerate(jobs):
        _need(ref, "ref", torch.float32)
        S, C, T, H = ref.shape
        _need(h, "h", torch.float16, (S, C, T, H))
        kw = dict(kw)
        for name in ("bscale", "tscale"):
            if kw.get(name) is not None:
                _need(kw[name], name, torch.float32, (S, C))
        p = sim_params(**kw)
        keep.append((p, ref, h, kw.get("bscale"), kw.get("tscale")))
        arr[i] = SimJob(S, C, T, H, ctypes.pointer(p), ref.data_ptr(), h.data_ptr())
    nbytes = max(16, lib().cdt_sim_batch_workspace_bytes(n))
    ws = _empty((nbytes,), torch.uint8, jobs[0][0] if n else None)
    return Batch(arr, n, keep, ws)


def canary_sim_batch(jobs):
    """The live pass of several runs in one launch (cdt_canary_sim_batch):
    jobs is a Batch from sim_batch or its list of jobs."""
    b = jobs if isinstance(jobs, Batch) else sim_batch(jobs)
    _check(lib().cdt_canary_sim_batch(b.n, b.arr, _ptr(b.ws), b.ws.numel(), _stream()))


def drift_batch(jobs):
    """Prepare a batched Eq. 4.  jobs: list of (h fp16, ref fp32, score out
    [C][S] fp32, num_den out [C][S][2] fp64 or None).  Jobs in a row over
    one reference tensor share its reads (cdt_drift_score_batch)."""
    torch = _torch()
    n = len(jobs)
    arr = (DriftJob * max(1, n))()
    keep = []
    for i, (h, ref, score, nd) in enumerate(jobs):
        _need(h, "h", torch.float16)
        S, C, T, H = h.shape
        _need(ref, "ref", torch.float32, (S, C, T, H))
        _need(score, "score", torch.float32, (C, S))
        if nd is not None:
            _need(nd, "num_den", torch.float64, (C, S, 2))
        keep.append((h, ref, score, nd))
        arr[i] = DriftJob(S, C, T, H, h.data_ptr(), ref.data_ptr(), score.data_ptr(),
                          None if nd is None else nd.data_ptr())
    nbytes = max(16, lib().cdt_drift_batch_workspace_bytes(n, arr))
    ws = _empty((nbytes,), torch.uint8, jobs[0][0] if n else None)
    return Batch(arr, n, keep, ws)


def drift_score_batch(jobs):
    """Eq. 4 over several arrays in one launch (cdt_drift_score_batch): jobs
    is a Batch from drift_batch or its list of jobs; every job's scores are
    bitwise those of drift_score on it."""
    b = jobs if isinstance(jobs, Batch) else drift_batch(jobs)
    _check(lib().cdt_drift_score_batch(b.n, b.arr, _ptr(b.ws), b.ws.numel(), _stream()))


def drift_read_stream_batch(jobs):
    """The batched Eq. 4's loads with no arithmetic (a measurement of that
    launch's memory bound): jobs is a Batch from drift_batch (or its list of
    jobs); nothing is written."""
    b = jobs if isinstance(jobs, Batch) else drift_batch(jobs)
    _check(lib().cdt_drift_read_stream_batch(b.n, b.arr, _ptr(b.ws), b.ws.numel(), _stream()))


def canary_sim_stream(ref, out=None):
    """The live pass's reads and writes with h = fp16(ref) and no random
    numbers (a measurement of the memory bound of canary_sim's access
    pattern); returns h."""
    torch = _torch()
    _need(ref, "ref", torch.float32)
    S, C, T, H = ref.shape
    out = _empty((S, C, T, H), torch.float16, ref) if out is None else out
    _need(out, "h", torch.float16, (S, C, T, H))
    _check(lib().cdt_canary_sim_stream(S, C, T, H, _ptr(ref), _ptr(out), _stream()))
    return out


def tamper_scale_exact(ref, eps, norms=None, ws=None, *, bscale=None, **kw):
    """Per-block scale [S][C] fp32 of the exact-norm Gaussian tamper
    (eps ||v|| N / ||N||) for the run described by the keywords (as
    sim_params); norms (optional, [S][C][2] fp64) receives sum v^2, sum N^2."""
    torch = _torch()
    _need(ref, "ref", torch.float32)
    S, C, T, H = ref.shape
    if bscale is not None:
        _need(bscale, "bscale", torch.float32, (S, C))
    if norms is not None:
        _need(norms, "norms", torch.float64, (S, C, 2))
    out = _empty((S, C), torch.float32, ref)
    ws, nbytes = _ws_arg(ws, S, C, T, H, ref)
    p = sim_params(bscale=bscale, **kw)
    _check(lib().cdt_tamper_scale_exact(S, C, T, H, ctypes.byref(p), _ptr(ref), eps, _ptr(out),
                                        _ptr(norms), _ptr(ws), nbytes, _stream()))
    return out


def sim_score(ref, h=None, out=None, num_den=None, ws=None, *, bscale=None, tscale=None, **kw):
    """Live pass and Eq. 4 in one launch: ref [S][C][T][H] fp32 -> scores
    [C][S] fp32, bitwise those of canary_sim then drift_score.  h (fp16,
    optional) also receives the live activations.  Keywords as sim_params."""
    torch = _torch()
    _need(ref, "ref", torch.float32)
    S, C, T, H = ref.shape
    for name, t in (("bscale", bscale), ("tscale", tscale)):
        if t is not None:
            _need(t, name, torch.float32, (S, C))
    if h is not None:
        _need(h, "h", torch.float16, (S, C, T, H))
    out = _empty((C, S), torch.float32, ref) if out is None else out
    _need(out, "score", torch.float32, (C, S))
    if num_den is not None:
        _need(num_den, "num_den", torch.float64, (C, S, 2))
    ws, nbytes = _ws_arg(ws, S, C, T, H, ref)
    p = sim_params(bscale=bscale, tscale=tscale, **kw)
    _check(lib().cdt_sim_score(S, C, T, H, ctypes.byref(p), _ptr(ref), _ptr(h), _ptr(out),
                               _ptr(num_den), _ptr(ws), nbytes, _stream()))
    return out


def _drift(fn, h, ref, ref_dtype, out, sums, nsums, ws):
    torch = _torch()
    _need(h, "h", torch.float16)
    S, C, T, H = h.shape
    _need(ref, "ref", ref_dtype, (S, C, T, H))
    out = _empty((C, S), torch.float32, h) if out is None else out
    _need(out, "score", torch.float32, (C, S))
    if sums is not None:
        _need(sums, "sums", torch.float64, (C, S, nsums))
    ws, nbytes = _ws_arg(ws, S, C, T, H, h)
    _check(fn(S, C, T, H, _ptr(h), _ptr(ref), _ptr(out), _ptr(sums), _ptr(ws), nbytes,
              _stream()))
    return out


def drift_score(h, ref, out=None, num_den=None, ws=None):
    """Eq. 4 per block -> scores [C][S] fp32 (and optional [C][S][2] fp64)."""
    return _drift(lib().cdt_drift_score, h, ref, _torch().float32, out, num_den, 2, ws)


NOALLOC_SCRATCH_BYTES = 8388608  # CDT_NOALLOC_SCRATCH_BYTES


def drift_score_noalloc(h, ref, out=None, num_den=None):
    """Eq. 4 through cdt_drift_score_noalloc: no workspace; the library's
    own fixed scratch holds the partial sums (shapes up to its limit).  The
    outputs must be passed in (out [C][S] fp32, optional num_den [C][S][2]
    fp64) so that the call allocates nothing."""
    torch = _torch()
    _need(h, "h", torch.float16)
    S, C, T, H = h.shape
    _need(ref, "ref", torch.float32, (S, C, T, H))
    _need(out, "score", torch.float32, (C, S))
    if num_den is not None:
        _need(num_den, "num_den", torch.float64, (C, S, 2))
    _check(lib().cdt_drift_score_noalloc(S, C, T, H, _ptr(h), _ptr(ref), _ptr(out), _ptr(num_den),
                                         _stream()))
    return out


def drift_read_stream(h, ref, ws=None):
    """drift_score's reads of h and ref with no arithmetic (a measurement of
    the memory bound of Eq. 4's access pattern); returns nothing."""
    torch = _torch()
    _need(h, "h", torch.float16)
    S, C, T, H = h.shape
    _need(ref, "ref", torch.float32, (S, C, T, H))
    ws, nbytes = _ws_arg(ws, S, C, T, H, h)
    _check(lib().cdt_drift_read_stream(S, C, T, H, _ptr(h), _ptr(ref), _ptr(ws), nbytes,
                                       _stream()))


def drift_score_f16ref(h, r, out=None, num_den=None, ws=None):
    """Eq. 4 against an fp16 reference (a second live pass) -> [C][S] fp32."""
    return _drift(lib().cdt_drift_score_f16ref, h, r, _torch().float16, out, num_den, 2, ws)


def cosine_score(h, ref, out=None, sums=None, ws=None):
    """Cosine mismatch 1 - cos(h, a) per block -> [C][S] fp32 (sums: [C][S][3])."""
    return _drift(lib().cdt_cosine_score, h, ref, _torch().float32, out, sums, 3, ws)


def cosine_score_f16ref(h, r, out=None, sums=None, ws=None):
    """Cosine mismatch against an fp16 reference (a second live pass)."""
    return _drift(lib().cdt_cosine_score_f16ref, h, r, _torch().float16, out, sums, 3, ws)


def auroc_cfg_array(cfgs):
    """cfgs: iterable of (S, C, score_off, pos_mask, cfg_id[, canary_base])
    -> ctypes array."""
    cfgs = list(cfgs)
    arr = (AurocCfg * max(1, len(cfgs)))()
    for i, cfg in enumerate(cfgs):
        S, C, off, mask, cid = cfg[:5]
        arr[i] = AurocCfg(S, C, off, mask, cid, cfg[5] if len(cfg) > 5 else 0)
    return arr, len(cfgs)


def auroc(cfgs, scores, *, seed=0, flags=AUROC_CONTROL | AUROC_POOLED, counts=None, pooled=None,
          baseline=None, ws=None):
    """Batched AUROC counts.  cfgs: iterable of (S, C, score_off, pos_mask,
    cfg_id[, canary_base]); scores: flat (or any contiguous) fp32 device tensor.
    Returns (counts [n][6], pooled [n][3] or None, baseline [n][3] or None),
    uint64 counts held in int64 tensors."""
    torch = _torch()
    _need(scores, "scores", torch.float32)
    arr, n = auroc_cfg_array(cfgs)
    counts = _empty((n, 6), torch.int64, scores) if counts is None else counts
    _need(counts, "counts", torch.int64, (n, 6))
    if flags & AUROC_POOLED:
        pooled = _empty((n, 3), torch.int64, scores) if pooled is None else pooled
        _need(pooled, "pooled", torch.int64, (n, 3))
    if flags & AUROC_RANDOM:
        baseline = _empty((n, 3), torch.int64, scores) if baseline is None else baseline
        _need(baseline, "baseline", torch.int64, (n, 3))
    if ws is None:
        ws = _empty((max(16, lib().cdt_auroc_workspace_bytes(n)),), torch.uint8, scores)
    _need(ws, "ws", torch.uint8)
    _check(lib().cdt_auroc(n, arr, _ptr(scores), scores.numel(), seed, flags, _ptr(counts),
                           _ptr(pooled), _ptr(baseline), _ptr(ws), ws.numel(), _stream()))
    return (counts, pooled if flags & AUROC_POOLED else None,
            baseline if flags & AUROC_RANDOM else None)


def auroc_upload(cfgs, n_scores, *, flags=AUROC_CONTROL | AUROC_POOLED, table=None, like=None):
    """Validate a configuration table (as auroc does) against n_scores scores
    and copy it to the device.  Returns (table, n_cfg) for auroc_launch."""
    torch = _torch()
    arr, n = auroc_cfg_array(cfgs)
    nbytes = max(16, lib().cdt_auroc_workspace_bytes(n))
    table = _empty((nbytes,), torch.uint8, like) if table is None else table
    _need(table, "table", torch.uint8)
    _check(lib().cdt_auroc_upload(n, arr, n_scores, flags, _ptr(table), table.numel(), _stream()))
    return table, n


def auroc_launch(table, n_cfg, scores, *, seed=0, flags=AUROC_CONTROL | AUROC_POOLED,
                 counts=None, pooled=None, baseline=None):
    """Score `scores` against an uploaded table: kernel launches only, so it
    can be recorded by a stream capture.  Returns what auroc returns."""
    torch = _torch()
    _need(scores, "scores", torch.float32)
    _need(table, "table", torch.uint8)
    counts = _empty((n_cfg, 6), torch.int64, scores) if counts is None else counts
    _need(counts, "counts", torch.int64, (n_cfg, 6))
    if flags & AUROC_POOLED:
        pooled = _empty((n_cfg, 3), torch.int64, scores) if pooled is None else pooled
        _need(pooled, "pooled", torch.int64, (n_cfg, 3))
    if flags & AUROC_RANDOM:
        baseline = _empty((n_cfg, 3), torch.int64, scores) if baseline is None else baseline
        _need(baseline, "baseline", torch.int64, (n_cfg, 3))
    _check(lib().cdt_auroc_launch(n_cfg, _ptr(table), _ptr(scores), scores.numel(), seed, flags,
                                  _ptr(counts), _ptr(pooled), _ptr(baseline), _stream()))
    return (counts, pooled if flags & AUROC_POOLED else None,
            baseline if flags & AUROC_RANDOM else None)


def auroc_canaries(cfgs, scores, *, seed=0, flags=AUROC_CONTROL | AUROC_RANDOM, out=None,
                   ws=None):
    """Eq. 5 per canary (cdt_auroc_canaries).  cfgs as for auroc; returns
    int32 [sum of C][6] holding the uint32 counts (G_t, E_t of the detector,
    the control and the random baseline), configurations in order."""
    torch = _torch()
    _need(scores, "scores", torch.float32)
    arr, n = auroc_cfg_array(cfgs)
    total = sum(int(c[1]) for c in cfgs)
    out = _empty((max(total, 1), 6), torch.int32, scores) if out is None else out
    _need(out, "out", torch.int32)
    if out.numel() < 6 * total:
        raise ValueError(f"out holds {out.numel()} counts, {6 * total} needed")
    if ws is None:
        ws = _empty((max(16, lib().cdt_auroc_canaries_workspace_bytes(n)),), torch.uint8, scores)
    _need(ws, "ws", torch.uint8)
    _check(lib().cdt_auroc_canaries(n, arr, _ptr(scores), scores.numel(), seed, flags, _ptr(out),
                                    _ptr(ws), ws.numel(), _stream()))
    return out[:total]


VALUE_NAMES = ("auroc", "auroc_mw", "control", "control_mw", "pooled", "pooled_mw", "random",
               "random_mw")


def auroc_values(counts, pooled=None, baseline=None, out=None):
    """Eq. 6 from the counts of auroc(), computed on the device
    (cdt_auroc_values): [n][8] fp64, columns VALUE_NAMES (strict and
    Mann-Whitney for the detector, the control, the pooled ranking and the
    random baseline; NaN where there are no pairs or no such counts)."""
    torch = _torch()
    _need(counts, "counts", torch.int64)
    n = counts.shape[0]
    _need(counts, "counts", torch.int64, (n, 6))
    for name, t in (("pooled", pooled), ("baseline", baseline)):
        if t is not None:
            _need(t, name, torch.int64, (n, 3))
    out = _empty((n, 8), torch.float64, counts) if out is None else out
    _need(out, "values", torch.float64, (n, 8))
    _check(lib().cdt_auroc_values(n, _ptr(counts), _ptr(pooled), _ptr(baseline), _ptr(out),
                                  _stream()))
    return out


def u64(counts):
    """View int64 count tensors (copied to host) as uint64 numpy arrays."""
    return counts.cpu().numpy().view(np.uint64)
