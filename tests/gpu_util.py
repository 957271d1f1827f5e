"""Helpers shared by the GPU parity tests (no arithmetic of the method)."""

import numpy as np
import pytest


def require_gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    from paper_2607_19490_amd import cdt
    cdt.lib()  # raises when libcdt.so is missing: no fallback
    return torch, cdt


def to_dev(torch, a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def h_bits(t):
    """fp16 device tensor -> uint16 numpy bits."""
    return t.cpu().numpy().view(np.uint16)


def announce(msg):
    print(f"[gpu-case] {msg}", flush=True)


def rel_err(got, want):
    got = np.asarray(got, np.float64)
    want = np.asarray(want, np.float64)
    both_inf = np.isinf(got) & np.isinf(want) & (np.sign(got) == np.sign(want))
    denom = np.maximum(np.abs(want), 1e-300)
    r = np.where(both_inf, 0.0, np.abs(got - want) / denom)
    r = np.where((got == 0) & (want == 0), 0.0, r)
    return float(r.max()) if r.size else 0.0


def ulp_diff_f32(a, b):
    a = np.asarray(a, np.float32).view(np.int32).astype(np.int64)
    b = np.asarray(b, np.float32).view(np.int32).astype(np.int64)
    return np.abs(a - b)
