"""Per-block digests of activation arrays, for comparing whole full-size
workloads with stored oracle results without storing the arrays.

A block's digest is  sum_e bits(x_e) * (2e + 1)  mod 2^64  over its
elements e = 0 .. n-1 (bits: the element's fp16 or fp32 bit pattern as an
unsigned integer).  Any single-element difference changes it, since 2e + 1
is odd and so invertible mod 2^64.  Test infrastructure: no arithmetic of
the method is here.  The numpy form digests the oracle's blocks, the torch
form the device's arrays; both wrap mod 2^64.
"""
import numpy as np

_W = {}


def _weights(n):
    w = _W.get(n)
    if w is None:
        w = 2 * np.arange(n, dtype=np.uint64) + np.uint64(1)
        _W[n] = w
    return w


def digest_np(bits):
    """bits: uint16 (fp16) or float32 array of one block -> uint64 digest."""
    a = np.ascontiguousarray(bits).ravel()
    if a.dtype == np.float32:
        x = a.view(np.uint32).astype(np.uint64)
    elif a.dtype == np.uint16:
        x = a.astype(np.uint64)
    else:
        raise TypeError(a.dtype)
    with np.errstate(over="ignore"):
        return np.uint64((x * _weights(a.size)).sum(dtype=np.uint64))


def digest_torch(torch, x):
    """x: device tensor [..., n] of fp16 or fp32 -> int64 tensor [...] of the
    digests of its rows (view the result as uint64 on the host)."""
    n = x.shape[-1]
    w = 2 * torch.arange(n, dtype=torch.int64, device=x.device) + 1
    if x.dtype == torch.float16:
        v = x.view(torch.int16).to(torch.int64) & 0xFFFF
    elif x.dtype == torch.float32:
        v = x.view(torch.int32).to(torch.int64) & 0xFFFFFFFF
    else:
        raise TypeError(x.dtype)
    return (v * w).sum(dim=-1)
