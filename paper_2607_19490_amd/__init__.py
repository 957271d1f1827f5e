"""Canary-versus-reference activation drift detector for MI355X (gfx950).

The compute path lives in ``libcdt.so`` (hand-written HIP kernels behind a C
ABI, declared in ``include/cdt.h``); ``paper_2607_19490_amd.cdt`` is its thin
Python binding.  ``workloads`` and ``inputs`` hold workload shapes and seeded
synthetic inputs only.
"""
