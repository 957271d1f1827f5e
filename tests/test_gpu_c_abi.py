"""The C ABI used from C alone (tests/c_abi/detect.c: hipMalloc'd buffers,
one stream, no Python or torch in the process): its Eq. 4 scores and
Eqs. 5-6 counts on a synthetic run against the oracle's."""
import os
import subprocess

import numpy as np
import pytest

import oracle
from paper_2607_19490_amd import workloads as W
from tests.conftest import ROOT
from tests.gpu_util import announce, rel_err

pytestmark = pytest.mark.gpu

EXE = os.path.join(ROOT, "tests", "c_abi", "detect")


@pytest.mark.parametrize("shape", [(4, 8, 16, 256), (16, 32, 64, 1024)])
def test_c_program_matches_oracle(shape):
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    if not os.path.exists(EXE):
        pytest.fail("tests/c_abi/detect is not built; run __graft_entry__.build()")
    S, C, T, H = shape
    seed, eps, sigma = 3, 0.05, 1e-3
    announce(f"C program {shape}")
    r = subprocess.run([EXE, str(S), str(C), str(T), str(H), str(seed), str(eps), str(sigma)],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stderr
    lines = dict(l.split(" ", 1) for l in r.stdout.strip().splitlines())
    scores = np.array(lines["scores"].split(), np.float32).reshape(C, S)
    counts = np.array(lines["counts"].split(), np.uint64)
    gain = oracle.outlier_gain(H, W.n_outliers(H), 20.0, seed, 0)
    ref = oracle.ref_synth(S, C, T, H, seed, 0, gain)
    q, m = oracle.ref_stats(ref)
    ts, _ = oracle.block_scales(T, H, q, m, eps, 0.0)
    mal = 1 << (S // 2)
    h = oracle.canary_sim(ref, seed=seed, cfg_id=1, sigma_b=sigma, mal_mask=mal, tamper=1,
                          tscale=ts)
    s64, s32, _ = oracle.drift_score(h, ref)
    assert rel_err(scores, s64) < 1e-5
    want, _ = oracle.auroc_config(s32, mal, seed=seed, cfg_id=1, flags=1)
    np.testing.assert_array_equal(counts, want)
