"""The stored full-size oracle results (tests/golden/fullsize_*.npz) against
the oracle as it is now: sampled blocks of every workload are regenerated
(reference, block scales, live pass, Eq. 4) and must reproduce the stored
digests bit for bit and the stored scores exactly.  This keeps the files
that the full-size GPU tests compare against tied to oracle/, which alone
wrote them (tests/golden/make_fullsize.py)."""
import json
import os

import numpy as np
import pytest

import oracle
from paper_2607_19490_amd import workloads as W
from tests.digest import digest_np
from tests.golden import make_fullsize as M

GOLDEN = os.path.dirname(M.__file__)


def _load(name):
    z = np.load(M.path_for(name))
    return z["score64"], z["hdig"], z["refdig"], json.loads(str(z["meta"]))


# (workload, reference set index, blocks): first, last and a middle block,
# malicious shards included
SAMPLES = [("snr", 0, [(8, 77)]),
           ("llama70b", 0, [(0, 0), (8, 255)]),
           ("sweep", 0, [(4, 31)]),
           ("sweep", 4, [(8, 0)]),
           ("sweep", 8, [(31, 17)])]


@pytest.mark.parametrize("name", M.NAMES)
def test_files_match_the_workloads(name):
    wl = W.get(name)
    score64, hdig, refdig, meta = _load(name)
    set_off, run_off, n_set, n_run = M.layout(wl)
    assert score64.shape == hdig.shape == (n_run,) and refdig.shape == (n_set,)
    assert meta["cfg_ids"] == [r.cfg_id for rs in wl.ref_sets for r in rs.runs]
    assert meta["shapes"] == [[rs.S, rs.C, rs.T, rs.H] for rs in wl.ref_sets]
    assert np.isfinite(score64).all() and (score64 >= 0).all()


@pytest.mark.parametrize("name,set_index,blocks", SAMPLES,
                         ids=[f"{s[0]}-set{s[1]}" for s in SAMPLES])
def test_sampled_blocks_regenerate(name, set_index, blocks):
    wl = W.get(name)
    score64, hdig, refdig, _ = _load(name)
    set_off, run_off, _, _ = M.layout(wl)
    rs = wl.ref_sets[set_index]
    k0 = sum(len(r.runs) for r in wl.ref_sets[:set_index])
    gain = oracle.outlier_gain(rs.H, rs.n_out, W.OUTLIER_GAIN, wl.seed, rs.ref_set_id)
    for s, c in blocks:
        _, _, rd, runs = M.block_job(wl, rs, gain, s, c)
        assert refdig[set_off[set_index] + s * rs.C + c] == rd, (s, c)
        for r, (m64, hd) in enumerate(runs):
            o = run_off[k0 + r]
            assert hdig[o + s * rs.C + c] == hd, (rs.runs[r].label, s, c)
            assert score64[o + c * rs.S + s] == m64, (rs.runs[r].label, s, c)


def test_digest_detects_single_element_changes():
    """The digest changes under any single-element change (the weight 2e+1 is
    odd, so invertible mod 2^64) and does not depend on anything else."""
    rng = np.random.default_rng(0)
    h = rng.integers(0, 1 << 16, 4096, dtype=np.uint16)
    d0 = digest_np(h)
    for e in (0, 1, 2047, 4095):
        for delta in (1, 0x8000, 0xFFFF):
            g = h.copy()
            g[e] = np.uint16((int(g[e]) + delta) & 0xFFFF)
            assert digest_np(g) != d0
    a = rng.standard_normal(4096).astype(np.float32)
    b = a.copy()
    b[100] = np.nextafter(b[100], np.float32(np.inf))
    assert digest_np(a) != digest_np(b)
    assert digest_np(h) == digest_np(h.copy())
