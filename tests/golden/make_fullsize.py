"""Writes tests/golden/fullsize_<workload>.npz: the CPU oracle's result for
every (shard, canary) block of every run of the full-size workloads
  snr       16 x 128 x 128 x 4096, 40 runs (20 noise levels, Gaussian and
            Student-t benign noise, Gaussian tamper 0.02);
  sweep     the 216-configuration factorial over nine reference sets;
  llama70b  16 x 256 x 256 x 8192, 3 runs (Gaussian 0.05, flip 0.1%,
            rescale 1.05).
Per block: the Eq. 4 score (fp64), the digest of its fp32 references and the
digest of its fp16 live activations (tests/digest.py).  Every value comes
from oracle/ alone (the workload module only supplies shapes and
parameters).  The GPU tests compare all blocks against these files and
recount Eqs. 5-6 from the stored scores with the oracle.

Blocks are regenerated one at a time (reference, block scales, live pass,
Eq. 4 for every run), spread over host threads; ctypes releases the
interpreter lock inside the oracle's C routines.

Usage: python tests/golden/make_fullsize.py [snr|sweep|llama70b ...] [--threads N]
"""
import argparse
import hashlib
import json
import os
import sys
import time
from concurrent.futures import ThreadPoolExecutor

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import oracle  # noqa: E402
from paper_2607_19490_amd import workloads as W  # noqa: E402
from tests.digest import digest_np  # noqa: E402

NAMES = ("snr", "sweep", "llama70b")


def path_for(name):
    return os.path.join(HERE, f"fullsize_{name}.npz")


def layout(wl):
    """Offsets of every reference set's blocks and every run's blocks in the
    flat arrays, in the workload's order (sets, then runs within a set)."""
    set_off, run_off, o_set, o_run = [], [], 0, 0
    for rs in wl.ref_sets:
        set_off.append(o_set)
        o_set += rs.S * rs.C
        for _ in rs.runs:
            run_off.append(o_run)
            o_run += rs.S * rs.C
    return set_off, run_off, o_set, o_run


def block_job(wl, rs, gain, s, c):
    """One block through every run of its reference set."""
    ref = oracle.ref_block(s, c, rs.T, rs.H, wl.seed, rs.ref_set_id, gain)
    q, m = oracle.ref_stats_block(ref)
    out = []
    for run in rs.runs:
        assert not run.exact_norm and run.carry == 0.0
        ts, bs = oracle.block_scales(rs.T, rs.H, np.array([q]), np.array([m]), run.eps,
                                     run.sigma_b)
        h = oracle.sim_block(s, c, ref, seed=wl.seed, cfg_id=run.cfg_id,
                             benign_mode=run.benign_mode, benign_dist=run.benign_dist,
                             sigma_b=run.sigma_b, bscale=bs[0], malicious=s in rs.mal_shards,
                             tamper=run.tamper, tamper_base=run.tamper_base, tscale=ts[0],
                             flip_p=run.flip_p, scale=run.scale)
        m64, _, _ = oracle.drift_block(h, ref)
        out.append((m64, digest_np(h)))
    return s, c, digest_np(ref), out


def oracle_sha256():
    with open(os.path.join(ROOT, "oracle", "oracle.c"), "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()


def make(name, threads):
    wl = W.get(name)
    set_off, run_off, n_set, n_run = layout(wl)
    score64 = np.full(n_run, np.nan)
    hdig = np.zeros(n_run, np.uint64)
    refdig = np.zeros(n_set, np.uint64)
    t0 = time.time()
    k = 0
    for i, rs in enumerate(wl.ref_sets):
        gain = oracle.outlier_gain(rs.H, rs.n_out, W.OUTLIER_GAIN, wl.seed, rs.ref_set_id)
        blocks = [(s, c) for s in range(rs.S) for c in range(rs.C)]
        with ThreadPoolExecutor(max_workers=threads) as ex:
            for done, (s, c, rd, runs) in enumerate(
                    ex.map(lambda b: block_job(wl, rs, gain, *b), blocks)):
                refdig[set_off[i] + s * rs.C + c] = rd
                for r, (m64, hd) in enumerate(runs):
                    o = run_off[k + r]
                    score64[o + c * rs.S + s] = m64
                    hdig[o + s * rs.C + c] = hd
                if done % 256 == 255:
                    print(f"{name} set {i}: {done + 1}/{len(blocks)} blocks, "
                          f"{time.time() - t0:.0f} s", flush=True)
        k += len(rs.runs)
    assert not np.isnan(score64).any()
    meta = {"workload": name, "seed": wl.seed, "oracle_c_sha256": oracle_sha256(),
            "cfg_ids": [r.cfg_id for rs in wl.ref_sets for r in rs.runs],
            "shapes": [[rs.S, rs.C, rs.T, rs.H] for rs in wl.ref_sets],
            "score_layout": "per run [C][S]", "digest_layout": "per set / run [S][C]",
            "seconds": round(time.time() - t0, 1), "threads": threads}
    np.savez_compressed(path_for(name), score64=score64, hdig=hdig, refdig=refdig,
                        meta=np.array(json.dumps(meta)))
    print(f"{name}: wrote {path_for(name)} in {time.time() - t0:.0f} s", flush=True)


def main():
    p = argparse.ArgumentParser()
    p.add_argument("names", nargs="*", default=list(NAMES))
    p.add_argument("--threads", type=int, default=max(1, min(16, len(os.sched_getaffinity(0)))))
    a = p.parse_args()
    for name in a.names:
        assert name in NAMES, name
        make(name, a.threads)


if __name__ == "__main__":
    main()
