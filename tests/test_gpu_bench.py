"""bench.py's result line on the tiny workload, in this process: the keys
the benchmark contract names and the consistency of its figures."""
import types

import pytest

from tests.gpu_util import announce, require_gpu

pytestmark = pytest.mark.gpu


def _args(**kw):
    a = dict(gpus=1, steps=3, warmup=1, workload="tiny", no_sweep=True, sweep_only=False,
             sweep_reps=1, no_cpu_baseline=True, no_ablations=True, cpu_canaries=2,
             copy_calibration=False)
    a.update(kw)
    return types.SimpleNamespace(**a)


def test_bench_line_on_tiny():
    torch, cdt = require_gpu()
    import bench
    from paper_2607_19490_amd import workloads as W
    announce("bench line on tiny")
    res, _ = bench.run_main(torch, cdt, W, _args())
    for k in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step",
              "higher_is_better", "scaling", "vs_baseline", "dtype", "data", "config",
              "roofline"):
        assert k in res, k
    assert res["n_gpus"] == 1 and res["steps"] == 3 and res["warmup"] == 1
    assert res["config"]["workload"] == "tiny"
    assert res["value"] > 0 and res["ms_per_step"] > 0
    rs = W.tiny().ref_sets[0]
    scored = len(rs.runs) * (rs.elems * bench.DRIFT_BYTES_PER_ELEM
                             + rs.S * rs.C * bench.DRIFT_BYTES_PER_BLOCK)
    assert res["value"] == pytest.approx(scored / (res["ms_per_step"] * 1e-3) / 1e9, rel=1e-3)
    r = res["roofline"]
    for k in ("bound", "achieved", "peak", "unit", "frac", "traffic"):
        assert k in r, k
    assert r["bound"] == "hbm" and r["unit"] == "GB/s" and r["peak"] == bench.HBM_PEAK_GBPS
    assert r["frac"] == pytest.approx(r["achieved"] / r["peak"], abs=1e-4)
    assert r["traffic"] is None  # counters are committed for the 70B workload only
    nr = len(rs.runs)
    assert r["runs_per_launch"] == nr
    assert r["bytes_per_launch"] == (rs.elems * (2 * nr + 4)
                                     + nr * rs.S * rs.C * bench.DRIFT_BYTES_PER_BLOCK)
    assert r["achieved"] == pytest.approx(
        r["bytes_per_launch"] / (r["avg_launch_ms"] * 1e-3) / 1e9, rel=1e-2)  # rounded ms
    pr = res["per_run_launches"]
    assert pr["read_stream_GBps"] > 0 and pr["ms_per_step"] > 0
    assert res["detection"]["add0.05"] == 1.0
