"""bench.py's host-side pieces (CPU only): the multi-GPU refusal and the
reading of the committed rocprofv3 summaries that feed `roofline.traffic`
and the live pass's VALU figures."""
import os
import subprocess
import sys

from tests.conftest import ROOT

sys.path.insert(0, ROOT)
import bench  # noqa: E402

ELEMS_70B = 16 * 256 * 256 * 8192


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode != 0
    assert "one GPU" in r.stdout + r.stderr


def test_traffic_is_read_only_for_its_workload_and_sources(tmp_path):
    assert bench.measured_traffic("llama7b") is None
    t = bench.measured_traffic("llama70b")
    if t is not None:  # None once the drift sources change before a new counter pass
        # the step's batched launch over the 3 runs sharing the reference:
        # every run's fp16 activations and the reference once, and the scores
        alg = ELEMS_70B * (3 * 2 + 4) + 3 * 16 * 256 * bench.DRIFT_BYTES_PER_BLOCK
        assert abs(t / alg - 1.0) < 0.01
    # a summary whose recorded source hash does not match is ignored
    fake = tmp_path / "traffic.md"
    fake.write_text("drift_score_traffic_bytes_per_launch: 123\n"
                    "drift_score_source_sha256: 0000\n")
    assert bench._profile_fields(str(fake), "drift_score_", bench.DRIFT_SOURCES,
                                 "llama70b") is None


def test_valu_figures_are_plausible():
    assert bench.measured_valu("sweep") == (None, None)
    busy, per = bench.measured_valu("llama70b")
    if busy is not None:
        assert 0.0 < busy <= 1.05
        assert 10.0 < per < 100.0


def test_cpu_baseline_fields_on_tiny():
    """The oracle leg on the tiny workload (CPU only): the fields the
    benchmark contract names."""
    import types

    from paper_2607_19490_amd import workloads as W
    args = types.SimpleNamespace(workload="tiny", cpu_canaries=2)
    cb = bench.cpu_baseline(W, args)
    assert cb["kind"] == "oracle" and cb["unit"] == "GB/s" and cb["cores"] >= 1
    assert cb["value"] > 0 and isinstance(cb["sample"], str) and cb["sample"]
