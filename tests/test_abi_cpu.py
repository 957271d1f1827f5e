"""The C ABI without a GPU: the library loads, exports every symbol the
header declares, and rejects bad arguments before any device work."""
import ctypes
import os
import re
import subprocess

import pytest

from tests.conftest import ROOT

HEADER = os.path.join(ROOT, "include", "cdt.h")


@pytest.fixture(scope="module")
def cdt():
    from paper_2607_19490_amd import build, cdt as binding
    if not os.path.exists(binding.LIB_PATH):
        build.build()
    binding.lib()
    return binding


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(cdt_[a-z0-9_]+)\s*\(", text)))


def test_header_declarations_are_exported(cdt):
    names = _declared()
    assert "cdt_drift_score" in names and "cdt_canary_sim" in names and "cdt_auroc" in names
    L = cdt.lib()
    for n in names:
        assert hasattr(L, n), n
    assert sorted(names) == sorted(cdt.exported_symbols())


def test_version_and_sizes(cdt):
    L = cdt.lib()
    assert L.cdt_version() == 11 == cdt.ABI_VERSION
    assert L.cdt_reduce_workspace_bytes(16, 256, 256, 8192) == 4096 * 64 * 24
    assert L.cdt_reduce_workspace_bytes(4, 8, 16, 256) == 32 * 1 * 24
    assert L.cdt_reduce_workspace_bytes(4, 8, 0, 256) == 0
    assert L.cdt_auroc_workspace_bytes(216) == 216 * 32


def STRUCTS(cdt):
    return (("cdt_sim_params", cdt.SimParams), ("cdt_auroc_cfg", cdt.AurocCfg),
            ("cdt_drift_job", cdt.DriftJob), ("cdt_sim_job", cdt.SimJob))


def test_struct_layouts_match_the_header(cdt, tmp_path):
    """Compile the header with the host C compiler and compare every field
    offset and struct size with the ctypes mirrors of the binding."""
    src = tmp_path / "layout.c"
    lines = ['#include <stdio.h>', '#include <stddef.h>', '#include "cdt.h"', "int main(void){"]
    for cname, py in STRUCTS(cdt):
        lines.append(f'printf("{cname} size %zu\\n", sizeof({cname}));')
        for f, _ in py._fields_:
            lines.append(f'printf("{cname} {f} %zu\\n", offsetof({cname}, {f}));')
    lines.append("return 0;}")
    src.write_text("\n".join(lines))
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-I", os.path.join(ROOT, "include"), str(src), "-o", str(exe)],
                   check=True)
    out = subprocess.run([str(exe)], check=True, capture_output=True, text=True).stdout
    got = {tuple(l.split()[:2]): int(l.split()[2]) for l in out.strip().splitlines()}
    for cname, py in STRUCTS(cdt):
        assert got[(cname, "size")] == ctypes.sizeof(py)
        for f, _ in py._fields_:
            assert got[(cname, f)] == getattr(py, f).offset, (cname, f)


def _err(cdt):
    return cdt.lib().cdt_last_error().decode()


def test_shape_and_pointer_validation(cdt):
    L = cdt.lib()
    assert L.cdt_drift_score(2, 2, 3, 12, None, None, None, None, None, 0, None) == cdt.EINVAL
    assert "multiple of 8" in _err(cdt)
    assert L.cdt_drift_score(2, 2, 1 << 16, 1 << 16, 16, 16, 16, None, 16, 1 << 40, None) == cdt.ELIMIT
    assert L.cdt_drift_score(2, 2, 3, 16, None, None, 16, None, 16, 1 << 20, None) == cdt.EINVAL
    assert L.cdt_drift_score(2, 2, 3, 16, 8, 16, 16, None, 16, 1 << 20, None) == cdt.EALIGN
    # workspace too small
    assert L.cdt_drift_score(2, 2, 3, 16, 16, 16, 16, None, 16, 15, None) == cdt.EINVAL
    assert "workspace" in _err(cdt)
    for fn in (L.cdt_drift_score_f16ref, L.cdt_cosine_score):
        assert fn(2, 2, 3, 12, None, None, None, None, None, 0, None) == cdt.EINVAL
        assert fn(2, 2, 3, 16, 8, 16, 16, None, 16, 1 << 20, None) == cdt.EALIGN
        assert fn(2, 2, 3, 16, 16, 16, 16, None, 16, 15, None) == cdt.EINVAL
        assert fn(0, 2, 3, 16, None, None, None, None, None, 0, None) == cdt.OK
    # the compute-free read of Eq. 4's stream checks its arguments the same way
    rs = L.cdt_drift_read_stream
    assert rs(2, 2, 3, 12, None, None, None, 0, None) == cdt.EINVAL
    assert rs(2, 2, 3, 16, None, 16, 16, 1 << 20, None) == cdt.EINVAL
    assert rs(2, 2, 3, 16, 8, 16, 16, 1 << 20, None) == cdt.EALIGN
    assert rs(2, 2, 3, 16, 16, 16, 16, 15, None) == cdt.EINVAL
    assert "workspace" in _err(cdt)
    assert rs(2, 2, 3, 16, 16, 16, 24, 1 << 20, None) == cdt.EALIGN
    assert rs(2, 2, 0, 16, None, None, None, 0, None) == cdt.OK
    assert rs(1 << 16, 1 << 16, 1 << 10, 8, 16, 16, 16, 1 << 20, None) == cdt.ELIMIT
    # empty shapes are accepted without touching the device
    assert L.cdt_drift_score(0, 2, 3, 16, None, None, None, None, None, 0, None) == cdt.OK
    # block count and total size limits (sizes derived from the shape stay exact)
    assert L.cdt_drift_score(1 << 20, 1 << 13, 1, 8, 16, 16, 16, None, 16, 1 << 20,
                             None) == cdt.ELIMIT
    assert "S*C=" in _err(cdt)
    assert L.cdt_drift_score(1 << 16, 1 << 16, 1 << 10, 8, 16, 16, 16, None, 16, 1 << 20,
                             None) == cdt.ELIMIT
    assert "2^40" in _err(cdt)
    assert L.cdt_ref_synth(2, 0, 3, 16, 0, 0, 0, None, None, None) == cdt.OK
    assert L.cdt_ref_synth(2, 2, 3, 16, 0, 1 << 24, 0, 16, 16, None) == cdt.ELIMIT
    # global canary indices must fit the 32-bit counter word
    # (2 canaries from 2^32 - 2 pass that check and stop at the NULL arrays)
    assert L.cdt_ref_synth(2, 2, 3, 16, 0, 0, (1 << 32) - 2, None, None, None) == cdt.EINVAL
    assert "NULL" in _err(cdt)
    assert L.cdt_ref_synth(2, 3, 3, 16, 0, 0, (1 << 32) - 2, 16, 16, None) == cdt.ELIMIT
    assert "canary_base" in _err(cdt)


def test_sim_param_validation(cdt):
    L = cdt.lib()

    def call(S=4, **kw):
        base = dict(seed=0, cfg_id=0, sigma_b=1e-3)
        base.update(kw)
        tscale = base.pop("tscale_ptr", 16)
        p = cdt.sim_params(**base)
        p.tscale = tscale
        return L.cdt_canary_sim(S, 2, 2, 16, ctypes.byref(p), 16, 16, None)

    assert call(S=65) == cdt.ELIMIT
    assert call(cfg_id=1 << 24) == cdt.ELIMIT
    assert call(benign_mode=2) == cdt.EINVAL
    assert call(benign_dist=2) == cdt.EINVAL
    assert call(tamper=8) == cdt.EINVAL
    assert call(sigma_b=-1.0) == cdt.EINVAL
    assert call(sigma_b=float("nan")) == cdt.EINVAL
    assert call(flip_p=1.5) == cdt.EINVAL
    assert call(scale=float("inf")) == cdt.EINVAL
    assert call(benign_mode=1) == cdt.EINVAL  # BLOCK noise without bscale
    assert "bscale" in _err(cdt)
    assert call(mal_mask=1, tamper=1, tscale_ptr=None) == cdt.EINVAL
    # the fused launch validates the same parameters
    p = cdt.sim_params(seed=0, cfg_id=1 << 24)
    assert L.cdt_sim_score(4, 2, 2, 16, ctypes.byref(p), 16, None, 16, None, 16, 1 << 20,
                           None) == cdt.ELIMIT
    p = cdt.sim_params(seed=0, cfg_id=0)
    assert L.cdt_sim_score(4, 2, 2, 16, ctypes.byref(p), 16, None, None, None, 16, 1 << 20,
                           None) == cdt.EINVAL
    assert L.cdt_sim_score(4, 2, 2, 16, ctypes.byref(p), 16, 8, 16, None, 16, 1 << 20,
                           None) == cdt.EALIGN
    assert L.cdt_sim_score(4, 2, 2, 16, ctypes.byref(p), 16, None, 16, None, 16, 1,
                           None) == cdt.EINVAL
    assert call(canary_base=(1 << 32) - 1) == cdt.ELIMIT  # C = 2 canaries from 2^32 - 1
    assert "canary_base" in _err(cdt)
    p = cdt.sim_params(seed=0, cfg_id=0)
    p.reserved = 1
    assert L.cdt_canary_sim(4, 2, 2, 16, ctypes.byref(p), 16, 16, None) == cdt.EINVAL
    assert call(carry=1.5) == cdt.EINVAL
    assert call(carry=-0.1) == cdt.EINVAL
    p = cdt.sim_params(seed=0, cfg_id=0, carry=0.5)
    assert L.cdt_sim_score(4, 2, 2, 16, ctypes.byref(p), 16, None, 16, None, 16, 1 << 20,
                           None) == cdt.EINVAL
    assert "carry" in _err(cdt)
    # under the propagation model the exact-norm scale is defined (from the
    # attacker's untampered live output); its argument checks still apply
    assert L.cdt_tamper_scale_exact(65, 2, 2, 16, ctypes.byref(p), 16, 0.1, 16, None, 16,
                                    1 << 20, None) == cdt.ELIMIT
    assert L.cdt_tamper_scale_exact(4, 2, 2, 16, ctypes.byref(p), 16, 0.1, None, None, 16,
                                    1 << 20, None) == cdt.EINVAL
    assert "tscale is NULL" in _err(cdt)
    assert L.cdt_tamper_scale_exact(4, 2, 2, 16, ctypes.byref(p), 16, 0.1, 16, None, 16,
                                    8, None) == cdt.EINVAL
    assert "workspace" in _err(cdt)
    p = cdt.sim_params(seed=0, cfg_id=0)
    p.redraw = 2
    assert L.cdt_canary_sim(4, 2, 2, 16, ctypes.byref(p), 16, 16, None) == cdt.EINVAL
    assert L.cdt_canary_sim(4, 2, 2, 16, None, 16, 16, None) == cdt.EINVAL


def test_auroc_validation(cdt):
    L = cdt.lib()
    arr, n = cdt.auroc_cfg_array([(65, 4, 0, 1, 0)])
    assert L.cdt_auroc(n, arr, 16, 1000, 0, 0, 16, None, None, 16, 64, None) == cdt.ELIMIT
    arr, n = cdt.auroc_cfg_array([(8, 4, 0, 1, 0), (8, 4, 30, 1, 1)])
    assert L.cdt_auroc(n, arr, 16, 60, 0, 0, 16, None, None, 16, 64, None) == cdt.EINVAL
    assert "outside" in _err(cdt)
    arr, n = cdt.auroc_cfg_array([(64, 300, 0, 1, 0)])
    assert L.cdt_auroc(n, arr, 16, 64 * 300, 0, 2, 16, 16, None, 16, 64, None) == cdt.ELIMIT
    assert L.cdt_auroc(n, arr, 16, 64 * 300, 0, 2, 16, None, None, 16, 64, None) == cdt.EINVAL
    assert L.cdt_auroc(n, arr, 16, 64 * 300, 0, 8, 16, None, None, 16, 64, None) == cdt.EINVAL
    arr, n = cdt.auroc_cfg_array([(8, 4, 0, 1, 0)])
    assert L.cdt_auroc(n, arr, 16, 32, 0, 0, 16, None, None, 16, 31, None) == cdt.EINVAL
    assert L.cdt_auroc(0, arr, None, 0, 0, 0, None, None, None, None, 0, None) == cdt.OK
    arr, n = cdt.auroc_cfg_array([(8, 4, 0, 1, 0)])
    assert L.cdt_auroc(n, arr, 16, 32, 0, 8, 16, None, None, 16, 64, None) == cdt.EINVAL
    assert "baseline" in _err(cdt)
    assert L.cdt_auroc(n, arr, 16, 32, 0, 16, 16, None, None, 16, 64, None) == cdt.EINVAL
    arr, n = cdt.auroc_cfg_array([(8, 4, 0, 1, 0, (1 << 32) - 3)])
    assert L.cdt_auroc(n, arr, 16, 32, 0, 0, 16, None, None, 16, 64, None) == cdt.ELIMIT
    assert "canary_base" in _err(cdt)


def test_auroc_upload_and_launch_validation(cdt):
    """The upload checks the table as cdt_auroc does; the launch checks its
    own arguments (the table itself is re-checked by the kernels)."""
    L = cdt.lib()
    up, run = L.cdt_auroc_upload, L.cdt_auroc_launch
    arr, n = cdt.auroc_cfg_array([(65, 4, 0, 1, 0)])
    assert up(n, arr, 1000, 0, 16, 64, None) == cdt.ELIMIT
    arr, n = cdt.auroc_cfg_array([(8, 4, 0, 1, 0), (8, 4, 30, 1, 1)])
    assert up(n, arr, 60, 0, 16, 64, None) == cdt.EINVAL and "outside" in _err(cdt)
    arr, n = cdt.auroc_cfg_array([(64, 300, 0, 1, 0)])
    assert up(n, arr, 64 * 300, cdt.AUROC_POOLED, 16, 64, None) == cdt.ELIMIT
    arr, n = cdt.auroc_cfg_array([(8, 4, 0, 1, 0)])
    assert up(n, arr, 32, 0, 16, 31, None) == cdt.EINVAL  # table too small
    assert up(n, arr, 32, 0, 8, 64, None) == cdt.EALIGN
    assert up(n, None, 32, 0, 16, 64, None) == cdt.EINVAL
    assert up(n, arr, 32, 16, 16, 64, None) == cdt.EINVAL  # bad flags
    assert up(0, None, 0, 0, None, 0, None) == cdt.OK
    assert run(1, 16, 16, 32, 0, 16, 16, None, None, None) == cdt.EINVAL  # bad flags
    assert run(1, 16, 16, 32, 0, 0, None, None, None, None) == cdt.EINVAL  # no counts
    assert run(1, 16, 16, 32, 0, cdt.AUROC_POOLED, 16, None, None, None) == cdt.EINVAL
    assert run(1, 16, 16, 32, 0, cdt.AUROC_RANDOM, 16, None, None, None) == cdt.EINVAL
    assert run(1, None, 16, 32, 0, 0, 16, None, None, None) == cdt.EINVAL
    assert run(1, 16, None, 32, 0, 0, 16, None, None, None) == cdt.EINVAL
    assert run(1, 8, 16, 32, 0, 0, 16, None, None, None) == cdt.EALIGN
    assert run((1 << 24) + 1, 16, 16, 32, 0, 0, 16, None, None, None) == cdt.ELIMIT
    assert run(0, None, None, 0, 0, 0, None, None, None, None) == cdt.OK


def test_auroc_canaries_validation(cdt):
    """Eq. 5 per canary: the table is checked as cdt_auroc checks it, the
    pooled flag is refused (it has no per-canary form), and the outputs and
    the workspace (table plus canary offsets) are checked before any device
    work."""
    L = cdt.lib()
    f = L.cdt_auroc_canaries
    need = L.cdt_auroc_canaries_workspace_bytes
    assert need(0) == 0 and need(1) == 256 + 8 and need(9) == 512 + 72
    arr, n = cdt.auroc_cfg_array([(8, 4, 0, 1, 0)])
    assert f(n, arr, 16, 32, 0, cdt.AUROC_POOLED, 16, 16, 264, None) == cdt.EINVAL
    assert "pooled" in _err(cdt)
    assert f(n, arr, 16, 32, 0, 16, 16, 16, 264, None) == cdt.EINVAL  # bad flags
    arr65, n65 = cdt.auroc_cfg_array([(65, 4, 0, 1, 0)])
    assert f(n65, arr65, 16, 1000, 0, 0, 16, 16, 264, None) == cdt.ELIMIT
    arr2, n2 = cdt.auroc_cfg_array([(8, 4, 0, 1, 0), (8, 4, 30, 1, 1)])
    assert f(n2, arr2, 16, 60, 0, 0, 16, 16, 264, None) == cdt.EINVAL and "outside" in _err(cdt)
    assert f(n, None, 16, 32, 0, 0, 16, 16, 264, None) == cdt.EINVAL
    assert f(n, arr, 16, 32, 0, 0, None, 16, 264, None) == cdt.EINVAL  # no per_canary
    assert "per_canary" in _err(cdt)
    assert f(n, arr, None, 32, 0, 0, 16, 16, 264, None) == cdt.EINVAL  # no scores
    assert f(n, arr, 16, 32, 0, 0, 16, 16, 263, None) == cdt.EINVAL  # workspace too small
    assert f(n, arr, 16, 32, 0, 0, 16, None, 264, None) == cdt.EINVAL
    assert f(n, arr, 16, 32, 0, 0, 16, 8, 264, None) == cdt.EALIGN
    assert f(0, None, None, 0, 0, 0, None, None, 0, None) == cdt.OK
    empty, ne = cdt.auroc_cfg_array([(8, 0, 0, 1, 0)])  # no canaries: nothing to write
    assert f(ne, empty, None, 0, 0, 1, None, None, 0, None) == cdt.OK


def test_scale_and_outlier_validation(cdt):
    L = cdt.lib()
    assert L.cdt_block_scales(4, 2, 8, 16, 16, -1.0, 0.0, 16, 16, None) == cdt.EINVAL
    assert L.cdt_block_scales(4, 2, 8, None, 16, 0.1, 0.0, 16, None, None) == cdt.EINVAL
    assert L.cdt_block_scales(0, 2, 8, None, None, 0.1, 0.0, 16, None, None) == cdt.OK
    assert L.cdt_outlier_gain(40000, 1, 20.0, 0, 0, 16, None) == cdt.ELIMIT
    assert L.cdt_outlier_gain(16, 17, 20.0, 0, 0, 16, None) == cdt.EINVAL
    assert L.cdt_outlier_gain(16, 1, 20.0, 0, 0, None, None) == cdt.EINVAL
    assert L.cdt_outlier_gain(0, 0, 20.0, 0, 0, None, None) == cdt.OK


def test_noalloc_limit_is_checked_on_the_host(cdt):
    """cdt_drift_score_noalloc rejects a shape whose partial sums exceed the
    library's scratch, and a bad shape, before any device call."""
    L = cdt.lib()
    # 16 x 1024 blocks of 64 chunks: 16 MiB of partial sums against 8 MiB
    assert L.cdt_drift_score_noalloc(16, 1024, 256, 8192, None, None, None, None, None) == \
        cdt.ELIMIT
    assert "scratch" in _err(cdt) and "8388608" in _err(cdt)
    assert L.cdt_drift_score_noalloc(2, 2, 3, 12, None, None, None, None, None) == cdt.EINVAL
    assert "multiple of 8" in _err(cdt)
    # one-chunk blocks use no scratch: any number of them passes the limit
    # and fails only on the NULL score pointer
    assert L.cdt_drift_score_noalloc(64, 1 << 20, 1, 8, None, None, None, None, None) == \
        cdt.EINVAL
    assert "score is NULL" in _err(cdt)


def test_batch_calls_validate_every_job_on_the_host(cdt):
    """The batched live pass and Eq. 4 reject a bad job (and name it) before
    any device call; a batch whose jobs are all empty does nothing."""
    L = cdt.lib()
    jobs = (cdt.DriftJob * 2)()
    jobs[0] = cdt.DriftJob(2, 2, 3, 16, 16, 16, 16, None)
    jobs[1] = cdt.DriftJob(2, 2, 3, 12, 16, 16, 16, None)
    assert L.cdt_drift_score_batch(2, jobs, 16, 1 << 20, None) == cdt.EINVAL
    assert "multiple of 8" in _err(cdt)
    assert L.cdt_drift_batch_workspace_bytes(2, jobs) == 0
    jobs[1] = cdt.DriftJob(2, 2, 3, 16, 8, 16, 16, None)
    assert L.cdt_drift_score_batch(2, jobs, 16, 1 << 20, None) == cdt.EALIGN
    assert "job 1" in _err(cdt)
    jobs[1] = cdt.DriftJob(2, 2, 3, 16, 16, 16, None, None)
    assert L.cdt_drift_score_batch(2, jobs, 16, 1 << 20, None) == cdt.EINVAL
    # sizes: the job table and the group table (each rounded to 256 B), then
    # the multi-chunk jobs' partials
    jobs[0] = cdt.DriftJob(16, 256, 256, 8192, 16, 16, 16, None)
    jobs[1] = cdt.DriftJob(4, 8, 16, 256, 16, 16, 16, None)  # one chunk per block
    nbytes = L.cdt_drift_batch_workspace_bytes(2, jobs)
    assert nbytes == 256 + 256 + 4096 * 64 * 16
    assert L.cdt_drift_score_batch(2, jobs, 16, nbytes - 16, None) == cdt.EINVAL
    empty = (cdt.DriftJob * 1)(cdt.DriftJob(0, 2, 3, 16, None, None, None, None))
    assert L.cdt_drift_score_batch(1, empty, None, 0, None) == cdt.OK
    # the read-stream aid takes the same arguments and checks them the same way
    rs = L.cdt_drift_read_stream_batch
    assert rs(2, jobs, 16, nbytes - 16, None) == cdt.EINVAL
    assert rs(2, jobs, 8, nbytes, None) == cdt.EALIGN
    assert rs(1, empty, None, 0, None) == cdt.OK
    bad = (cdt.DriftJob * 1)(cdt.DriftJob(2, 2, 3, 12, 16, 16, 16, None))
    assert rs(1, bad, 16, 1 << 20, None) == cdt.EINVAL and "multiple of 8" in _err(cdt)
    p = cdt.sim_params(seed=0, cfg_id=0)
    p3 = cdt.sim_params(seed=0, cfg_id=0, benign_dist=1)
    sj = (cdt.SimJob * 2)()
    sj[0] = cdt.SimJob(4, 2, 2, 16, ctypes.pointer(p), 16, 16)
    sj[1] = cdt.SimJob(4, 2, 2, 16, ctypes.pointer(p3), 16, 16)
    assert L.cdt_canary_sim_batch(2, sj, 16, 1 << 20, None) == cdt.EINVAL
    assert "same benign noise" in _err(cdt)
    pc = cdt.sim_params(seed=0, cfg_id=0, carry=0.5)
    sj[1] = cdt.SimJob(4, 2, 2, 16, ctypes.pointer(pc), 16, 16)
    assert L.cdt_canary_sim_batch(2, sj, 16, 1 << 20, None) == cdt.EINVAL
    assert "carry" in _err(cdt)
    sj[1] = cdt.SimJob(65, 2, 2, 16, ctypes.pointer(p), 16, 16)
    assert L.cdt_canary_sim_batch(2, sj, 16, 1 << 20, None) == cdt.ELIMIT
    sj[1] = cdt.SimJob(4, 2, 2, 16, ctypes.pointer(p), 16, 16)
    assert L.cdt_canary_sim_batch(2, sj, 16, 8, None) == cdt.EINVAL
    assert "workspace" in _err(cdt)
    assert L.cdt_canary_sim_stream(2, 2, 3, 12, None, None, None) == cdt.EINVAL
