"""GPU parity of the propagation model (the live error of each stage carried
into the next, cdt_canary_sim with carry > 0) against the oracle's chain,
bit for bit, and the substudies it enables (Sections 4.4, 5.3-5.5)."""
import numpy as np
import pytest

import oracle
from paper_2607_19490_amd import workloads as W
from tests.gpu_util import announce, h_bits, rel_err, require_gpu, to_dev, ulp_diff_f32

pytestmark = pytest.mark.gpu

CASES = {
    "gauss_add": dict(sigma_b=1e-3, tamper=1, eps=0.05),
    "t3_flip": dict(benign_dist=1, sigma_b=2e-2, tamper=2, flip_p=0.3),
    "block_scale": dict(benign_mode=1, sigma_b=2e-3, tamper=4, scale=1.05),
    "mixed_clean": dict(sigma_b=1e-2, tamper=7, eps=0.02, flip_p=0.02, scale=1.02, tamper_base=1),
    "redraw": dict(sigma_b=1e-2, redraw=True),
}
SHAPES = [(4, 8, 16, 256), (3, 5, 7, 264), (2, 3, 41, 1000), (64, 2, 3, 16), (12, 3, 5, 768)]


@pytest.fixture(scope="module")
def gpu():
    return require_gpu()


@pytest.mark.parametrize("carry", [0.3, 1.0])
@pytest.mark.parametrize("case", sorted(CASES))
@pytest.mark.parametrize("shape", SHAPES)
def test_chain_bit_exact(gpu, shape, case, carry):
    torch, cdt = gpu
    S, C, T, H = shape
    kw = dict(CASES[case])
    eps = kw.pop("eps", 0.0)
    announce(f"chain {case} carry={carry} {shape}")
    ref = oracle.ref_synth(S, C, T, H, 7, 1, oracle.outlier_gain(H, max(1, H // 100), 20.0, 7, 1))
    q, m = oracle.ref_stats(ref)
    ts, bs = oracle.block_scales(T, H, q, m, eps, kw.get("sigma_b", 0.0))
    mal = (1 << (S // 2)) | (1 << (S - 1))
    h = cdt.canary_sim(to_dev(torch, ref), seed=31, cfg_id=9, mal_mask=mal,
                       bscale=to_dev(torch, bs), tscale=to_dev(torch, ts), carry=carry, **kw)
    torch.cuda.synchronize()
    want = oracle.canary_sim(ref, seed=31, cfg_id=9, mal_mask=mal, bscale=bs, tscale=ts,
                             carry=carry, **kw)
    bad = int((h_bits(h) != want).sum())
    assert bad == 0, f"{bad} of {want.size} fp16 words differ"


# Exact-norm Gaussian tamper under the propagation model: which stages are
# malicious (indices into the shape's stages; -1 = the last) and the run.
EXACT_CASES = {
    "first_stage": ((0,), dict(sigma_b=1e-2)),
    "middle_block": ((None,), dict(benign_mode=1, sigma_b=2e-3)),
    "colluders_mixed": ((1, None, -1), dict(sigma_b=1e-2, tamper=7, flip_p=0.1, scale=1.05)),
    "t3_clean": ((None, -1), dict(benign_dist=1, sigma_b=2e-2, tamper_base=1)),
}


@pytest.mark.parametrize("case", sorted(EXACT_CASES))
@pytest.mark.parametrize("shape", [(4, 8, 16, 256), (3, 5, 7, 264), (6, 3, 41, 1000),
                                   (12, 3, 48, 768)])
def test_chain_exact_norm(gpu, shape, case):
    """Per-stage scales of the paper's Gaussian attack v + eps ||v|| N / ||N||
    when the live error is carried between stages (v depends on everything
    upstream): the fp32 scales within one ulp of the oracle's and the fp64
    norms within 1e-8 (sums of n terms in different orders, on inputs that
    differ by a scale ulp upstream), benign entries 0; then the carried live
    pass with those scales bit for bit against the oracle's."""
    torch, cdt = gpu
    S, C, T, H = shape
    stages, kw = EXACT_CASES[case]
    mal = 0
    for x in stages:
        mal |= 1 << (S // 2 if x is None else x % S)
    kw = dict(kw)
    kw.setdefault("tamper", 1)
    eps, g = 0.05, 0.7
    announce(f"chain exact norm {case} {shape} mal={mal:#x}")
    ref = oracle.ref_synth(S, C, T, H, 12, 0, oracle.outlier_gain(H, max(1, H // 100), 20.0, 12, 0))
    q, m = oracle.ref_stats(ref)
    _, bs = oracle.block_scales(T, H, q, m, 0.0, kw.get("sigma_b", 0.0))
    ref_d = to_dev(torch, ref)
    norms = torch.empty((S, C, 2), dtype=torch.float64, device="cuda")
    ts = cdt.tamper_scale_exact(ref_d, eps, norms=norms, bscale=to_dev(torch, bs), seed=14,
                                cfg_id=6, mal_mask=mal, carry=g, **kw)
    torch.cuda.synchronize()
    ts_o, norms_o = oracle.tamper_scale_exact(ref, eps, seed=14, cfg_id=6, bscale=bs,
                                              mal_mask=mal, carry=g, **kw)
    ts_d, norms_d = ts.cpu().numpy(), norms.cpu().numpy()
    assert ulp_diff_f32(ts_d, ts_o).max() <= 1
    assert rel_err(norms_d, norms_o) < 1e-8
    for s in range(S):
        if not (mal >> s) & 1:
            assert (ts_d[s] == 0).all() and (norms_d[s] == 0).all()
    assert (ts_d[[s for s in range(S) if (mal >> s) & 1]] > 0).all()
    h = cdt.canary_sim(ref_d, seed=14, cfg_id=6, mal_mask=mal, bscale=to_dev(torch, bs),
                       tscale=ts, carry=g, **kw)
    torch.cuda.synchronize()
    want = oracle.canary_sim(ref, seed=14, cfg_id=6, mal_mask=mal, bscale=bs, tscale=ts_d,
                             carry=g, **kw)
    assert int((h_bits(h) != want).sum()) == 0


def test_substudy_parity(gpu):
    """One substudy configuration (depth k = 4, the attacker's exact-norm
    Gaussian under the propagation model, Section 5.3) compared whole with
    the oracle's chain.  The substudies' outcomes are checked against a
    statistical model in tests/test_gpu_statistical.py."""
    torch, cdt = gpu
    announce("substudy parity")
    # whole-configuration parity: depth k = 4
    wl = W.substudies()
    rs = [r for r in wl.ref_sets if r.runs[0].label == "depth:k4"][0]
    run = rs.runs[0]
    gain = oracle.outlier_gain(rs.H, rs.n_out, W.OUTLIER_GAIN, wl.seed, rs.ref_set_id)
    ref_o = oracle.ref_synth(rs.S, rs.C, rs.T, rs.H, wl.seed, rs.ref_set_id, gain)
    assert run.exact_norm
    kw = dict(seed=wl.seed, cfg_id=run.cfg_id, benign_mode=run.benign_mode,
              sigma_b=run.sigma_b, mal_mask=rs.mal_mask, tamper=run.tamper, carry=run.carry)
    q, m = oracle.ref_stats(ref_o)
    _, bs_o = oracle.block_scales(rs.T, rs.H, q, m, run.eps, run.sigma_b)
    ts_o, _ = oracle.tamper_scale_exact(ref_o, run.eps, bscale=bs_o, **kw)
    ref = to_dev(torch, ref_o)
    _, bs = cdt.block_scales(*cdt.ref_stats(ref), rs.T, rs.H, run.eps, run.sigma_b)
    ts = cdt.tamper_scale_exact(ref, run.eps, bscale=bs, **kw)
    h = cdt.canary_sim(ref, bscale=bs, tscale=ts, **kw)
    score = cdt.drift_score(h, ref)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(bs.cpu().numpy(), bs_o)
    assert ulp_diff_f32(ts.cpu().numpy(), ts_o).max() <= 1
    # the live pass given the same scales: bit for bit
    h_o = oracle.canary_sim(ref_o, bscale=bs_o, tscale=ts.cpu().numpy(), **kw)
    np.testing.assert_array_equal(h_bits(h), h_o)
    s64, _, _ = oracle.drift_score(h_o, ref_o)
    assert rel_err(score.cpu().numpy(), s64) < 1e-5
