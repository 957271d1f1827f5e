"""The fused live-pass-and-score launch (cdt_sim_score) against the two-launch
path it replaces (cdt_canary_sim, then cdt_drift_score) and the oracle: the
scores, the fp64 sums and the stored activations are bitwise identical."""
import pytest

import oracle
from tests.gpu_util import announce, h_bits, rel_err, require_gpu, to_dev

pytestmark = pytest.mark.gpu

SHAPES = [(4, 8, 16, 256), (3, 5, 7, 264), (2, 3, 41, 1000), (5, 2, 1, 8), (1, 1, 130, 8192),
          (2, 3, 5, 4800), (1, 2, 9, 8000)]
CASES = {
    "gauss_add": dict(sigma_b=1e-3, tamper=1, eps=0.05),
    "t3_flip": dict(benign_dist=1, sigma_b=2e-2, tamper=2, flip_p=0.3),
    "block_scale": dict(benign_mode=1, sigma_b=2e-3, tamper=4, scale=1.05),
    "t3_block_mixed": dict(benign_mode=1, benign_dist=1, sigma_b=1e-2, tamper=7, eps=0.1,
                           flip_p=0.05, scale=1.1),
    "redraw": dict(sigma_b=1e-3, redraw=True),
}


@pytest.fixture(scope="module")
def gpu():
    return require_gpu()


@pytest.mark.parametrize("case", sorted(CASES))
@pytest.mark.parametrize("shape", SHAPES)
def test_fused_equals_two_launches(gpu, case, shape):
    torch, cdt = gpu
    S, C, T, H = shape
    kw = dict(CASES[case])
    eps = kw.pop("eps", 0.0)
    announce(f"sim_score {case} {shape}")
    ref = oracle.ref_synth(S, C, T, H, 2, 0, oracle.outlier_gain(H, max(1, H // 100), 20.0, 2, 0))
    q, m = oracle.ref_stats(ref)
    ts, bs = oracle.block_scales(T, H, q, m, eps, kw.get("sigma_b", 0.0))
    ref_d, ts_d, bs_d = to_dev(torch, ref), to_dev(torch, ts), to_dev(torch, bs)
    common = dict(seed=99, cfg_id=3, mal_mask=(1 << (S // 2)) | 1, bscale=bs_d, tscale=ts_d, **kw)
    h2 = cdt.canary_sim(ref_d, **common)
    nd2 = torch.empty((C, S, 2), dtype=torch.float64, device="cuda")
    s2 = cdt.drift_score(h2, ref_d, num_den=nd2)
    hf = torch.empty_like(h2)
    ndf = torch.empty_like(nd2)
    sf = cdt.sim_score(ref_d, h=hf, num_den=ndf, **common)
    nd0 = torch.empty_like(nd2)
    s0 = cdt.sim_score(ref_d, num_den=nd0, **common)  # no store
    torch.cuda.synchronize()
    assert torch.equal(hf, h2)
    assert torch.equal(sf, s2) and torch.equal(ndf, nd2)
    assert torch.equal(s0, s2) and torch.equal(nd0, nd2)
    # and against the oracle
    want_h = oracle.canary_sim(ref, seed=99, cfg_id=3, mal_mask=(1 << (S // 2)) | 1, bscale=bs,
                               tscale=ts, **kw)
    assert int((h_bits(hf) != want_h).sum()) == 0
    s64, _, _ = oracle.drift_score(want_h, ref)
    assert rel_err(sf.cpu().numpy(), s64) < 1e-5


def test_fused_empty_blocks(gpu):
    torch, cdt = gpu
    announce("sim_score empty")
    ref = torch.empty((3, 2, 0, 16), dtype=torch.float32, device="cuda")
    s = cdt.sim_score(ref, seed=0, cfg_id=0)
    torch.cuda.synchronize()
    assert torch.equal(s, torch.zeros((2, 3), dtype=torch.float32, device="cuda"))
