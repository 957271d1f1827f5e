"""Canary sharding on one GPU.  A caller that holds canaries [c0, c0 + C')
of a run passes canary_base = c0.  It must get, bit for bit, the whole
run's values for those canaries: references, live activations (with and
without propagation), exact-norm scales, drift scores and per-canary AUROC
counts, also with every slice as one job of the batched launches.  The integer counts of the slices must also add up to the whole
run's.  The whole run is computed both by the oracle and by one unsharded
GPU call.  This checks, on one device, the by-canary split of the detector:
no exchange but one sum of integer counts per configuration."""
import numpy as np
import pytest

import oracle
from tests.gpu_util import announce, h_bits, require_gpu, to_dev

pytestmark = pytest.mark.gpu

# (S, C, T, H, canaries per slice): uneven, single-canary and even splits
SPLITS = [(4, 12, 16, 256, (5, 4, 3)), (3, 7, 9, 64, (1, 6)), (16, 32, 8, 512, (8, 8, 8, 8)),
          (12, 10, 5, 768, (3, 3, 3, 1))]
SEED, REF_ID, CFG = 5, 1, 3


@pytest.fixture(scope="module")
def gpu():
    return require_gpu()


def _slices(parts):
    c0 = 0
    for n in parts:
        yield c0, slice(c0, c0 + n)
        c0 += n


@pytest.mark.parametrize("split", SPLITS, ids=[f"{s[:4]}-{s[4]}" for s in SPLITS])
def test_canary_slices_match_the_whole_run(gpu, split):
    torch, cdt = gpu
    S, C, T, H, parts = split
    assert sum(parts) == C
    announce(f"sharding {split}")
    mal = (1 << (S // 2)) | (1 << (S - 1))
    gain = oracle.outlier_gain(H, max(1, H // 100), 20.0, SEED, REF_ID)
    ref = oracle.ref_synth(S, C, T, H, SEED, REF_ID, gain)
    q, m = oracle.ref_stats(ref)
    ts, bs = oracle.block_scales(T, H, q, m, 0.05, 2e-3)
    kw = dict(seed=SEED, cfg_id=CFG, benign_mode=1, sigma_b=2e-3, mal_mask=mal, tamper=7,
              flip_p=0.1, scale=1.1)
    h_want = oracle.canary_sim(ref, bscale=bs, tscale=ts, **kw)
    chain_want = oracle.canary_sim(ref, bscale=bs, tscale=ts, carry=0.5, **kw)

    gain_d, bs_d, ts_d = (to_dev(torch, x) for x in (gain, bs, ts))
    ref_d = to_dev(torch, ref)
    h_all = cdt.canary_sim(ref_d, bscale=bs_d, tscale=ts_d, **kw)
    score_all = cdt.drift_score(h_all, ref_d)
    exact_all = cdt.tamper_scale_exact(ref_d, 0.05, bscale=bs_d,
                                       **dict(kw, mal_mask=0, tamper=0))
    torch.cuda.synchronize()
    assert int((h_bits(h_all) != h_want).sum()) == 0

    tables, cfgs, off = [], [], 0
    sim_jobs, drift_jobs, batch_out = [], [], []
    for c0, sl in _slices(parts):
        Cp = sl.stop - sl.start
        bs_p = bs_d[:, sl].contiguous()
        ts_p = ts_d[:, sl].contiguous()
        ref_p = cdt.ref_synth(S, Cp, T, H, SEED, REF_ID, gain_d, canary_base=c0)
        h_p = cdt.canary_sim(ref_p, bscale=bs_p, tscale=ts_p, canary_base=c0, **kw)
        chain_p = cdt.canary_sim(ref_p, bscale=bs_p, tscale=ts_p, carry=0.5, canary_base=c0,
                                 **kw)
        score_p = cdt.drift_score(h_p, ref_p)
        fused_p = cdt.sim_score(ref_p, bscale=bs_p, tscale=ts_p, canary_base=c0, **kw)
        exact_p = cdt.tamper_scale_exact(ref_p, 0.05, bscale=bs_p, canary_base=c0,
                                         **dict(kw, mal_mask=0, tamper=0))
        torch.cuda.synchronize()
        where = f"canaries [{c0}, {sl.stop})"
        np.testing.assert_array_equal(ref_p.cpu().numpy().view(np.uint32),
                                      ref[:, sl].view(np.uint32), err_msg=where)
        assert int((h_bits(h_p) != h_want[:, sl]).sum()) == 0, where
        assert int((h_bits(chain_p) != chain_want[:, sl]).sum()) == 0, where
        assert torch.equal(score_p, score_all[sl]), where
        assert torch.equal(fused_p, score_all[sl]), where
        assert torch.equal(exact_p, exact_all[:, sl]), where
        # the slice as one job of the batched launches (its own canary_base)
        hb, sb = torch.empty_like(h_p), torch.empty_like(score_p)
        sim_jobs.append((ref_p, hb, dict(kw, bscale=bs_p, tscale=ts_p, canary_base=c0)))
        drift_jobs.append((hb, ref_p, sb, None))
        batch_out.append((hb, sb, h_want[:, sl], score_all[sl], where))
        tables.append(score_p.reshape(-1))
        cfgs.append((S, Cp, off, mal, CFG, c0))
        off += Cp * S

    # every slice in one batched live pass and one batched Eq. 4
    cdt.canary_sim_batch(sim_jobs)
    cdt.drift_score_batch(drift_jobs)
    torch.cuda.synchronize()
    for hb, sb, h_w, s_w, where in batch_out:
        assert int((h_bits(hb) != h_w).sum()) == 0, "batched " + where
        assert torch.equal(sb, s_w), "batched " + where

    # per-canary counts: slices add up to the whole run, bit for bit
    flags = cdt.AUROC_CONTROL | cdt.AUROC_RANDOM
    whole, _, whole_base = cdt.auroc([(S, C, 0, mal, CFG)], score_all.reshape(-1), seed=SEED,
                                     flags=flags)
    part, _, part_base = cdt.auroc(cfgs, torch.cat(tables), seed=SEED, flags=flags)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(cdt.u64(part).sum(axis=0), cdt.u64(whole)[0])
    np.testing.assert_array_equal(cdt.u64(part_base).sum(axis=0), cdt.u64(whole_base)[0])
    # and the whole run's counts are the oracle's
    want, _ = oracle.auroc_config(score_all.cpu().numpy(), mal, seed=SEED, cfg_id=CFG, flags=1)
    np.testing.assert_array_equal(cdt.u64(whole)[0], want)
    np.testing.assert_array_equal(cdt.u64(whole_base)[0],
                                  oracle.random_baseline(C, S, mal, seed=SEED, cfg_id=CFG))


def test_canary_base_changes_the_draws(gpu):
    """The offset is used: a slice generated without it repeats canary 0's
    draws instead of its own."""
    torch, cdt = gpu
    announce("sharding offset used")
    S, C, T, H = 2, 4, 4, 64
    gain = oracle.outlier_gain(H, 1, 20.0, SEED, REF_ID)
    ref = oracle.ref_synth(S, C, T, H, SEED, REF_ID, gain)
    gain_d = to_dev(torch, gain)
    no_base = cdt.ref_synth(S, 2, T, H, SEED, REF_ID, gain_d).cpu().numpy()
    based = cdt.ref_synth(S, 2, T, H, SEED, REF_ID, gain_d, canary_base=2).cpu().numpy()
    np.testing.assert_array_equal(no_base, ref[:, :2])
    np.testing.assert_array_equal(based, ref[:, 2:])
    assert not np.array_equal(no_base, based)


def test_last_canary_indices(gpu):
    """A slice at the top of the 32-bit canary word (canary_base = 2^32 - 3,
    three canaries, the last one 2^32 - 1): references and live activations
    equal the oracle's blocks generated at those global indices directly."""
    torch, cdt = gpu
    announce("sharding last canary indices")
    S, C, T, H = 4, 3, 6, 128
    c0 = (1 << 32) - C
    gain = oracle.outlier_gain(H, 2, 20.0, SEED, REF_ID)
    ref_d = cdt.ref_synth(S, C, T, H, SEED, REF_ID, to_dev(torch, gain), canary_base=c0)
    mal = 1 << 2
    ts = np.full((S, C), 0.03, np.float32)
    kw = dict(seed=SEED, cfg_id=CFG, sigma_b=1e-2, mal_mask=mal, tamper=3, flip_p=0.2)
    h_d = cdt.canary_sim(ref_d, tscale=to_dev(torch, ts), canary_base=c0, **kw)
    torch.cuda.synchronize()
    ref, h = ref_d.cpu().numpy(), h_bits(h_d)
    for s in range(S):
        for c in range(C):
            a = oracle.ref_block(s, c0 + c, T, H, SEED, REF_ID, gain)
            np.testing.assert_array_equal(ref[s, c], a, err_msg=f"ref block ({s}, {c0 + c})")
            want = oracle.sim_block(s, c0 + c, a, seed=SEED, cfg_id=CFG, sigma_b=1e-2,
                                    malicious=bool((mal >> s) & 1), tamper=3, tscale=0.03,
                                    flip_p=0.2)
            assert int((h[s, c] != want).sum()) == 0, f"live block ({s}, {c0 + c})"
    # one canary further would leave the counter word
    with pytest.raises(RuntimeError):
        cdt.ref_synth(S, C + 1, T, H, SEED, REF_ID, to_dev(torch, gain), canary_base=c0)


def test_largest_seed_and_configuration_id(gpu):
    """Counter and key words at their maxima: seed 2^64 - 1 (both key words
    all ones) and cfg_id 2^24 - 1 (the 24-bit id field of the stream word),
    for the live pass, the control and the random baseline."""
    torch, cdt = gpu
    announce("largest seed and cfg_id")
    S, C, T, H = 5, 6, 4, 64
    seed, cid = (1 << 64) - 1, (1 << 24) - 1
    gain = oracle.outlier_gain(H, 1, 20.0, seed, REF_ID)
    ref = oracle.ref_synth(S, C, T, H, seed, REF_ID, gain)
    ts = np.full((S, C), 0.05, np.float32)
    kw = dict(seed=seed, cfg_id=cid, sigma_b=2e-2, mal_mask=1 << 2, tamper=3, flip_p=0.3)
    h_d = cdt.canary_sim(to_dev(torch, ref), tscale=to_dev(torch, ts), **kw)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(
        cdt.ref_synth(S, C, T, H, seed, REF_ID, to_dev(torch, gain)).cpu().numpy(), ref)
    want = oracle.canary_sim(ref, tscale=ts, **kw)
    assert int((h_bits(h_d) != want).sum()) == 0
    score = cdt.drift_score(h_d, to_dev(torch, ref))
    counts, _, base = cdt.auroc([(S, C, 0, 1 << 2, cid)], score.view(-1), seed=seed,
                                flags=cdt.AUROC_CONTROL | cdt.AUROC_RANDOM)
    torch.cuda.synchronize()
    c_o, _ = oracle.auroc_config(score.cpu().numpy(), 1 << 2, seed=seed, cfg_id=cid, flags=1)
    np.testing.assert_array_equal(cdt.u64(counts)[0], c_o)
    np.testing.assert_array_equal(cdt.u64(base)[0],
                                  oracle.random_baseline(C, S, 1 << 2, seed=seed, cfg_id=cid))
