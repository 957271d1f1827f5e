"""The detector as a fixed pipeline for repeated scoring: the AUROC table is
uploaded once (cdt_auroc_upload), and each scoring pass only launches
kernels (cdt_auroc_launch).  That lets a stream capture record a whole
step, the live pass, Eq. 4 and Eqs. 5-6, into a HIP graph for replay.

Checked through the C ABI:
- upload + launch gives bitwise the counts of cdt_auroc and of the oracle;
- the kernels' own bounds checks mark a configuration that a launch's score
  array does not cover, and leave the others exact;
- a captured step, replayed several times with new references copied in
  and eager work in between, equals the eager step every time.
"""
import numpy as np
import pytest

import oracle
from paper_2607_19490_amd import inputs
from tests.gpu_util import announce, h_bits, require_gpu, to_dev
from tests.test_gpu_kernels import _auroc_batch

pytestmark = pytest.mark.gpu

ALL = 1 | 2 | 8  # control, pooled, random baseline
BAD = np.uint64(2**64 - 1)


@pytest.fixture(scope="module")
def gpu():
    return require_gpu()


def test_upload_launch_equals_auroc(gpu):
    torch, cdt = gpu
    announce("auroc upload + launch")
    tables, cfgs = _auroc_batch()
    flat = to_dev(torch, np.concatenate([t.ravel() for t in tables]).astype(np.float32))
    want = cdt.auroc(cfgs, flat, seed=42, flags=ALL)
    table, n = cdt.auroc_upload(cfgs, flat.numel(), flags=ALL)
    got = cdt.auroc_launch(table, n, flat, seed=42, flags=ALL)
    again = cdt.auroc_launch(table, n, flat, seed=42, flags=ALL)
    torch.cuda.synchronize()
    for w, g, a in zip(want, got, again):
        np.testing.assert_array_equal(cdt.u64(g), cdt.u64(w))
        np.testing.assert_array_equal(cdt.u64(a), cdt.u64(w))
    for k, (t, (S, C, off, mask, cid)) in enumerate(zip(tables, cfgs)):
        c_o, p_o = oracle.auroc_config(t, mask, seed=42, cfg_id=cid, flags=3)
        np.testing.assert_array_equal(cdt.u64(got[0])[k], c_o)
        np.testing.assert_array_equal(cdt.u64(got[1])[k], p_o)


def test_upload_from_pinned_memory_is_reusable_at_return(gpu):
    """The table is taken from the caller during the call, also when it sits
    in pinned host memory (where a device copy could still be reading it
    after the call): overwriting it right after cdt_auroc_upload and
    cdt_auroc return, before the stream has run, changes nothing."""
    import ctypes
    torch, cdt = gpu
    announce("auroc upload from pinned host memory")
    tables, cfgs = _auroc_batch()
    flat = to_dev(torch, np.concatenate([t.ravel() for t in tables]).astype(np.float32))
    want = cdt.auroc(cfgs, flat, seed=7, flags=ALL)
    arr, n = cdt.auroc_cfg_array(cfgs)
    nbytes = ctypes.sizeof(arr)
    pinned = torch.empty(nbytes, dtype=torch.uint8, pin_memory=True)
    ctypes.memmove(pinned.data_ptr(), ctypes.addressof(arr), nbytes)
    cfg_ptr = ctypes.cast(pinned.data_ptr(), ctypes.POINTER(cdt.AurocCfg))
    L, stream = cdt.lib(), torch.cuda.current_stream().cuda_stream
    # keep the stream busy so that an asynchronous read of `pinned` would
    # still be pending when it is overwritten
    busy = torch.empty(1 << 26, dtype=torch.float32, device="cuda")
    busy.uniform_()
    for _ in range(4):
        busy.mul_(1.0001)
    table = torch.empty(max(16, L.cdt_auroc_workspace_bytes(n)), dtype=torch.uint8, device="cuda")
    assert L.cdt_auroc_upload(n, cfg_ptr, flat.numel(), ALL, table.data_ptr(), table.numel(),
                              stream) == 0
    pinned.fill_(0xFF)  # S = C = 2^32 - 1 everywhere: never a valid table
    got = cdt.auroc_launch(table, n, flat, seed=7, flags=ALL)
    ctypes.memmove(pinned.data_ptr(), ctypes.addressof(arr), nbytes)
    ws = torch.empty(max(16, L.cdt_auroc_workspace_bytes(n)), dtype=torch.uint8, device="cuda")
    counts = torch.empty((n, 6), dtype=torch.int64, device="cuda")
    pooled = torch.empty((n, 3), dtype=torch.int64, device="cuda")
    base = torch.empty((n, 3), dtype=torch.int64, device="cuda")
    assert L.cdt_auroc(n, cfg_ptr, flat.data_ptr(), flat.numel(), 7, ALL, counts.data_ptr(),
                       pooled.data_ptr(), base.data_ptr(), ws.data_ptr(), ws.numel(),
                       stream) == 0
    pinned.fill_(0xFF)
    torch.cuda.synchronize()
    for w, g, d in zip(want, got, (counts, pooled, base)):
        np.testing.assert_array_equal(cdt.u64(g), cdt.u64(w))
        np.testing.assert_array_equal(cdt.u64(d), cdt.u64(w))


def test_launch_bounds_checks(gpu):
    """A table uploaded for N scores, launched with a score array that claims
    fewer: configurations past the claim get all-ones counts; the others are
    exact.  Pooled ranking asked of a configuration beyond the LDS sort's
    16384 scores (uploaded without the pooled flag) is marked the same way.
    The score buffer itself always holds all N scores."""
    torch, cdt = gpu
    announce("auroc launch bounds checks")
    small = inputs.scores(10, 8, seed=1, mal=(3,), gap=0.2)
    big = inputs.scores(300, 64, seed=2, mal=(9,), gap=0.2)  # 19200 scores
    cfgs = [(8, 10, 0, 1 << 3, 1), (64, 300, small.size, 1 << 9, 2)]
    flat = to_dev(torch, np.concatenate([small.ravel(), big.ravel()]).astype(np.float32))
    table, n = cdt.auroc_upload(cfgs, flat.numel(), flags=1 | 8)
    # the whole array but a claim that ends inside the second table
    counts, _, base = cdt.auroc_launch(table, n, flat[: small.size + 100], seed=3, flags=1 | 8)
    # pooled ranking on the full array: the second configuration is too large
    counts2, pooled2, _ = cdt.auroc_launch(table, n, flat, seed=3, flags=1 | 2)
    torch.cuda.synchronize()
    c_o, p_o = oracle.auroc_config(small, 1 << 3, seed=3, cfg_id=1, flags=3)
    np.testing.assert_array_equal(cdt.u64(counts)[0], c_o)
    np.testing.assert_array_equal(cdt.u64(base)[0],
                                  oracle.random_baseline(10, 8, 1 << 3, seed=3, cfg_id=1))
    assert np.all(cdt.u64(counts)[1] == BAD) and np.all(cdt.u64(base)[1] == BAD)
    np.testing.assert_array_equal(cdt.u64(pooled2)[0], p_o)
    assert np.all(cdt.u64(pooled2)[1] == BAD)
    c_big, _ = oracle.auroc_config(big, 1 << 9, seed=3, cfg_id=2, flags=1)
    np.testing.assert_array_equal(cdt.u64(counts2)[1], c_big)


def _step(cdt, ref, h, score, ws, table, n_cfg, counts, pooled, kw):
    cdt.canary_sim(ref, out=h, **kw)
    cdt.drift_score(h, ref, out=score, ws=ws)
    cdt.auroc_launch(table, n_cfg, score.view(-1), seed=kw["seed"], flags=1 | 2,
                     counts=counts, pooled=pooled)


@pytest.mark.parametrize("shape", [(4, 8, 16, 256), (12, 10, 48, 768)])
def test_captured_step_replays_exactly(gpu, shape):
    torch, cdt = gpu
    S, C, T, H = shape
    announce(f"graph capture {shape}")
    mal = 1 << (S // 2)
    kw = dict(seed=5, cfg_id=2, sigma_b=1e-3, mal_mask=mal, tamper=1)
    refs = [oracle.ref_synth(S, C, T, H, 5, k, np.ones(H, np.float32)) for k in range(3)]
    ref = to_dev(torch, refs[0])
    ts = torch.full((S, C), 0.05, dtype=torch.float32, device="cuda")
    kw["tscale"] = ts
    h = torch.empty((S, C, T, H), dtype=torch.float16, device="cuda")
    score = torch.empty((C, S), dtype=torch.float32, device="cuda")
    ws = cdt.workspace(S, C, T, H, ref)
    table, n = cdt.auroc_upload([(S, C, 0, mal, 2)], C * S, flags=1 | 2)
    counts = torch.empty((1, 6), dtype=torch.int64, device="cuda")
    pooled = torch.empty((1, 3), dtype=torch.int64, device="cuda")
    torch.cuda.synchronize()

    # eager results for each reference set
    want = []
    for r in refs:
        ref.copy_(to_dev(torch, r))
        _step(cdt, ref, h, score, ws, table, n, counts, pooled, kw)
        torch.cuda.synchronize()
        want.append((h_bits(h).copy(), score.cpu().numpy().copy(), cdt.u64(counts).copy(),
                     cdt.u64(pooled).copy()))

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):  # warm-up on the capture stream
        _step(cdt, ref, h, score, ws, table, n, counts, pooled, kw)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        _step(cdt, ref, h, score, ws, table, n, counts, pooled, kw)
    torch.cuda.synchronize()

    for rep in range(2):
        for k, r in enumerate(refs):
            ref.copy_(to_dev(torch, r))
            h.zero_()
            score.fill_(-1.0)  # eager work between replays
            torch.cuda.synchronize()
            graph.replay()
            torch.cuda.synchronize()
            wh, ws_, wc, wp = want[k]
            assert int((h_bits(h) != wh).sum()) == 0, (rep, k)
            np.testing.assert_array_equal(score.cpu().numpy(), ws_)
            np.testing.assert_array_equal(cdt.u64(counts), wc)
            np.testing.assert_array_equal(cdt.u64(pooled), wp)
    # and the eager result is the oracle's
    h_o = oracle.canary_sim(refs[-1], seed=5, cfg_id=2, sigma_b=1e-3, mal_mask=mal, tamper=1,
                            tscale=np.full((S, C), 0.05, np.float32))
    np.testing.assert_array_equal(want[-1][0], h_o)
    del graph
