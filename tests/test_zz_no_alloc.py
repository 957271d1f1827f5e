"""cdt_drift_score_noalloc, the entry point for callers that cannot
allocate device memory, against cdt_drift_score (the same Eq. 4 with a
caller workspace) and the CPU oracle, through the C ABI.

Calls run back to back on one GPU: a large multi-chunk shape, then a
smaller ragged one that reuses the library's scratch (its partial sums
must not leak from the first call), then a shape whose blocks are single
chunks (scored directly).  Scores and fp64 sums must equal the workspace
entry point's bit for bit, and the oracle's within 1e-5 relative.  A
stream capture of the call replays exactly, with other calls using the
scratch between replays.
"""
import numpy as np
import pytest

import oracle
from paper_2607_19490_amd import inputs
from tests.gpu_util import announce, rel_err, require_gpu, to_dev

pytestmark = pytest.mark.gpu

DRIFT_RTOL = 1e-5

# (S, C, T, H): 16 chunks per block; 2 chunks per block with a ragged last
# chunk (41000 elements); one chunk per block.
CALLS = [(16, 32, 128, 4096), (3, 5, 41, 1000), (4, 8, 16, 256)]


def test_noalloc_matches_workspace_entry_point():
    torch, cdt = require_gpu()
    for k, shape in enumerate(CALLS):
        S, C, T, H = shape
        announce(f"drift_score_noalloc call {k}: {shape}")
        a = inputs.ref_normal(shape, seed=70 + k, outlier_frac=0.01)
        h = inputs.live_near(a, seed=80 + k, rel=1e-3, flip_frac=0.001)
        ad = to_dev(torch, a)
        hd = to_dev(torch, h).view(torch.float16)
        out = torch.full((C, S), -1.0, dtype=torch.float32, device="cuda")
        nd = torch.full((C, S, 2), -1.0, dtype=torch.float64, device="cuda")
        cdt.drift_score_noalloc(hd, ad, out=out, num_den=nd)
        nd_w = torch.empty_like(nd)
        want = cdt.drift_score(hd, ad, num_den=nd_w)
        torch.cuda.synchronize()
        assert torch.equal(out, want), f"call {k}: scores differ from cdt_drift_score"
        assert torch.equal(nd, nd_w), f"call {k}: sums differ from cdt_drift_score"
        if k == 0:  # oracle on every shard of two canaries of the large call
            for c in (0, C - 1):
                for s in range(S):
                    m_o, _, _ = oracle.drift_block(h[s, c], a[s, c])
                    assert rel_err(out[c, s].item(), m_o) < DRIFT_RTOL, (s, c)
        else:
            s64, _, _ = oracle.drift_score(h, a)
            assert rel_err(out.cpu().numpy(), s64) < DRIFT_RTOL
        del ad, hd


def test_noalloc_rejects_shapes_beyond_its_scratch():
    torch, cdt = require_gpu()
    L = cdt.lib()
    # 16 x 1024 blocks of 64 chunks: 16 MiB of partial sums, above the 8 MiB
    rc = L.cdt_drift_score_noalloc(16, 1024, 256, 8192, None, None, None, None, None)
    assert rc == cdt.ELIMIT and "scratch" in cdt.last_error()
    # a rejected call launches nothing; the next call runs as before
    announce("drift_score_noalloc after a rejection")
    S, C, T, H = 2, 3, 9, 8000
    a = inputs.ref_normal((S, C, T, H), seed=90)
    h = inputs.live_near(a, seed=91, rel=1e-2)
    ad, hd = to_dev(torch, a), to_dev(torch, h).view(torch.float16)
    out = torch.empty((C, S), dtype=torch.float32, device="cuda")
    cdt.drift_score_noalloc(hd, ad, out=out)
    want = cdt.drift_score(hd, ad)
    torch.cuda.synchronize()
    assert torch.equal(out, want)


def test_noalloc_under_graph_capture():
    """The caller it exists for: a stream capture records the no-allocation
    call (kernel launches only), and each replay scores the inputs copied in
    before it, equal to cdt_drift_score's eager result, also after an eager
    call of another shape has overwritten the library's scratch in between."""
    torch, cdt = require_gpu()
    S, C, T, H = 4, 6, 64, 1024  # two chunks per block: the scratch is used
    announce(f"drift_score_noalloc under graph capture {(S, C, T, H)}")
    cases = []
    for k in range(3):
        a = inputs.ref_normal((S, C, T, H), seed=100 + k, outlier_frac=0.01)
        h = inputs.live_near(a, seed=110 + k, rel=1e-3 * (k + 1), flip_frac=0.001)
        cases.append((to_dev(torch, a), to_dev(torch, h).view(torch.float16)))
    ad = torch.empty_like(cases[0][0])
    hd = torch.empty_like(cases[0][1])
    out = torch.empty((C, S), dtype=torch.float32, device="cuda")
    want = [cdt.drift_score(h_, a_) for a_, h_ in cases]
    # another shape's eager call between replays reuses the scratch
    a2 = inputs.ref_normal((3, 5, 41, 1000), seed=120)
    ad2 = to_dev(torch, a2)
    hd2 = to_dev(torch, inputs.live_near(a2, seed=121, rel=1e-2)).view(torch.float16)
    out2 = torch.empty((5, 3), dtype=torch.float32, device="cuda")
    want2 = cdt.drift_score(hd2, ad2)
    torch.cuda.synchronize()

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):  # warm-up on the capture stream
        cdt.drift_score_noalloc(hd, ad, out=out)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        cdt.drift_score_noalloc(hd, ad, out=out)
    torch.cuda.synchronize()
    for rep in range(2):
        for k, (a_, h_) in enumerate(cases):
            ad.copy_(a_)
            hd.copy_(h_)
            out.fill_(-1.0)
            cdt.drift_score_noalloc(hd2, ad2, out=out2)
            torch.cuda.synchronize()
            graph.replay()
            torch.cuda.synchronize()
            assert torch.equal(out, want[k]), (rep, k)
            assert torch.equal(out2, want2), (rep, k)
    del graph
