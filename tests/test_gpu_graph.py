"""HIP graph capture of the library's launches.

The benchmark replays captured launches, so captured watermark and detect calls
must give the eager results on every replay, with eager work and host
synchronisation between replays.  The library records no memset nodes.
"""
import numpy as np
import pytest

import oracle
import workloads

pytestmark = pytest.mark.gpu


def test_graph_replays_match_eager_and_oracle():
    import torch
    import paper_2609_03844_amd as sbw
    dev = torch.device("cuda:0")
    key, gamma, delta = workloads.PAPER_KEY, 0.25, 2.0
    rng = np.random.default_rng(314)
    B, V, N, L = 8, 40003, 64, 300
    x = rng.standard_normal((B, V)).astype(np.float32)
    prev = rng.integers(0, V, B).astype(np.int32)
    tok = rng.integers(0, V, (N, L)).astype(np.int32)
    src = torch.from_numpy(x).to(dev)
    p = torch.from_numpy(prev).to(dev)
    t = torch.from_numpy(tok).to(dev)
    bufs = {s: torch.empty_like(src) for s in ("context", "self_salt")}
    counts = {s: torch.empty(N, dtype=torch.int32, device=dev) for s in bufs}
    zs = {s: torch.empty(N, dtype=torch.float64, device=dev) for s in bufs}

    def work():
        for s in bufs:
            bufs[s].copy_(src)
            sbw.watermark(bufs[s], p, key, gamma, delta, s)
            sbw.detect(t, key, gamma, s, counts=counts[s], z=zs[s])

    expect = {s: (oracle.watermark(x, prev, key, gamma, delta, s), oracle.detect(tok, key, gamma, s))
              for s in bufs}
    work()  # eager warmup
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        work()
    scratch = torch.randn(1 << 20, device=dev)
    for replay in range(4):
        for s in bufs:                      # clobber the outputs between replays
            bufs[s].fill_(float("nan"))
            counts[s].fill_(-1)
            zs[s].fill_(0.0)
        scratch.mul_(1.0001)                # eager work between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for s in bufs:
            got = bufs[s].cpu().numpy()
            assert np.array_equal(got.view(np.uint32), expect[s][0].view(np.uint32)), (replay, s)
            assert np.array_equal(counts[s].cpu().numpy(), expect[s][1][0]), (replay, s)
            np.testing.assert_allclose(zs[s].cpu().numpy(), expect[s][1][1], rtol=1e-6, atol=1e-6)
