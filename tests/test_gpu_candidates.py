"""GPU parity of the candidate-restricted watermark (sbw_watermark_candidates; SBW-ss of
the scheme table, Sec. 4: self-salt of width 4 on the top-40 candidates).

Bit-exact against the oracle (NaN as NaN) over both dtypes, both seedings, widths 1
and 4, candidate counts 1..1024 with repeats (adjacent and not) and ids outside
[0, V), padded rows, gamma = 0 and 1 and delta < 0, graph replay, and the c4 batch
with its top-40 ids at full size; the logits outside the candidates keep their bits.
"""
import numpy as np
import pytest

import oracle
import workloads
from test_gpu_parity import (KEY, WIDE, _from_device, _to_device, assert_logits_equal, env,  # noqa: F401
                             say, special_logits)

pytestmark = pytest.mark.gpu


def topk_ids(x, k):
    xf = (x.astype(np.uint32) << 16).view(np.float32) if x.dtype == np.uint16 else x
    xf = np.where(np.isnan(xf), -np.inf, xf)
    return np.argsort(-xf, axis=1, kind="stable")[:, :k].astype(np.int32)


def noisy_candidates(rng, x, k):
    """top-k ids with repeats and out-of-range ids planted (k total per row)."""
    B, V = x.shape
    c = topk_ids(x, k)
    if k >= 8:
        c[:, 1] = c[:, 0]                       # adjacent repeat
        c[:, k - 1] = c[:, k // 2]              # far repeat
        c[:, 2] = -1
        c[:, 3] = V
        c[:, 4] = 2**31 - 1
    return np.ascontiguousarray(c)


def run_candidates(env, x, cand, ctx, key, gamma, delta, seeding, stride_pad=0):
    torch, sbw, dev = env
    B, V = x.shape
    stride = V + stride_pad
    host = np.zeros((B, stride), dtype=x.dtype)
    host[:, :V] = x
    if stride_pad:
        host[:, V:] = x[:, :stride_pad] if V >= stride_pad else 0
    tb = _to_device(torch, dev, host)
    t = tb[:, :V]
    c = torch.from_numpy(np.ascontiguousarray(cand, dtype=np.int32)).to(dev)
    p = torch.from_numpy(np.ascontiguousarray(ctx, dtype=np.int32)).to(dev)
    sbw.watermark_candidates(t, p, c, key, gamma, delta, seeding)
    torch.cuda.synchronize()
    out = _from_device(torch, tb)
    assert np.array_equal(out[:, V:].view(np.uint8), host[:, V:].view(np.uint8)), "padding written"
    return np.ascontiguousarray(out[:, :V])


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("seeding", ["self_salt", "context"])
@pytest.mark.parametrize("width", [1, 4])
@pytest.mark.parametrize("B,V,k", [(1, 1, 1), (3, 100, 40), (5, 1000, 40), (4, 32000, 257),
                                   (2, 5000, 1024)])
def test_candidates_small(env, dtype, seeding, width, B, V, k):
    rng = np.random.default_rng(150 + width * 7 + B * 13 + k)
    x = special_logits(rng, B, V, dtype)
    cand = noisy_candidates(rng, x, k) if V >= k else rng.integers(-2, V + 2, (B, k)).astype(np.int32)
    ctx = workloads.context_tokens(B, width, max(V, 2), rng)
    for gamma, delta in [(0.25, 2.0), (0.5, -1.5), (1.0, 0.5), (0.0, 3.0)]:
        say(f"candidates {dtype} {seeding} h={width} B={B} V={V} k={k} gamma={gamma}")
        got = run_candidates(env, x, cand, ctx, WIDE, gamma, delta, seeding, stride_pad=3)
        expect = oracle.watermark_candidates(x, cand, ctx, WIDE, gamma, delta, seeding)
        assert_logits_equal(got, expect, f"{dtype}/{seeding}/{B}x{V}/k={k}/{gamma}")


def test_candidates_graph_replay(env):
    torch, sbw, dev = env
    rng = np.random.default_rng(160)
    B, V, k = 32, 20000, 40
    x = rng.standard_normal((B, V)).astype(np.float32)
    cand = noisy_candidates(rng, x, k)
    ctx = workloads.context_tokens(B, 4, V, rng)
    expect = oracle.watermark_candidates(x, cand, ctx, KEY, 0.25, 2.0, "self_salt")
    src = torch.from_numpy(x).to(dev)
    t = src.clone()
    c = torch.from_numpy(cand).to(dev)
    p = torch.from_numpy(ctx).to(dev)
    sbw.watermark_candidates(t, p, c, KEY, 0.25, 2.0, "self_salt")
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    t.copy_(src)
    torch.cuda.synchronize()
    with torch.cuda.graph(g):
        sbw.watermark_candidates(t, p, c, KEY, 0.25, 2.0, "self_salt")
    for replay in range(4):
        t.copy_(src)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert_logits_equal(t.cpu().numpy(), expect, f"replay {replay}")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_candidates_c4_top40_full_size(env, dtype):
    """SBW-ss on the c4 batch: B = 256, V = 152064, top-40 ids, width-4 windows."""
    c = workloads.C4
    x, _ = workloads.watermark_inputs("c4")
    if dtype == "bf16":
        x = workloads.f32_to_bf16_bits(x)
    rng = workloads.rng_for("c4", salt=7)
    ctx = workloads.context_tokens(x.shape[0], 4, c["V"], rng)
    cand = topk_ids(x, 40)
    say(f"candidates c4 top-40 {dtype}")
    got = run_candidates(env, x, cand, ctx, KEY, c["gamma"], c["delta"], "self_salt")
    expect = oracle.watermark_candidates(x, cand, ctx, KEY, c["gamma"], c["delta"], "self_salt")
    assert_logits_equal(got, expect, f"c4 top-40 {dtype}")
    moved = int((got.view(np.uint8) != x.view(np.uint8)).reshape(x.shape[0], -1).any(axis=1).sum())
    assert moved > 0.9 * x.shape[0]      # nearly every row has a green candidate (1 - 0.75^40)
