"""GPU parity when rows (or row groups) outnumber the 65535 workgroups of a grid's y
dimension, so every row-parallel kernel runs its grid-stride loop: many short rows
for the watermark (both seedings; self-salt through the slab kernel with a window of
one token and through the row-group kernel with a window of 4), greedy decoding,
sampling, candidates and both detection kernels."""
import numpy as np
import pytest

import oracle
import workloads
from test_gpu_parity import (KEY, WIDE, _from_device, _to_device, assert_detect_equal,  # noqa: F401
                             assert_logits_equal, env, say)

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("seeding", ["context", "self_salt"])
@pytest.mark.parametrize("B,V", [(70001, 37), (300001, 8)])
def test_watermark_many_rows(env, seeding, B, V):
    torch, sbw, dev = env
    rng = np.random.default_rng(240 + V)
    x = rng.standard_normal((B, V)).astype(np.float32)
    prev = rng.integers(0, 50000, B).astype(np.int32)
    say(f"watermark many rows {seeding} B={B} V={V}")
    t = _to_device(torch, dev, x)
    sbw.watermark(t, torch.from_numpy(prev).to(dev), WIDE, 0.5, 1.5, seeding)
    torch.cuda.synchronize()
    assert_logits_equal(_from_device(torch, t), oracle.watermark(x, prev, WIDE, 0.5, 1.5, seeding))


def test_watermark_window_many_rows(env):
    """Self-salt with a window of 4 keeps one row per workgroup: 70001 aligned rows of
    40 logits run the row-group kernel's grid-stride loop."""
    torch, sbw, dev = env
    rng = np.random.default_rng(245)
    B, V = 70001, 40
    x = rng.standard_normal((B, V)).astype(np.float32)
    ctx = workloads.context_tokens(B, 4, V, rng)
    say(f"watermark many rows, window 4, B={B} V={V}")
    t = _to_device(torch, dev, x)
    sbw.watermark(t, torch.from_numpy(ctx).to(dev), WIDE, 0.5, 1.5, "self_salt")
    torch.cuda.synchronize()
    assert_logits_equal(_from_device(torch, t), oracle.watermark_w(x, ctx, WIDE, 0.5, 1.5, "self_salt"))


@pytest.mark.parametrize("seeding", ["context", "self_salt"])
def test_argmax_and_candidates_many_rows(env, seeding):
    torch, sbw, dev = env
    rng = np.random.default_rng(250)
    B, V = 70001, 40
    x = rng.standard_normal((B, V)).astype(np.float32)
    ctx = workloads.context_tokens(B, 4, V, rng)
    c = torch.from_numpy(ctx).to(dev)
    say(f"argmax many rows {seeding}")
    tok, val = sbw.watermark_argmax(_to_device(torch, dev, x), c, WIDE, 0.5, 1.5, seeding)
    torch.cuda.synchronize()
    et, ev = oracle.watermark_argmax(x, ctx, WIDE, 0.5, 1.5, seeding)
    assert np.array_equal(tok.cpu().numpy(), et) and np.array_equal(val.cpu().numpy(), ev)
    # sampling: the same rows, one noise seed per row
    seeds = rng.integers(0, 2**63, B, dtype=np.int64).astype(np.uint64)
    say(f"sample many rows {seeding}")
    tok, sc = sbw.watermark_sample(_to_device(torch, dev, x), c, WIDE, 0.5, 1.5,
                                   torch.from_numpy(seeds.view(np.int64)).to(dev), seeding, 0.9)
    torch.cuda.synchronize()
    et, es = oracle.watermark_sample(x, ctx, WIDE, 0.5, 1.5, seeding, seeds, 0.9)
    assert np.array_equal(tok.cpu().numpy(), et)
    assert np.array_equal(sc.cpu().numpy().view(np.uint32), es.view(np.uint32))
    # candidates: one workgroup per row, at most 2^20 workgroups
    B, V = 1100001, 8
    x = rng.standard_normal((B, V)).astype(np.float32)
    ctx = workloads.context_tokens(B, 4, V, rng)
    cand = rng.integers(-1, V + 1, (B, 3)).astype(np.int32)
    say(f"candidates many rows {seeding}")
    t = _to_device(torch, dev, x)
    sbw.watermark_candidates(t, torch.from_numpy(ctx).to(dev), torch.from_numpy(cand).to(dev),
                             WIDE, 0.5, 1.5, seeding)
    torch.cuda.synchronize()
    assert_logits_equal(_from_device(torch, t),
                        oracle.watermark_candidates(x, cand, ctx, WIDE, 0.5, 1.5, seeding))


@pytest.mark.parametrize("ignore", [False, True])
def test_detect_many_sequences(env, ignore):
    torch, sbw, dev = env
    rng = np.random.default_rng(260)
    # 4 sequences per workgroup (1 with the repeat rule), at most 2^20 workgroups
    N, L = 4200003, 5
    tok = rng.integers(0, 6, (N, L)).astype(np.int32)
    lengths = rng.integers(0, L + 1, N).astype(np.int32)
    say(f"detect many sequences ignore={ignore}")
    counts, scored, z = sbw.detect_ex(torch.from_numpy(tok).to(dev), KEY, 0.25, "self_salt", width=2,
                                      lengths=torch.from_numpy(lengths).to(dev),
                                      ignore_repeated=ignore)
    torch.cuda.synchronize()
    ec, es, ez = oracle.detect_ex(tok, 2, KEY, 0.25, "self_salt", lengths=lengths,
                                  ignore_repeated=ignore)
    assert np.array_equal(scored.cpu().numpy(), es)
    assert_detect_equal((counts.cpu().numpy(), z.cpu().numpy()), (ec, ez))
