"""GPU parity of the vocabulary-shard calls (sbw_watermark_shard,
sbw_watermark_argmax_shard, sbw_watermark_sample_shard).

A shard holds columns [a, b) of the vocabulary; column c is token a + c.  Checked:
  * the watermarked shards, put side by side, equal the oracle's full rows bit for bit;
  * each shard's greedy token and value, and its sampled token and score, equal the
    best of its slice assembled from the oracle's watermark and noise;
  * the shards' winners, reduced as a tensor-parallel head would (largest value,
    smallest id among equal ones, NaN above all), equal the oracle's full-row decode;
  * shards whose first id is or is not a multiple of 4 (fp32) / 8 (bf16), so both the
    vector and the element kernels run, and ids up to 2^31 - 1;
  * the 8-way split of the 152064-token vocabulary at B = 256, as views of one tensor;
  * detection split along the text, each shard reading a halo of width tokens.
"""
import numpy as np
import pytest

import oracle
import workloads
from test_gpu_argmax import assert_argmax_equal, hard_rows
from test_gpu_parity import WIDE, _from_device, _to_device, assert_logits_equal, env, say  # noqa: F401

pytestmark = pytest.mark.gpu

# Boundaries of a 40001-token vocabulary: shard starts 0, 8192 and 20000 are multiples
# of 8; 24004 is a multiple of 4 only (fp32 vector kernels, bf16 element kernels); 8195
# and 27331 are odd; one shard is 3 tokens long.
BOUNDS = [0, 8192, 8195, 20000, 24004, 27331, 40001]


def widen(w):
    return (w.astype(np.uint32) << np.uint32(16)).view(np.float32) if w.dtype == np.uint16 else w


def shard_tensor(env, x, a, b):
    """Columns [a, b) of x as their own device tensor, rows padded to 16 bytes."""
    torch, _, dev = env
    B = x.shape[0]
    n = b - a
    stride = -(-n // 8) * 8
    buf = np.zeros((B, stride), dtype=x.dtype)
    buf[:, :n] = x[:, a:b]
    return _to_device(torch, dev, buf)[:, :n]


def combine(parts):
    """Row-wise reduction of per-shard (tokens, values), shards in id order."""
    toks = np.stack([p[0] for p in parts])
    vals = np.stack([p[1] for p in parts])
    B = toks.shape[1]
    out_t = np.empty(B, dtype=np.int32)
    out_v = np.empty(B, dtype=np.float32)
    for r in range(B):
        k = 0
        for s in range(1, len(parts)):
            if np.isnan(vals[k, r]):
                break
            if np.isnan(vals[s, r]) or vals[s, r] > vals[k, r]:
                k = s
        out_t[r], out_v[r] = toks[k, r], vals[k, r]
    return out_t, out_v


def slice_best(scores, a):
    """Greedy pick of a slice of per-token scores (first maximum, first NaN)."""
    j = np.argmax(scores, axis=1)
    return (j + a).astype(np.int32), scores[np.arange(scores.shape[0]), j].astype(np.float32)


def seeds_for(rng, B):
    return rng.integers(0, 2**63, B, dtype=np.int64).astype(np.uint64) * np.uint64(2) + np.uint64(1)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("seeding", ["context", "self_salt"])
@pytest.mark.parametrize("width", [1, 4])
def test_watermark_shards_tile_the_row(env, dtype, seeding, width):
    torch, sbw, dev = env
    rng = np.random.default_rng(900 + width)
    B, V = 5, BOUNDS[-1]
    x = hard_rows(rng, B, V, dtype)
    ctx = workloads.context_tokens(B, width, V, rng)
    c = torch.from_numpy(np.ascontiguousarray(ctx, dtype=np.int32)).to(dev)
    for gamma, delta in [(0.25, 2.0), (0.5, -1.5)]:
        expect = oracle.watermark_w(x, ctx, WIDE, gamma, delta, seeding)
        for a, b in zip(BOUNDS[:-1], BOUNDS[1:]):
            say(f"watermark shard {dtype} {seeding} h={width} [{a},{b}) gamma={gamma}")
            t = shard_tensor(env, x, a, b)
            sbw.watermark_shard(t, c, a, WIDE, gamma, delta, seeding)
            assert_logits_equal(_from_device(torch, t), expect[:, a:b],
                                f"{dtype}/{seeding}/[{a},{b})")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("seeding", ["context", "self_salt"])
@pytest.mark.parametrize("width", [1, 4])
def test_decode_shards_reduce_to_the_full_row(env, dtype, seeding, width):
    torch, sbw, dev = env
    rng = np.random.default_rng(910 + width)
    B, V = 6, BOUNDS[-1]
    x = hard_rows(rng, B, V, dtype)
    ctx = workloads.context_tokens(B, width, V, rng)
    seeds = seeds_for(rng, B)
    c = torch.from_numpy(np.ascontiguousarray(ctx, dtype=np.int32)).to(dev)
    s_dev = torch.from_numpy(seeds.view(np.int64)).to(dev)
    v_all = np.arange(V, dtype=np.uint32)
    noise = np.stack([oracle.gumbel_many(v_all, seeds[r]) for r in range(B)])
    for gamma, delta, inv_t in [(0.25, 2.0, 1.0), (0.5, -1.0, 0.37)]:
        w = widen(oracle.watermark_w(x, ctx, WIDE, gamma, delta, seeding))
        with np.errstate(invalid="ignore"):       # the NaN and -inf rows
            sample_scores = (w * np.float32(inv_t)).astype(np.float32) + noise
        greedy_parts, sample_parts = [], []
        for a, b in zip(BOUNDS[:-1], BOUNDS[1:]):
            say(f"decode shard {dtype} {seeding} h={width} [{a},{b}) gamma={gamma}")
            t = shard_tensor(env, x, a, b)
            got = sbw.watermark_argmax_shard(t, c, a, WIDE, gamma, delta, seeding)
            got = (got[0].cpu().numpy(), got[1].cpu().numpy())
            assert_argmax_equal(got, slice_best(w[:, a:b], a), f"greedy [{a},{b})")
            greedy_parts.append(got)
            got = sbw.watermark_sample_shard(t, c, a, WIDE, gamma, delta, s_dev, seeding, inv_t)
            got = (got[0].cpu().numpy(), got[1].cpu().numpy())
            assert_argmax_equal(got, slice_best(sample_scores[:, a:b], a), f"sample [{a},{b})")
            sample_parts.append(got)
        assert_argmax_equal(combine(greedy_parts),
                            oracle.watermark_argmax(x, ctx, WIDE, gamma, delta, seeding), "greedy")
        assert_argmax_equal(combine(sample_parts),
                            oracle.watermark_sample(x, ctx, WIDE, gamma, delta, seeding, seeds,
                                                    inv_t), "sample")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("seeding", ["context", "self_salt"])
@pytest.mark.parametrize("a,n", [((1 << 31) - 40000, 40000), ((1 << 31) - 40003, 40003)])
def test_shards_with_large_ids(env, dtype, seeding, a, n):
    """A shard ending at id 2^31 - 1, its first id a multiple of 8 or not; expected
    values from the oracle's per-token membership, bias and noise at the global ids."""
    torch, sbw, dev = env
    rng = np.random.default_rng(920 + n)
    B, width = 3, 2
    x = hard_rows(rng, B, n, dtype)
    ctx = workloads.context_tokens(B, width, 1 << 30, rng)
    seeds = seeds_for(rng, B)
    ids = np.arange(a, a + n, dtype=np.int64)
    gamma, delta, inv_t = 0.25, 2.0, 0.8
    green = np.stack([oracle.is_green_w_many(WIDE, np.repeat(ctx[r:r + 1], n, axis=0),
                                             ids.astype(np.int32), gamma, seeding)
                      for r in range(B)])
    if dtype == "bf16":
        w = np.where(green, oracle.bias_bf16_many(x, delta), x)
    else:
        w = np.where(green, oracle.bias_f32_many(x, delta), x)
    c = torch.from_numpy(np.ascontiguousarray(ctx, dtype=np.int32)).to(dev)
    say(f"large ids {dtype} {seeding} [{a},{a + n})")
    t = shard_tensor(env, x, 0, n)
    tok, val = sbw.watermark_argmax_shard(t, c, a, WIDE, gamma, delta, seeding)
    assert_argmax_equal((tok.cpu().numpy(), val.cpu().numpy()), slice_best(widen(w), a), "greedy")
    noise = np.stack([oracle.gumbel_many(ids.astype(np.uint32), seeds[r]) for r in range(B)])
    with np.errstate(invalid="ignore"):
        scores = (widen(w) * np.float32(inv_t)).astype(np.float32) + noise
    s_dev = torch.from_numpy(seeds.view(np.int64)).to(dev)
    tok, sc = sbw.watermark_sample_shard(t, c, a, WIDE, gamma, delta, s_dev, seeding, inv_t)
    assert_argmax_equal((tok.cpu().numpy(), sc.cpu().numpy()), slice_best(scores, a), "sample")
    sbw.watermark_shard(t, c, a, WIDE, gamma, delta, seeding)
    assert_logits_equal(_from_device(torch, t), w, "watermark")


@pytest.mark.parametrize("seeding", ["context", "self_salt"])
def test_tensor_parallel_split_of_the_c4_vocabulary(env, seeding):
    """B = 256 rows of the 152064-token vocabulary split 8 ways (19008 tokens per shard,
    views of one fp32 tensor): watermark, greedy and sampling per shard, then the
    reduction, against the oracle's full rows."""
    torch, sbw, dev = env
    rng = np.random.default_rng(930)
    B, V, parts = 256, 152064, 8
    n = V // parts
    x = workloads.logits(B, V, sigma=3.0, rng=rng)
    prev = workloads.prev_tokens(B, V, rng)
    seeds = seeds_for(rng, B)
    gamma, delta = 0.25, 2.0
    c = torch.from_numpy(prev.astype(np.int32)).to(dev)
    s_dev = torch.from_numpy(seeds.view(np.int64)).to(dev)
    full = torch.from_numpy(x).to(dev)
    g_parts, s_parts = [], []
    for k in range(parts):
        say(f"tp8 decode {seeding} shard {k}")
        view = full[:, k * n:(k + 1) * n]
        tok, val = sbw.watermark_argmax_shard(view, c, k * n, WIDE, gamma, delta, seeding)
        g_parts.append((tok.cpu().numpy(), val.cpu().numpy()))
        tok, sc = sbw.watermark_sample_shard(view, c, k * n, WIDE, gamma, delta, s_dev, seeding)
        s_parts.append((tok.cpu().numpy(), sc.cpu().numpy()))
    assert_argmax_equal(combine(g_parts), oracle.watermark_argmax(x, prev, WIDE, gamma, delta,
                                                                  seeding), "greedy")
    assert_argmax_equal(combine(s_parts), oracle.watermark_sample(x, prev, WIDE, gamma, delta,
                                                                  seeding, seeds, 1.0), "sample")
    for k in range(parts):
        say(f"tp8 watermark {seeding} shard {k}")
        sbw.watermark_shard(full[:, k * n:(k + 1) * n], c, k * n, WIDE, gamma, delta, seeding)
    torch.cuda.synchronize()
    assert_logits_equal(full.cpu().numpy(), oracle.watermark(x, prev, WIDE, gamma, delta, seeding),
                        f"tp8 {seeding}")


@pytest.mark.parametrize("seeding", ["context", "self_salt"])
@pytest.mark.parametrize("width", [1, 4])
def test_detection_sharded_along_the_text(env, seeding, width):
    """Positions [a, b) of every text scored on their own, each shard reading the width
    tokens before a as its halo: the shards' green counts and scored positions add up
    to the whole texts' (the oracle's), and z from the sums equals the oracle's z."""
    torch, sbw, dev = env
    rng = np.random.default_rng(940 + width)
    N, L, V, gamma = 64, 1000, 128256, 0.25
    tok = workloads.uniform_tokens(N, L, V, rng)
    td = torch.from_numpy(tok).to(dev)
    cuts = [width, 250, 503, 777, L]
    counts = np.zeros(N, dtype=np.int64)
    scored = np.zeros(N, dtype=np.int64)
    for a, b in zip(cuts[:-1], cuts[1:]):
        say(f"detect shard {seeding} h={width} positions [{a},{b})")
        c, t, _ = sbw.detect_ex(td[:, a - width:b], WIDE, gamma, seeding, width=width)
        counts += c.cpu().numpy()
        scored += t.cpu().numpy()
    ec, ez = oracle.detect_w(tok, width, WIDE, gamma, seeding)
    assert np.array_equal(counts, ec)
    assert np.all(scored == L - width)
    z = (counts - scored * gamma) / np.sqrt(scored * gamma * (1 - gamma))
    np.testing.assert_allclose(z, ez, rtol=1e-6, atol=1e-9)


def test_shard_calls_replay_in_a_graph(env):
    """Two shards watermarked and decoded inside one captured graph: every replay, with
    eager work and the outputs clobbered in between, gives the oracle's results."""
    torch, sbw, dev = env
    rng = np.random.default_rng(950)
    B, V, cut = 8, 40003, 20000
    key, gamma, delta = WIDE, 0.25, 2.0
    x = rng.standard_normal((B, V)).astype(np.float32)
    prev = rng.integers(0, V, B).astype(np.int32)
    seeds = seeds_for(rng, B)
    src = torch.from_numpy(x).to(dev)
    p = torch.from_numpy(prev).to(dev)
    s_dev = torch.from_numpy(seeds.view(np.int64)).to(dev)
    buf = torch.empty_like(src)
    halves = [(0, cut), (cut, V)]
    outs = [(torch.empty(B, dtype=torch.int32, device=dev), torch.empty(B, device=dev),
             torch.empty(B, dtype=torch.int32, device=dev), torch.empty(B, device=dev))
            for _ in halves]
    wss = [torch.empty(sbw.argmax_workspace_size(B, b - a), dtype=torch.int64, device=dev)
           for a, b in halves]

    def work():
        for (a, b), o, ws in zip(halves, outs, wss):
            view = src[:, a:b]
            sbw.watermark_argmax_shard(view, p, a, key, gamma, delta, "self_salt", tokens=o[0],
                                       values=o[1], workspace=ws)
            sbw.watermark_sample_shard(view, p, a, key, gamma, delta, s_dev, "self_salt",
                                       tokens=o[2], scores=o[3], workspace=ws)
        buf.copy_(src)
        for a, b in halves:
            sbw.watermark_shard(buf[:, a:b], p, a, key, gamma, delta, "self_salt")

    e_wm = oracle.watermark(x, prev, key, gamma, delta, "self_salt")
    e_am = oracle.watermark_argmax(x, prev, key, gamma, delta, "self_salt")
    e_sm = oracle.watermark_sample(x, prev, key, gamma, delta, "self_salt", seeds, 1.0)
    work()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        work()
    scratch = torch.randn(1 << 20, device=dev)
    for replay in range(4):
        buf.fill_(float("nan"))
        for o in outs:
            o[0].fill_(-1); o[1].fill_(0.0); o[2].fill_(-1); o[3].fill_(0.0)
        scratch.mul_(1.0001)
        torch.cuda.synchronize()
        say(f"shard graph replay {replay}")
        g.replay()
        torch.cuda.synchronize()
        assert np.array_equal(buf.cpu().numpy().view(np.uint32), e_wm.view(np.uint32)), replay
        greedy = combine([(o[0].cpu().numpy(), o[1].cpu().numpy()) for o in outs])
        sample = combine([(o[2].cpu().numpy(), o[3].cpu().numpy()) for o in outs])
        assert_argmax_equal(greedy, e_am, f"greedy replay {replay}")
        assert_argmax_equal(sample, e_sm, f"sample replay {replay}")
