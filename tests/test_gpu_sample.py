"""GPU parity of the fused watermark + Gumbel-max sampling (sbw_watermark_sample).

Tokens equal and scores bit-equal (NaN as NaN) to the oracle over ragged shapes,
both dtypes and seedings, windows, temperatures, unaligned rows, graph replay and
the c4 batch; the noise itself bit-exact at 65536 (token, seed) pairs; rows built
against the pass's skip bound (tokens within the noise's range of the maximum).
"""
import numpy as np
import pytest

import oracle
import workloads
from test_gpu_argmax import SMALL_DECODE_GRID, assert_argmax_equal, decode_segment, hard_rows
from test_gpu_parity import KEY, WIDE, _to_device, env, say  # noqa: F401

pytestmark = pytest.mark.gpu


def run_sample(env, x, ctx, seeds, key, gamma, delta, seeding, inv_t, offset=0, stride_pad=0):
    torch, sbw, dev = env
    B, V = x.shape
    stride = V + stride_pad
    base = np.zeros(offset + B * stride + 8, dtype=x.dtype)
    np.lib.stride_tricks.as_strided(base[offset:], shape=(B, V),
                                    strides=(stride * x.itemsize, x.itemsize))[...] = x
    tb = _to_device(torch, dev, base)
    t = tb[offset:offset + B * stride].view(B, stride)[:, :V]
    c = torch.from_numpy(np.ascontiguousarray(ctx, dtype=np.int32)).to(dev)
    s = torch.from_numpy(np.ascontiguousarray(seeds, dtype=np.uint64).view(np.int64)).to(dev)
    tokens, scores = sbw.watermark_sample(t, c, key, gamma, delta, s, seeding, inv_t)
    torch.cuda.synchronize()
    return tokens.cpu().numpy(), scores.cpu().numpy()


def seeds_for(rng, B):
    return rng.integers(0, 2**63, B, dtype=np.int64).astype(np.uint64) * np.uint64(2) + np.uint64(1)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("seeding", ["context", "self_salt"])
@pytest.mark.parametrize("width", [1, 4])
@pytest.mark.parametrize("B,V", [(1, 1), (4, 7), (5, 1000), (6, 4097), (4, 40001)])
def test_sample_small(env, dtype, seeding, width, B, V):
    rng = np.random.default_rng(400 + width * 3 + B * 11 + V)
    x = hard_rows(rng, B, V, dtype)
    ctx = workloads.context_tokens(B, width, max(V, 2), rng)
    seeds = seeds_for(rng, B)
    for gamma, delta, inv_t in [(0.25, 2.0, 1.0), (0.5, -1.0, 0.37), (1.0, 0.5, 3.0),
                                (0.0, 3.0, 1.0)]:
        say(f"sample {dtype} {seeding} h={width} B={B} V={V} gamma={gamma} inv_t={inv_t}")
        assert_argmax_equal(run_sample(env, x, ctx, seeds, WIDE, gamma, delta, seeding, inv_t),
                            oracle.watermark_sample(x, ctx, WIDE, gamma, delta, seeding, seeds, inv_t),
                            f"{dtype}/{seeding}/{B}x{V}/{gamma}")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("seeding", ["context", "self_salt"])
@pytest.mark.parametrize("offset,stride_pad", [(1, 0), (0, 3), (0, 7)])   # 9008: aligned in both dtypes
def test_sample_layouts(env, dtype, seeding, offset, stride_pad):
    rng = np.random.default_rng(410 + offset + stride_pad)
    B, V = 5, 9001
    x = hard_rows(rng, B, V, dtype)
    prev = rng.integers(0, V, B).astype(np.int32)
    seeds = seeds_for(rng, B)
    say(f"sample layout {dtype} {seeding} offset={offset} pad={stride_pad}")
    assert_argmax_equal(run_sample(env, x, prev, seeds, KEY, 0.25, 2.0, seeding, 1.0, offset, stride_pad),
                        oracle.watermark_sample(x, prev, KEY, 0.25, 2.0, seeding, seeds, 1.0))


def test_noise_bit_exact(env):
    """One finite logit per row: the score is that logit times 1/T plus its noise."""
    rng = np.random.default_rng(420)
    B, V = 65536, 64
    x = np.full((B, V), -np.inf, dtype=np.float32)
    idx = np.arange(B) % V
    x[np.arange(B), idx] = rng.standard_normal(B).astype(np.float32)
    prev = rng.integers(0, V, B).astype(np.int32)
    seeds = seeds_for(rng, B)
    say("sample noise bit-exact")
    tok, score = run_sample(env, x, prev, seeds, KEY, 0.0, 1.0, "context", 1.0)
    assert np.array_equal(tok, idx)
    expect = x[np.arange(B), idx] + oracle.gumbel_many(idx.astype(np.uint32), seeds)
    assert np.array_equal(score.view(np.uint32), expect.view(np.uint32))


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("seeding", ["context", "self_salt"])
def test_sample_skip_bound_edges(env, dtype, seeding):
    """A spike of 30 and tokens 19-21 below it: with noise in (-2.81, 16.64) some of
    them can still win and some cannot, so the skip test decides at its margin."""
    rng = np.random.default_rng(430)
    B, V = 512, 40001
    x = (0.05 * rng.standard_normal((B, V))).astype(np.float32)
    x[:, 777] = 30.0
    x[:, 100:V:97] = (30.0 - rng.uniform(19.0, 21.0, (B, len(range(100, V, 97))))).astype(np.float32)
    x[:5, 3000] = np.nan
    if dtype == "bf16":
        x = workloads.f32_to_bf16_bits(x)
    ctx = workloads.context_tokens(B, 4, V, rng)
    seeds = seeds_for(rng, B)
    for gamma, delta, inv_t in [(0.5, 2.0, 1.0), (0.5, -1.0, 1.0), (0.25, 2.0, 1.3)]:
        say(f"sample bound edges {dtype} {seeding} gamma={gamma} delta={delta} inv_t={inv_t}")
        got = run_sample(env, x, ctx, seeds, WIDE, gamma, delta, seeding, inv_t)
        expect = oracle.watermark_sample(x, ctx, WIDE, gamma, delta, seeding, seeds, inv_t)
        assert_argmax_equal(got, expect, f"{dtype}/{seeding}/{gamma}/{delta}")
        assert (expect[0] != 777).sum() > 0       # the spike does not always win


def test_sample_graph_replay(env):
    torch, sbw, dev = env
    rng = np.random.default_rng(440)
    B, V = 16, 50003
    x = rng.standard_normal((B, V)).astype(np.float32)
    ctx = workloads.context_tokens(B, 4, V, rng)
    seeds = seeds_for(rng, B)
    expect = oracle.watermark_sample(x, ctx, KEY, 0.25, 2.0, "self_salt", seeds, 1.0)
    t = torch.from_numpy(x).to(dev)
    c = torch.from_numpy(ctx).to(dev)
    s = torch.from_numpy(seeds.view(np.int64)).to(dev)
    tokens = torch.empty(B, dtype=torch.int32, device=dev)
    scores = torch.empty(B, dtype=torch.float32, device=dev)
    ws = torch.empty(sbw.argmax_workspace_size(B, V), dtype=torch.int64, device=dev)
    sbw.watermark_sample(t, c, KEY, 0.25, 2.0, s, "self_salt", 1.0, tokens=tokens, scores=scores,
                         workspace=ws)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        sbw.watermark_sample(t, c, KEY, 0.25, 2.0, s, "self_salt", 1.0, tokens=tokens,
                             scores=scores, workspace=ws)
    for replay in range(4):
        tokens.fill_(-7); scores.fill_(0.0); ws.fill_(123)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert_argmax_equal((tokens.cpu().numpy(), scores.cpu().numpy()), expect, f"replay {replay}")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("seeding", ["context", "self_salt"])
def test_sample_c4_full_size(env, seeding, dtype):
    c = workloads.C4
    x, prev = workloads.watermark_inputs("c4")
    if dtype == "bf16":
        x = workloads.f32_to_bf16_bits(x)
    seeds = seeds_for(workloads.rng_for("c4", salt=11), x.shape[0])
    say(f"sample c4 {seeding} {dtype}")
    got = run_sample(env, x, prev, seeds, KEY, c["gamma"], c["delta"], seeding, 1.0)
    expect = oracle.watermark_sample(x, prev, KEY, c["gamma"], c["delta"], seeding, seeds, 1.0)
    assert_argmax_equal(got, expect, f"c4 {seeding} {dtype}")
    green = oracle.is_green_many(KEY, prev, expect[0], c["gamma"], seeding)
    assert green.mean() > 0.5          # the watermark shows in the draws


def queue_rows(rng, V, dtype):
    """Rows where many tokens reach the best score's bound, so a wave's candidate
    queue fills and is scored in several rounds, with ties spread over lanes, waves
    and segments: all +inf, all -inf, all NaN, equal huge logits (the noise rounds
    away, every one of them ties) among small ones, and a row of equal logits."""
    rows = [np.full(V, np.inf, dtype=np.float32), np.full(V, -np.inf, dtype=np.float32),
            np.full(V, np.nan, dtype=np.float32)]
    r = (0.1 * rng.standard_normal(V)).astype(np.float32)
    r[rng.choice(V, 300, replace=False)] = 1e9
    rows.append(r)
    r = np.full(V, -5.0, dtype=np.float32); r[V - 3] = np.nan; r[V // 2:V // 2 + 2000] = 1e9
    rows.append(r)
    rows.append(np.full(V, 0.5, dtype=np.float32))
    x = np.stack(rows)
    return workloads.f32_to_bf16_bits(x) if dtype == "bf16" else x


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("seeding", ["context", "self_salt"])
@pytest.mark.parametrize("V", [20000, 40001])
def test_sample_queue_rounds(env, dtype, seeding, V):
    rng = np.random.default_rng(450 + V)
    x = queue_rows(rng, V, dtype)
    B = x.shape[0]
    ctx = workloads.context_tokens(B, 1, V, rng)[:, 0].copy()
    seeds = seeds_for(rng, B)
    for gamma, delta, inv_t in [(0.25, 2.0, 1.0), (0.5, -1.0, 1e-30), (1.0, 0.5, 1e30)]:
        say(f"sample queue rounds {dtype} {seeding} V={V} gamma={gamma} inv_t={inv_t}")
        assert_argmax_equal(run_sample(env, x, ctx, seeds, WIDE, gamma, delta, seeding, inv_t),
                            oracle.watermark_sample(x, ctx, WIDE, gamma, delta, seeding, seeds, inv_t),
                            f"{dtype}/{seeding}/{V}/{gamma}/{inv_t}")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("seeding", ["context", "self_salt"])
@pytest.mark.parametrize("width", [2, 8])
def test_sample_windows(env, dtype, seeding, width):
    """Windows of 2 and of the longest supported width, 8, on a ragged multi-segment row."""
    rng = np.random.default_rng(460 + width)
    B, V = 5, 30011
    x = hard_rows(rng, B, V, dtype)
    ctx = workloads.context_tokens(B, width, V, rng)
    seeds = seeds_for(rng, B)
    say(f"sample windows {dtype} {seeding} h={width}")
    assert_argmax_equal(run_sample(env, x, ctx, seeds, WIDE, 0.25, 2.0, seeding, 1.0),
                        oracle.watermark_sample(x, ctx, WIDE, 0.25, 2.0, seeding, seeds, 1.0),
                        f"{dtype}/{seeding}/h={width}")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("seeding", ["context", "self_salt"])
def test_sample_both_launch_shapes(env, dtype, seeding):
    """The queue-round rows tiled to 256 rows (the full-width decode kernel: more than
    900 workgroups) and to 8 rows (the half-width kernel for small grids)."""
    rng = np.random.default_rng(470)
    V = 40001
    edge = queue_rows(rng, V, dtype)
    seg = decode_segment(dtype, sample=True)
    for B in (8, 256):
        x = np.concatenate([edge] * (-(-B // edge.shape[0])))[:B].copy()
        ctx = workloads.context_tokens(B, 1, V, rng)[:, 0].copy()
        seeds = seeds_for(rng, B)
        big = B * (-(-V // seg)) >= SMALL_DECODE_GRID
        assert big == (B == 256), (B, seg)         # both launch shapes are exercised
        for gamma, delta, inv_t in [(0.25, 2.0, 1.0), (0.5, -1.0, 0.37)]:
            say(f"sample launch shapes {dtype} {seeding} B={B} gamma={gamma}")
            assert_argmax_equal(run_sample(env, x, ctx, seeds, WIDE, gamma, delta, seeding, inv_t),
                                oracle.watermark_sample(x, ctx, WIDE, gamma, delta, seeding, seeds,
                                                        inv_t),
                                f"{dtype}/{seeding}/B={B}/{gamma}")
