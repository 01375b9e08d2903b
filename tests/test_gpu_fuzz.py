"""Seeded random cases across the whole parameter space, each against the oracle.

Each case draws a shape (B, V), dtype, seeding, window width, gamma, delta, 1/T, row
padding and an unaligned row start, then checks the watermark (bit for bit), greedy
decoding and sampling (tokens and value bits), the row split into two vocabulary
shards at a random column, and detection with lengths and the repeat rule.  The cases
are fixed by the seed, so a failure names a reproducible case.
"""
import numpy as np
import pytest

import oracle
import workloads
from test_gpu_argmax import assert_argmax_equal
from test_gpu_parity import WIDE, _from_device, _to_device, assert_logits_equal, env, say  # noqa: F401

pytestmark = pytest.mark.gpu

CASES = 150


def draw_case(i):
    rng = np.random.default_rng(7000 + i)
    B = int(rng.integers(1, 10))
    V = int(rng.choice([1, 3, 7, 64, 255, 1000, 2049, int(rng.integers(1, 20000))]))
    dtype = str(rng.choice(["f32", "bf16"]))
    seeding = str(rng.choice(["context", "self_salt"]))
    width = int(rng.choice([1, 1, 2, 4, 8]))
    gamma = float(rng.choice([0.0, 0.25, 0.5, 1.0, rng.random()]))
    delta = float(rng.choice([2.0, -1.5, 0.0, rng.normal() * 4]))
    inv_t = float(rng.choice([1.0, 0.5, 3.0]))
    pad = int(rng.choice([0, 0, 3, 8]))
    offset = int(rng.choice([0, 0, 1]))
    return rng, B, V, dtype, seeding, width, gamma, delta, inv_t, pad, offset


def laid_out(env, x, pad, offset):
    torch, _, dev = env
    B, V = x.shape
    stride = V + pad
    base = np.zeros(offset + B * stride + 8, dtype=x.dtype)
    np.lib.stride_tricks.as_strided(base[offset:], shape=(B, V),
                                    strides=(stride * x.itemsize, x.itemsize))[...] = x
    tb = _to_device(torch, dev, base)
    return tb[offset:offset + B * stride].view(B, stride)[:, :V]


@pytest.mark.parametrize("i", range(CASES))
def test_random_case(env, i):
    torch, sbw, dev = env
    rng, B, V, dtype, seeding, width, gamma, delta, inv_t, pad, offset = draw_case(i)
    say(f"fuzz {i}: B={B} V={V} {dtype} {seeding} h={width} gamma={gamma:.3f} "
        f"delta={delta:.3f} inv_t={inv_t} pad={pad} offset={offset}")
    x = (rng.standard_normal((B, V)) * 3).astype(np.float32)
    x[rng.random((B, V)) < 0.01] = np.float32(rng.choice([np.inf, -np.inf, np.nan, 0.0, -0.0]))
    if dtype == "bf16":
        x = workloads.f32_to_bf16_bits(x)
    ctx = workloads.context_tokens(B, width, max(V, 2), rng)
    c = torch.from_numpy(np.ascontiguousarray(ctx, dtype=np.int32)).to(dev)

    t = laid_out(env, x, pad, offset)
    sbw.watermark(t, c, WIDE, gamma, delta, seeding)
    torch.cuda.synchronize()
    assert_logits_equal(_from_device(torch, t).copy(),
                        oracle.watermark_w(x, ctx, WIDE, gamma, delta, seeding), f"case {i}")

    if V > 1:                                  # the same row as two vocabulary shards
        cut = int(rng.integers(1, V))
        t = laid_out(env, x, pad, offset)
        sbw.watermark_shard(t[:, :cut], c, 0, WIDE, gamma, delta, seeding)
        sbw.watermark_shard(t[:, cut:], c, cut, WIDE, gamma, delta, seeding)
        torch.cuda.synchronize()
        assert_logits_equal(_from_device(torch, t).copy(),
                            oracle.watermark_w(x, ctx, WIDE, gamma, delta, seeding),
                            f"case {i} shards at {cut}")

    t = laid_out(env, x, pad, offset)
    tok, val = sbw.watermark_argmax(t, c, WIDE, gamma, delta, seeding)
    assert_argmax_equal((tok.cpu().numpy(), val.cpu().numpy()),
                        oracle.watermark_argmax(x, ctx, WIDE, gamma, delta, seeding), f"case {i}")
    seeds = rng.integers(0, 2**63, B, dtype=np.int64).astype(np.uint64)
    s_dev = torch.from_numpy(seeds.view(np.int64)).to(dev)
    tok, sc = sbw.watermark_sample(t, c, WIDE, gamma, delta, s_dev, seeding, inv_t)
    assert_argmax_equal((tok.cpu().numpy(), sc.cpu().numpy()),
                        oracle.watermark_sample(x, ctx, WIDE, gamma, delta, seeding, seeds, inv_t),
                        f"case {i}")

    if 0.0 < gamma < 1.0:
        N, L = int(rng.integers(1, 20)), int(rng.integers(0, 700))
        tokens = workloads.uniform_tokens(N, L, max(V, 2), rng)
        if N > 1 and L > 4:
            tokens[1, L // 2:] = tokens[1, :L - L // 2]          # a repeated stretch
        lens = rng.integers(-3, L + 5, N).astype(np.int32)
        td = torch.from_numpy(tokens).to(dev)
        ld = torch.from_numpy(lens).to(dev)
        for rule in (False, True):
            if rule and L - width > 4096:
                continue
            counts, scored, z = sbw.detect_ex(td, WIDE, gamma, seeding, width=width, lengths=ld,
                                              ignore_repeated=rule)
            ec, es, ez = oracle.detect_ex(tokens, width, WIDE, gamma, seeding, lengths=lens,
                                          ignore_repeated=rule)
            assert np.array_equal(counts.cpu().numpy(), ec), (i, rule)
            assert np.array_equal(scored.cpu().numpy(), es), (i, rule)
            zz = z.cpu().numpy()
            assert np.array_equal(np.isnan(zz), np.isnan(ez)), (i, rule)
            ok = ~np.isnan(ez)
            np.testing.assert_allclose(zz[ok], ez[ok], rtol=1e-6, atol=1e-9)
