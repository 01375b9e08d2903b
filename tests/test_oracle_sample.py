"""Pins of the oracle's Gumbel-max sampler of the watermarked distribution.

The fp32 logarithm against libm in double; the noise against the standard Gumbel
law (mean = Euler's constant, variance = pi^2/6, Kolmogorov-Smirnov); its range
over every one of the 2^23 values u can take (the bounds a sampling pass may use to
skip tokens that cannot win); the sampled tokens against softmax of the watermarked
logits (chi-square over 60000 draws); greedy decoding as the temperature goes to 0;
NaN handling as for the argmax.
"""
import math

import numpy as np
import pytest
from scipy import stats

import oracle
import workloads

KEY = oracle.PAPER_KEY
GUMBEL_LO, GUMBEL_HI = -3.0, 17.0   # the bounds a sampling pass may rely on


def test_sample_log_matches_libm():
    rng = np.random.default_rng(300)
    x = np.concatenate([np.exp(rng.uniform(math.log(1e-8), math.log(20.0), 200000)),
                        1.0 + rng.uniform(-1e-3, 1e-3, 20000), [1.0, 2.0, 0.5, 1.41421356, 1.4142137]])
    x = x.astype(np.float32)
    got = oracle.sample_log(x).astype(np.float64)
    exact = np.log(x.astype(np.float64))
    err = np.abs(got - exact)
    # a few ulp of the result, or a few 1e-8 where log x is near 0
    assert np.all(err <= np.maximum(4 * np.spacing(np.abs(exact).astype(np.float32)), 5e-8)), err.max()
    assert oracle.sample_log(np.float32([1.0]))[0] == 0.0


def test_gumbel_range_over_every_u():
    # u = (k + 1/2) * 2^-23 for every 23-bit k: the noise's full range
    k = np.arange(1 << 23, dtype=np.float32)
    u = (k + np.float32(0.5)) * np.float32(2.0 ** -23)
    assert u.min() > 0 and u.max() < 1
    g = -oracle.sample_log(-oracle.sample_log(u))
    assert np.all(np.isfinite(g))
    assert GUMBEL_LO < g.min() < -2.8 and 16.6 < g.max() < GUMBEL_HI
    # u -> G is increasing, so the range is reached at the ends
    assert g[0] == g.min() and g[-1] == g.max()


def test_noise_of_every_draw():
    """Over all 2^23 values of the draw's top 23 bits (and random low bits, which must
    not matter): finite, inside the range above, non-decreasing, and at the middle draw
    (u just above 1/2) equal to -log(log 2) to within the log's rounding."""
    rng = np.random.default_rng(301)
    k = np.arange(1 << 23, dtype=np.uint32)
    g = oracle.gumbel_of_draws(k << np.uint32(9)).astype(np.float64)
    assert np.all(np.isfinite(g))
    assert -2.8116 < g.min() < -2.8114 and 16.6355 < g.max() < 16.6356
    assert np.all(np.diff(g) >= 0)
    assert abs(g[1 << 22] - (-math.log(math.log(2.0)))) < 1e-6
    low = rng.integers(0, 512, 1 << 16, dtype=np.uint32)
    sel = rng.integers(0, 1 << 23, 1 << 16, dtype=np.uint32)
    assert np.array_equal(oracle.gumbel_of_draws((sel << np.uint32(9)) | low), g[sel].astype(np.float32))


def test_noise_of_a_token_is_its_cbrng_draw():
    """The noise of token v under seed r is the noise of CBRNG(v, r), the stream the
    green lists use (pinned against Philox test vectors and two engines)."""
    v = np.arange(20000, dtype=np.uint32)
    for seed in (0xC0FFEE, 2**64 - 1, 15485863):
        x = oracle.cbrng_many(v, seed).astype(np.uint32)
        assert np.array_equal(oracle.gumbel_many(v, seed).view(np.uint32),
                              oracle.gumbel_of_draws(x).view(np.uint32))


def test_gumbel_noise_is_standard_gumbel():
    v = np.arange(400000, dtype=np.uint32)
    g = oracle.gumbel_many(v, 0x5EED).astype(np.float64)
    n = g.size
    assert abs(g.mean() - np.euler_gamma) < 5 * math.sqrt(math.pi ** 2 / 6 / n)
    assert abs(g.var() - math.pi ** 2 / 6) < 0.03
    assert stats.kstest(g, "gumbel_r").pvalue > 1e-3
    # another seed gives other noise
    assert np.mean(oracle.gumbel_many(v[:1000], 0x5EED) == oracle.gumbel_many(v[:1000], 0x5EEE)) < 0.01


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("seeding", ["context", "self_salt"])
def test_samples_follow_the_watermarked_softmax(seeding, dtype):
    rng = np.random.default_rng(310)
    V, B, inv_t = 6, 60000, 0.7
    row = np.array([1.0, 0.25, -0.5, 2.0, 0.0, 1.5], dtype=np.float32)   # exact in bf16
    if dtype == "bf16":
        row = workloads.f32_to_bf16_bits(row)
    x = np.tile(row, (B, 1))
    ctx = np.full((B, 4), 17, dtype=np.int32)            # one context: one green list
    wm = oracle.watermark_w(row[None, :], ctx[:1], KEY, 0.5, 1.0, seeding)[0]
    if dtype == "bf16":
        wm = (wm.astype(np.uint32) << np.uint32(16)).view(np.float32)
    wm = wm.astype(np.float64)
    p = np.exp(wm * inv_t - (wm * inv_t).max())
    p /= p.sum()
    seeds = rng.integers(0, 2**63, B, dtype=np.int64).astype(np.uint64)
    tok, score = oracle.watermark_sample(x, ctx, KEY, 0.5, 1.0, seeding, seeds, inv_t)
    counts = np.bincount(tok, minlength=V)
    assert stats.chisquare(counts, p * B).pvalue > 1e-4
    # the score is the winner's perturbed logit
    g = oracle.gumbel_many(tok.astype(np.uint32), seeds)
    np.testing.assert_array_equal(score, (wm[tok].astype(np.float32) * np.float32(inv_t)) + g)


def test_low_temperature_is_greedy_and_nan_wins():
    rng = np.random.default_rng(320)
    B, V = 8, 3001
    x = rng.standard_normal((B, V)).astype(np.float32)
    ctx = workloads.context_tokens(B, 1, V, rng)
    seeds = rng.integers(0, 2**63, B, dtype=np.int64).astype(np.uint64)
    greedy, _ = oracle.watermark_argmax(x, ctx, KEY, 0.25, 2.0, "self_salt")
    tok, _ = oracle.watermark_sample(x, ctx, KEY, 0.25, 2.0, "self_salt", seeds, 1e6)
    assert np.array_equal(tok, greedy)
    x[3, 100] = np.nan
    x[3, 2000] = np.nan
    tok, score = oracle.watermark_sample(x, ctx, KEY, 0.25, 2.0, "self_salt", seeds, 1.0)
    assert tok[3] == 100 and np.isnan(score[3])


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("seeding", ["context", "self_salt"])
@pytest.mark.parametrize("width", [1, 4])
def test_sampler_composes_the_pinned_parts(dtype, seeding, width):
    """Consistency of the two dtype paths: token and score equal
    argmax_v(w_v * (1/T) + G(v, seed)) assembled in numpy from the pinned watermark (w,
    widened exactly from bf16) and the noise, the product and the sum each rounded to
    fp32; ties and NaN as numpy's argmax (first).  (The law of the draw is pinned by
    the chi-square test above.)"""
    rng = np.random.default_rng(330 + width)
    B, V, inv_t = 6, 2500, np.float32(0.8)
    x = rng.standard_normal((B, V)).astype(np.float32) * np.float32(2.0)
    x[1, 17] = np.nan
    x[2, :] = 1.25                                    # all equal before bias and noise
    if dtype == "bf16":
        x = workloads.f32_to_bf16_bits(x)
    ctx = workloads.context_tokens(B, width, V, rng)
    seeds = rng.integers(0, 2**63, B, dtype=np.int64).astype(np.uint64)
    w = oracle.watermark_w(x, ctx, KEY, 0.25, 2.0, seeding)
    if dtype == "bf16":
        w = (w.astype(np.uint32) << np.uint32(16)).view(np.float32)
    v = np.arange(V, dtype=np.uint32)
    g = np.stack([oracle.gumbel_many(v, seeds[b]) for b in range(B)])
    s = (w * inv_t).astype(np.float32) + g
    tok, score = oracle.watermark_sample(x, ctx, KEY, 0.25, 2.0, seeding, seeds, float(inv_t))
    expect = np.argmax(s, axis=1)
    assert np.array_equal(tok, expect)
    sel = s[np.arange(B), expect]
    assert np.array_equal(np.isnan(score), np.isnan(sel))
    ok = ~np.isnan(sel)
    assert np.array_equal(score[ok].view(np.uint32), sel[ok].view(np.uint32))
    assert tok[1] == 17
