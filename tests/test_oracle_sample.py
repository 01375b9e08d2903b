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


def test_gumbel_noise_is_standard_gumbel():
    v = np.arange(400000, dtype=np.uint32)
    g = oracle.gumbel_many(v, 0x5EED).astype(np.float64)
    n = g.size
    assert abs(g.mean() - np.euler_gamma) < 5 * math.sqrt(math.pi ** 2 / 6 / n)
    assert abs(g.var() - math.pi ** 2 / 6) < 0.03
    assert stats.kstest(g, "gumbel_r").pvalue > 1e-3
    # another seed gives other noise
    assert np.mean(oracle.gumbel_many(v[:1000], 0x5EED) == oracle.gumbel_many(v[:1000], 0x5EEE)) < 0.01


@pytest.mark.parametrize("seeding", ["context", "self_salt"])
def test_samples_follow_the_watermarked_softmax(seeding):
    rng = np.random.default_rng(310)
    V, B, inv_t = 6, 60000, 0.7
    row = np.array([1.0, 0.2, -0.5, 2.0, 0.0, 1.5], dtype=np.float32)
    x = np.tile(row, (B, 1))
    ctx = np.full((B, 4), 17, dtype=np.int32)            # one context: one green list
    wm = oracle.watermark_w(row[None, :], ctx[:1], KEY, 0.5, 1.0, seeding)[0].astype(np.float64)
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
