"""Pins of the oracle's context-width-h definitions (SBW-4, SBW-ss-V; App. D/E).

Width 1 must reduce to the width-1 definitions (pinned in test_oracle_pins); the
seeds are checked against Python big-int evaluations of the definitions; the
whole pipeline at width 4 against a brute-force composition built on the ATen
Philox engine; the statistics against Sec. 3 (T = L - h under H0).
"""
import math
from fractions import Fraction

import numpy as np
import pytest

import oracle
import workloads
from engines import engine_words

M = 1 << 64
KEY = oracle.PAPER_KEY
WIDE = 0x243F6A8885A308D3


def _J(a):
    return oracle.jenkins32(int(a) & 0xFFFFFFFF)


def test_width_one_reduces_to_the_width_one_definitions():
    rng = np.random.default_rng(40)
    B, V = 5, 3001
    prev = rng.integers(-10, 1 << 31, B).astype(np.int32)
    x = rng.standard_normal((B, V)).astype(np.float32)
    for seeding in ("context", "self_salt"):
        assert np.array_equal(oracle.green_mask_w(B, V, prev[:, None], WIDE, 0.3, seeding),
                              oracle.green_mask(B, V, prev, WIDE, 0.3, seeding))
        assert np.array_equal(oracle.watermark_w(x, prev[:, None], WIDE, 0.3, 2.0, seeding),
                              oracle.watermark(x, prev, WIDE, 0.3, 2.0, seeding))
        tok = rng.integers(0, V, (6, 50)).astype(np.int32)
        c1, z1 = oracle.detect_w(tok, 1, WIDE, 0.25, seeding)
        c0, z0 = oracle.detect(tok, WIDE, 0.25, seeding)
        assert np.array_equal(c1, c0) and np.array_equal(z1, z0)


def test_width_seeds_against_big_int_definitions():
    rng = np.random.default_rng(41)
    for h in (1, 2, 4, 7):
        ctx = rng.integers(-(1 << 31), 1 << 31, (300, h), dtype=np.int64).astype(np.int32)
        cand = rng.integers(0, 1 << 31, 300).astype(np.int32)
        k = int(rng.integers(0, 1 << 63))
        got_c = oracle.seed_w_many(k, ctx, cand, "context")
        got_s = oracle.seed_w_many(k, ctx, cand, "self_salt")
        for i in range(300):
            window = [int(t) & 0xFFFFFFFF for t in ctx[i]]
            assert int(got_c[i]) == k * sum(window) % M
            hv = _J(cand[i])
            terms = [k * _J(t) * hv % M for t in window] + [k * hv * hv % M]
            assert int(got_s[i]) == min(terms)


def test_width_seeds_ignore_window_order_and_additive_depends_on_the_sum():
    rng = np.random.default_rng(42)
    ctx = rng.integers(0, 150000, (200, 4)).astype(np.int32)
    cand = rng.integers(0, 150000, 200).astype(np.int32)
    perm = ctx[:, ::-1].copy()
    for seeding in ("context", "self_salt"):
        assert np.array_equal(oracle.seed_w_many(KEY, ctx, cand, seeding),
                              oracle.seed_w_many(KEY, perm, cand, seeding))
    # the additive PRF sees only the sum of the window
    same_sum = ctx.copy()
    same_sum[:, 0] += 5
    same_sum[:, 1] -= 5
    assert np.array_equal(oracle.seed_w_many(KEY, ctx, cand, "context"),
                          oracle.seed_w_many(KEY, same_sum, cand, "context"))
    assert not np.array_equal(oracle.seed_w_many(KEY, ctx, cand, "self_salt"),
                              oracle.seed_w_many(KEY, same_sum, cand, "self_salt"))


@pytest.mark.parametrize("seeding", ["context", "self_salt"])
def test_width_four_pipeline_brute_force(xcheck_libs, seeding):
    rng = np.random.default_rng(43)
    B, V, h, gamma, delta = 3, 53, 4, 0.25, np.float32(2.0)
    ctx = rng.integers(0, 1000, (B, h)).astype(np.int32)
    x = rng.standard_normal((B, V)).astype(np.float32)
    got = oracle.watermark_w(x, ctx, WIDE, gamma, float(delta), seeding)
    mask = oracle.green_mask_w(B, V, ctx, WIDE, gamma, seeding)
    for b in range(B):
        window = [int(t) for t in ctx[b]]
        if seeding == "context":
            r = [WIDE * sum(window) % M] * V
        else:
            r = [min([WIDE * _J(t) * _J(v) % M for t in window] + [WIDE * _J(v) ** 2 % M])
                 for v in range(V)]
        words = engine_words(xcheck_libs, "aten", np.arange(V, dtype=np.uint32),
                             np.array(r, dtype=np.uint64))
        green = np.array([Fraction(int(w), 1 << 32) < Fraction(gamma) for w in words])
        assert np.array_equal(got[b].view(np.uint32),
                              np.where(green, x[b] + delta, x[b]).view(np.uint32))
        bits = np.array([(mask[b, v // 32] >> (v % 32)) & 1 for v in range(V)], dtype=bool)
        assert np.array_equal(bits, green)

    tok = rng.integers(0, 3000, (4, 30)).astype(np.int32)
    counts, z = oracle.detect_w(tok, h, WIDE, gamma, seeding)
    for n in range(tok.shape[0]):
        g = 0
        for i in range(h, tok.shape[1]):
            window = [int(t) for t in tok[n, i - h:i]]
            v = int(tok[n, i])
            if seeding == "context":
                r = WIDE * sum(window) % M
            else:
                r = min([WIDE * _J(t) * _J(v) % M for t in window] + [WIDE * _J(v) ** 2 % M])
            w = engine_words(xcheck_libs, "aten", np.array([v], np.uint32), np.array([r], np.uint64))
            g += Fraction(int(w[0]), 1 << 32) < Fraction(gamma)
        assert counts[n] == g
        T = tok.shape[1] - h
        assert z[n] == pytest.approx((g - T * gamma) / math.sqrt(T * gamma * (1 - gamma)), rel=1e-12)


def test_width_detect_degenerate_lengths():
    for L in (0, 1, 3, 4):
        counts, z = oracle.detect_w(np.ones((2, L), np.int32), 4, KEY, 0.25, "self_salt")
        assert np.all(counts == 0) and np.all(np.isnan(z))
    counts, z = oracle.detect_w(np.ones((2, 5), np.int32), 4, KEY, 0.25, "context")
    assert not np.any(np.isnan(z))


@pytest.mark.parametrize("seeding", ["context", "self_salt"])
def test_width_four_null_detection_is_binomial(seeding):
    from scipy import stats
    rng = np.random.default_rng(44)
    N, L, h, gamma = 3000, 200, 4, 0.25
    tok = workloads.uniform_tokens(N, L, 128256, rng)
    counts, z = oracle.detect_w(tok, h, KEY, gamma, seeding)
    T = L - h
    mean, var = stats.binom(T, gamma).stats(moments="mv")
    assert abs(counts.mean() - mean) < 5 * math.sqrt(var / N)
    assert abs(counts.var() / var - 1) < 5 * math.sqrt(2 / N)
    assert abs(z.mean()) < 5 / math.sqrt(N)


@pytest.mark.parametrize("seeding", ["context", "self_salt"])
def test_width_four_green_fraction(seeding):
    rng = np.random.default_rng(45)
    B, V, gamma = 32, 32000, 0.25
    ctx = rng.integers(0, V, (B, 4)).astype(np.int32)
    counts = np.unpackbits(oracle.green_mask_w(B, V, ctx, KEY, gamma, seeding).view(np.uint8),
                           axis=1).sum(axis=1)
    sd = math.sqrt(V * gamma * (1 - gamma))
    assert np.all(np.abs(counts - gamma * V) < 5.5 * sd)
