"""Pins of the oracle's candidate-restricted watermark (SBW-ss of the scheme table,
Sec. 4: the self-salt watermark of width 4 applied to the top-40 candidates only).

With distinct in-range candidates it must equal the full-vocabulary watermark (pinned
in test_oracle_pins and test_oracle_width) at the candidate positions and leave every
other logit alone; a repeated id counts once; ids outside [0, V) are ignored; the
order of the candidates does not matter; and the green fraction over many candidate
sets is gamma.
"""
import numpy as np
import pytest

import oracle
import workloads

KEY = oracle.PAPER_KEY
WIDE = workloads.WIDE_KEY


def _topk(x, k):
    xf = (x.astype(np.uint32) << 16).view(np.float32) if x.dtype == np.uint16 else x
    return np.argsort(-xf, axis=1, kind="stable")[:, :k].astype(np.int32)


def _restricted_full(x, cand, ctx, key, gamma, delta, seeding):
    """The full-vocabulary watermark, taken at the candidates only."""
    full = oracle.watermark_w(x, ctx, key, gamma, delta, seeding)
    out = np.array(x, copy=True)
    for b in range(x.shape[0]):
        ids = np.unique(cand[b][(cand[b] >= 0) & (cand[b] < x.shape[1])])
        out[b, ids] = full[b, ids]
    return out


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("seeding", ["self_salt", "context"])
@pytest.mark.parametrize("width", [1, 4])
def test_candidates_equal_the_full_watermark_at_the_candidates(dtype, seeding, width):
    rng = np.random.default_rng(120 + width)
    B, V, k = 6, 3001, 40
    x = rng.standard_normal((B, V)).astype(np.float32)
    if dtype == "bf16":
        x = workloads.f32_to_bf16_bits(x)
    ctx = workloads.context_tokens(B, width, V, rng)
    cand = _topk(x, k)
    for gamma, delta in [(0.25, 2.0), (0.5, -1.5), (1.0, 0.5)]:
        got = oracle.watermark_candidates(x, cand, ctx, WIDE, gamma, delta, seeding)
        expect = _restricted_full(x, cand, ctx, WIDE, gamma, delta, seeding)
        assert np.array_equal(got.view(np.uint8), expect.view(np.uint8)), (gamma, delta)
        other = np.ones_like(x, dtype=bool)
        other[np.arange(B)[:, None], cand] = False
        assert np.array_equal(got[other].view(np.uint8), x[other].view(np.uint8))


def test_candidate_order_duplicates_and_range():
    rng = np.random.default_rng(130)
    B, V = 4, 500
    x = rng.standard_normal((B, V)).astype(np.float32)
    ctx = workloads.context_tokens(B, 4, V, rng)
    base = np.stack([rng.choice(V, 30, replace=False) for _ in range(B)]).astype(np.int32)
    ref = oracle.watermark_candidates(x, base, ctx, KEY, 1.0, 2.0)   # gamma=1: every candidate biased
    assert np.array_equal(ref[np.arange(B)[:, None], base], x[np.arange(B)[:, None], base] + 2.0)
    # any order
    perm = base[:, rng.permutation(30)]
    assert np.array_equal(oracle.watermark_candidates(x, perm, ctx, KEY, 0.5, 2.0),
                          oracle.watermark_candidates(x, base, ctx, KEY, 0.5, 2.0))
    # repeats count once, out-of-range ids are ignored
    noisy = np.concatenate([base, base[:, :7], np.full((B, 3), -1, np.int32),
                            np.full((B, 2), V, np.int32), np.full((B, 1), 2**31 - 1, np.int32)], axis=1)
    assert np.array_equal(oracle.watermark_candidates(x, noisy, ctx, KEY, 1.0, 2.0), ref)
    adjacent = np.repeat(base, 2, axis=1)          # every id twice, side by side
    assert np.array_equal(oracle.watermark_candidates(x, adjacent, ctx, KEY, 1.0, 2.0), ref)
    # no candidates, or gamma = 0: nothing changes
    assert np.array_equal(oracle.watermark_candidates(x, base[:, :0], ctx, KEY, 1.0, 2.0), x)
    assert np.array_equal(oracle.watermark_candidates(x, base, ctx, KEY, 0.0, 2.0), x)


def test_candidate_green_fraction_is_gamma():
    # 400 rows x 40 candidates under self-salt width 4: green count ~ Binomial(16000, gamma)
    rng = np.random.default_rng(140)
    B, V, k, gamma = 400, 20000, 40, 0.25
    x = np.zeros((B, V), dtype=np.float32)
    ctx = workloads.context_tokens(B, 4, V, rng)
    cand = np.stack([rng.choice(V, k, replace=False) for _ in range(B)]).astype(np.int32)
    got = oracle.watermark_candidates(x, cand, ctx, KEY, gamma, 1.0)
    greens = int((got != 0).sum())
    n = B * k
    assert abs(greens - gamma * n) < 5 * np.sqrt(n * gamma * (1 - gamma))
    assert int((got[np.arange(B)[:, None], cand] != 0).sum()) == greens   # only candidates move
