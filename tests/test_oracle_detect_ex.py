"""Pins of the oracle's detection with per-sequence lengths and repeated n-grams
scored once (a production-detector extension of the Sec. 3 z-test; the paper leaves
both open).

Without lengths or the repeat rule it must equal oracle_detect_w (pinned in
test_oracle_width); with lengths, detect_w of each truncated sequence, lengths
clamped to [0, L]; with the repeat rule, a brute force over Python sets of
(window, token) tuples, the membership taken from is_green_w_many (pinned
separately); closed forms on periodic sequences.
"""
import math

import numpy as np
import pytest

import oracle
import workloads

KEY = oracle.PAPER_KEY


def _z(W, T, gamma):
    return (W - T * gamma) / math.sqrt(T * gamma * (1 - gamma)) if T > 0 else float("nan")


def _brute(tok, lengths, width, key, gamma, seeding, ignore):
    counts, scored, zs = [], [], []
    for n, seq in enumerate(tok):
        ln = tok.shape[1] if lengths is None else int(min(max(lengths[n], 0), tok.shape[1]))
        seen, grams = set(), []
        for i in range(width, ln):
            g = tuple(int(t) for t in seq[i - width:i + 1])
            if ignore and g in seen:
                continue
            seen.add(g)
            grams.append(g)
        if grams:
            ctx = np.array([g[:-1] for g in grams], dtype=np.int32).reshape(len(grams), width)
            cand = np.array([g[-1] for g in grams], dtype=np.int32)
            W = int(oracle.is_green_w_many(key, ctx, cand, gamma, seeding).sum())
        else:
            W = 0
        counts.append(W); scored.append(len(grams)); zs.append(_z(W, len(grams), gamma))
    return np.array(counts), np.array(scored), np.array(zs)


def _eq(got, expect):
    gc, gs, gz = got
    ec, es, ez = expect
    assert np.array_equal(gc, ec) and np.array_equal(gs, es)
    assert np.array_equal(np.isnan(gz), np.isnan(ez))
    ok = ~np.isnan(ez)
    np.testing.assert_allclose(gz[ok], ez[ok], rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("seeding", ["context", "self_salt"])
@pytest.mark.parametrize("width", [1, 4])
def test_plain_and_lengths_reduce_to_detect_w(seeding, width):
    rng = np.random.default_rng(170 + width)
    N, L, V = 12, 90, 500
    tok = rng.integers(0, V, (N, L)).astype(np.int32)
    c, s, z = oracle.detect_ex(tok, width, KEY, 0.25, seeding)
    ec, ez = oracle.detect_w(tok, width, KEY, 0.25, seeding)
    assert np.array_equal(c, ec) and np.array_equal(s, np.full(N, L - width))
    np.testing.assert_array_equal(z, ez)
    lengths = np.array([0, 1, width, width + 1, 17, 89, 90, 91, -5, 2**31 - 1, 50, 3], np.int32)
    c, s, z = oracle.detect_ex(tok, width, KEY, 0.25, seeding, lengths=lengths)
    for n in range(N):
        ln = min(max(int(lengths[n]), 0), L)
        ec, ez = oracle.detect_w(tok[n:n + 1, :ln], width, KEY, 0.25, seeding)
        assert c[n] == ec[0] and s[n] == max(ln - width, 0)
        assert (np.isnan(z[n]) and np.isnan(ez[0])) or z[n] == ez[0]


@pytest.mark.parametrize("seeding", ["context", "self_salt"])
@pytest.mark.parametrize("width", [1, 4])
def test_repeated_ngrams_match_a_set_brute_force(seeding, width):
    rng = np.random.default_rng(180 + width)
    N, L, V = 10, 120, 7          # a tiny vocabulary makes repeats common
    tok = rng.integers(0, V, (N, L)).astype(np.int32)
    tok[3, 60:100] = tok[3, 10:50]                  # a copied span
    tok[4, :] = 5                                    # one token throughout
    lengths = rng.integers(-3, L + 5, N).astype(np.int32)
    for lens in (None, lengths):
        _eq(oracle.detect_ex(tok, width, KEY, 0.5, seeding, lengths=lens, ignore_repeated=True),
            _brute(tok, lens, width, KEY, 0.5, seeding, True))
        _eq(oracle.detect_ex(tok, width, KEY, 0.5, seeding, lengths=lens),
            _brute(tok, lens, width, KEY, 0.5, seeding, False))


def test_repeat_rule_closed_forms():
    rng = np.random.default_rng(190)
    # no repeated n-gram: the rule changes nothing
    tok = np.stack([rng.permutation(1000)[:300] for _ in range(4)]).astype(np.int32)
    for width in (1, 4):
        a = oracle.detect_ex(tok, width, KEY, 0.25, "self_salt", ignore_repeated=True)
        b = oracle.detect_ex(tok, width, KEY, 0.25, "self_salt")
        _eq(a, b)
    # a period-P sequence of distinct tokens has exactly P distinct (h+1)-grams, and
    # its green count is that of one period
    P, R, width = 13, 9, 4
    period = rng.permutation(500)[:P].astype(np.int32)
    seq = np.tile(period, R)[None, :]
    c, s, _ = oracle.detect_ex(seq, width, KEY, 0.25, "context", ignore_repeated=True)
    assert s[0] == P
    c_one, s_one, _ = oracle.detect_ex(seq[:, :P + width], width, KEY, 0.25, "context")
    assert s_one[0] == P and c[0] == c_one[0]
    # one token repeated: a single distinct n-gram
    c, s, _ = oracle.detect_ex(np.full((1, 50), 42, np.int32), 1, KEY, 0.25, "context",
                               ignore_repeated=True)
    assert s[0] == 1
