"""Statistical pins of the oracle: the properties Sec. 3 and App. H derive.

All seeds are fixed and every bound is at least 5 sigma (or a p-value gate of
1e-6), so these never flake; a dropped term, wrong index or wrong sign in the
oracle moves a statistic by far more than the bound.
"""
import math
import os

import numpy as np
import pytest

import oracle
import workloads

HERE = os.path.dirname(os.path.abspath(__file__))


def _paper_numbers():
    vals = {}
    with open(os.path.join(HERE, "golden", "paper_numbers.txt")) as f:
        for line in f:
            if line.strip() and not line.startswith("#"):
                name, value, tol, _ = line.split()
                vals[name] = (float(value), float(tol))
    return vals


def _row_counts(mask: np.ndarray) -> np.ndarray:
    return np.unpackbits(mask.view(np.uint8), axis=1).sum(axis=1)


def test_paper_concentration_numbers():
    # App. H: Var(Gamma) = gamma (1 - gamma) / |V|; at gamma = 0.5, |V| = 151936
    # the paper prints sigma ~ 1.28 per mille, ~195 tokens of ~75968, and a
    # Hoeffding bound below 2e-13 for a 1 % deviation.
    nums = _paper_numbers()
    V, gamma = 151936, 0.5
    sigma = math.sqrt(gamma * (1 - gamma) / V)
    v, tol = nums["sigma_gamma_permille"]
    assert abs(sigma * 1000 - v) <= tol
    v, tol = nums["sigma_gamma_tokens"]
    assert abs(sigma * V - v) <= tol
    v, tol = nums["green_tokens_mean"]
    assert abs(gamma * V - v) <= tol
    assert 2 * math.exp(-2 * V * 1e-4) < nums["hoeffding_bound_max"][0]
    assert nums["paper_key"][0] == oracle.PAPER_KEY == workloads.PAPER_KEY


@pytest.mark.parametrize("seeding", ["context", "self_salt"])
@pytest.mark.parametrize("gamma", [0.25, 0.5])
def test_green_fraction_per_row(seeding, gamma):
    # E|G_t| = gamma |V| with binomial spread (Sec. 2.2; App. H).
    rng = np.random.default_rng(31)
    B, V = 64, 32000
    prev = rng.integers(0, 1 << 31, B).astype(np.int32)
    counts = _row_counts(oracle.green_mask(B, V, prev, oracle.PAPER_KEY, gamma, seeding))
    sd = math.sqrt(V * gamma * (1 - gamma))
    assert np.all(np.abs(counts - gamma * V) < 5.5 * sd)
    if seeding == "context":
        # Distinct context seeds give independent lists, so the mean over rows is
        # sqrt(B) tighter.  Self-salt rows are not independent: the K*J(v)*J(v) term
        # of the minimum does not depend on the context, so whenever it wins, v has
        # the same colour in every row (see test_self_salt_rows_share_colours).
        assert abs(counts.mean() - gamma * V) < 5 * sd / math.sqrt(B)


def test_self_salt_rows_share_colours():
    # Under self-salt a token whose self term K*J(v)^2 is the minimum for both
    # contexts has one colour in both rows, so two rows agree on more than the
    # gamma^2 + (1 - gamma)^2 of independent lists; context-seeded rows do not.
    B, V, gamma = 2, 200_000, 0.25
    prev = np.array([101, 202], np.int32)
    indep = gamma ** 2 + (1 - gamma) ** 2
    sd = math.sqrt(indep * (1 - indep) / V)
    for seeding, correlated in (("context", False), ("self_salt", True)):
        bits = np.unpackbits(oracle.green_mask(B, V, prev, oracle.PAPER_KEY, gamma, seeding)
                             .view(np.uint8), axis=1, bitorder="little")[:, :V]
        agree = (bits[0] == bits[1]).mean()
        if correlated:
            assert agree > indep + 10 * sd
        else:
            assert abs(agree - indep) < 5 * sd


def test_green_fraction_spread_matches_app_h():
    # std of the row proportion over many rows ~ sqrt(gamma (1 - gamma) / |V|).
    rng = np.random.default_rng(32)
    B, V, gamma = 1024, 16384, 0.5
    prev = rng.integers(1, V, B).astype(np.int32)
    frac = _row_counts(oracle.green_mask(B, V, prev, 0x243F6A8885A308D3, gamma)) / V
    expect = math.sqrt(gamma * (1 - gamma) / V)
    assert abs(frac.std(ddof=1) / expect - 1) < 0.12


def test_no_row_deviates_one_percent_at_paper_vocabulary():
    # App. H, Hoeffding: at |V| = 151936, P(|Gamma - gamma| > 0.01) < 2e-13 per row.
    rng = np.random.default_rng(39)
    B, V, gamma = 64, 151936, 0.5
    prev = rng.integers(1, V, B).astype(np.int32)
    frac = _row_counts(oracle.green_mask(B, V, prev, oracle.PAPER_KEY, gamma)) / V
    assert np.all(np.abs(frac - gamma) < 0.01)


def test_mask_bits_are_independent_across_positions():
    # Bernoulli lists: each token independently green with probability gamma, so
    # adjacent positions (which share a Philox block under context seeding) must
    # show no correlation.
    rng = np.random.default_rng(33)
    B, V, gamma = 256, 8192, 0.25
    prev = rng.integers(1, 1 << 30, B).astype(np.int32)
    mask = oracle.green_mask(B, V, prev, oracle.PAPER_KEY, gamma)
    bits = np.unpackbits(mask.view(np.uint8), axis=1, bitorder="little").astype(np.float64)
    for lag in (1, 2, 3, 4, 5):
        a, b = bits[:, :-lag].ravel(), bits[:, lag:].ravel()
        corr = np.corrcoef(a, b)[0, 1]
        assert abs(corr) < 5 / math.sqrt(a.size), lag


def test_null_detection_is_binomial():
    # Under H0 the count is Binomial(T, gamma) and z has mean 0, variance 1 (Sec. 3).
    from scipy import stats
    rng = np.random.default_rng(34)
    N, L, V, gamma = 3000, 200, 128256, 0.25
    for seeding in ("context", "self_salt"):
        tok = workloads.uniform_tokens(N, L, V, rng)
        counts, z = oracle.detect(tok, oracle.PAPER_KEY, gamma, seeding)
        T = L - 1
        pmf = stats.binom(T, gamma).pmf(np.arange(T + 1))
        # chi-square on binned counts (bins with expected >= 20)
        edges = [0]
        acc = 0.0
        for k in range(T + 1):
            acc += pmf[k] * N
            if acc >= 20:
                edges.append(k + 1)
                acc = 0.0
        edges[-1] = T + 1
        observed = np.array([((counts >= lo) & (counts < hi)).sum() for lo, hi in zip(edges, edges[1:])])
        expected = np.array([pmf[lo:hi].sum() * N for lo, hi in zip(edges, edges[1:])])
        expected *= observed.sum() / expected.sum()
        _, p = stats.chisquare(observed, expected)
        assert p > 1e-6, seeding
        assert abs(z.mean()) < 5 / math.sqrt(N)
        assert abs(z.var() - 1) < 5 * math.sqrt(2 / N)


def test_watermarked_detection_closed_form():
    # Watermarked text: P(green) = gamma e^delta / (gamma e^delta + 1 - gamma), so
    # E[z] = (q - gamma) T / sqrt(T gamma (1 - gamma)) (~24.1 at T = 511, gamma 1/4, delta 2).
    rng = np.random.default_rng(35)
    N, L, V, gamma, delta = 200, 512, 128256, 0.25, 2.0

    def member(p, c):
        return oracle.is_green_many(oracle.PAPER_KEY, p, c, gamma, "context")

    tok = workloads.sample_watermarked(N, L, V, gamma, delta, member, rng)
    counts, z = oracle.detect(tok, oracle.PAPER_KEY, gamma, "context")
    T = L - 1
    q = workloads.green_probability(gamma, delta)
    assert q == pytest.approx(0.7112, abs=1e-4)
    ez = (q - gamma) * T / math.sqrt(T * gamma * (1 - gamma))
    assert ez == pytest.approx(24.1, abs=0.05)
    sd_z = math.sqrt(T * q * (1 - q) / (T * gamma * (1 - gamma)))
    assert abs(z.mean() - ez) < 5 * sd_z / math.sqrt(N)
    assert abs(z.std() / sd_z - 1) < 0.25


def test_sampler_against_exact_softmax():
    # The rejection sampler stands in for sampling softmax(l + delta*[green]) of
    # fresh N(0,1) logits; compare green fractions with the exact O(V) sampler.
    rng = np.random.default_rng(36)
    V, gamma, delta, steps = 4096, 0.25, 2.0, 3000
    key = oracle.PAPER_KEY
    prev = 17
    exact_green = 0
    for _ in range(steps):
        green = oracle.is_green_many(key, np.full(V, prev, np.int32), np.arange(V, dtype=np.int32),
                                     gamma, "context")
        logits = rng.standard_normal(V) + delta * green
        p = np.exp(logits - logits.max())
        p /= p.sum()
        tok = int(rng.choice(V, p=p))
        exact_green += int(green[tok])
        prev = tok
    frac = exact_green / steps
    q = workloads.green_probability(gamma, delta)
    assert abs(frac - q) < 5 * math.sqrt(q * (1 - q) / steps) + 0.01


def test_determinism_and_key_sensitivity():
    rng = np.random.default_rng(37)
    B, V = 8, 5000
    prev = rng.integers(1, V, B).astype(np.int32)
    for seeding in ("context", "self_salt"):
        a = oracle.green_mask(B, V, prev, oracle.PAPER_KEY, 0.25, seeding)
        b = oracle.green_mask(B, V, prev, oracle.PAPER_KEY, 0.25, seeding)
        c = oracle.green_mask(B, V, prev, oracle.PAPER_KEY + 2, 0.25, seeding)
        assert np.array_equal(a, b)
        ba = np.unpackbits(a.view(np.uint8))
        bc = np.unpackbits(c.view(np.uint8))
        agree = (ba == bc).mean()
        # independent lists agree on gamma^2 + (1 - gamma)^2 = 0.625 of tokens
        assert abs(agree - 0.625) < 0.02, seeding


def test_self_salt_and_context_lists_are_unrelated():
    # Self-salt membership depends on the candidate: its list agrees with the
    # context list about as often as two independent lists do.
    rng = np.random.default_rng(38)
    B, V, gamma = 16, 20000, 0.25
    prev = rng.integers(1, V, B).astype(np.int32)
    words = (V + 31) // 32
    a = np.unpackbits(oracle.green_mask(B, V, prev, oracle.PAPER_KEY, gamma, "context")
                      .view(np.uint8), axis=1, bitorder="little")[:, :V]
    b = np.unpackbits(oracle.green_mask(B, V, prev, oracle.PAPER_KEY, gamma, "self_salt")
                      .view(np.uint8), axis=1, bitorder="little")[:, :V]
    assert a.shape == (B, V) and words * 32 >= V
    agree = (a == b).mean()
    expect = gamma ** 2 + (1 - gamma) ** 2
    assert abs(agree - expect) < 5 * math.sqrt(expect * (1 - expect) / (B * V))


def test_context_seed_zero_prev_is_key_independent():
    # Reading R3's wart: p = 0 gives r = 0, the same list for every key.
    a = oracle.green_mask(1, 3000, np.array([0], np.int32), oracle.PAPER_KEY, 0.25)
    b = oracle.green_mask(1, 3000, np.array([0], np.int32), 12345, 0.25)
    assert np.array_equal(a, b)
