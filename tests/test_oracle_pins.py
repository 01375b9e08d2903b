"""Pins of the CPU oracle against what the paper and the mathematics fix.

Nothing here compares the oracle with itself: every check is against published
known-answer vectors, independent open-source engines, exact rational or
arbitrary-precision arithmetic, library routines (numpy, torch, scipy) or a
statistical property the paper derives.  The Jenkins hash has no such value
available and is checked by properties only (parity unpinned).
"""
import ctypes
import math
import os
import shutil
import subprocess
from fractions import Fraction

import numpy as np
import pytest

import oracle
from engines import engine_words as _engine_words

HERE = os.path.dirname(os.path.abspath(__file__))
GOLDEN = os.path.join(HERE, "golden")
M64 = (1 << 64) - 1


# --- Philox4x32-10 and CBRNG(v, r)  (Sec. 2.2) ----------------------------------

def _kat():
    rows = []
    with open(os.path.join(GOLDEN, "philox4x32_10_kat.txt")) as f:
        for line in f:
            if line.strip() and not line.startswith("#"):
                w = [int(x, 16) for x in line.split()]
                rows.append((w[0:4], w[4:6], w[6:10]))
    return rows


@pytest.mark.parametrize("ctr,key,expect", _kat())
def test_philox_known_answers(ctr, key, expect):
    assert list(oracle.philox4x32_10(ctr, key)) == expect


@pytest.mark.parametrize("engine", ["aten", "rocrand"])
def test_cbrng_matches_open_source_engines(xcheck_libs, engine):
    if engine not in xcheck_libs:
        pytest.skip(f"{engine} harness not buildable here")
    rng = np.random.default_rng(7)
    n = 200_000
    v = rng.integers(0, 1 << 32, n, dtype=np.uint64).astype(np.uint32)
    r = rng.integers(0, 1 << 64, n, dtype=np.uint64)
    v[:8] = [0, 1, 2, 3, 4, 151935, (1 << 31) - 1, (1 << 32) - 1]
    r[:4] = [0, M64, 1 << 32, 0xFFFFFFFF]
    r[4:8] = [oracle.PAPER_KEY, oracle.PAPER_KEY * 7 & M64, 0x243F6A8885A308D3, 5]
    assert np.array_equal(oracle.cbrng_many(v, r), _engine_words(xcheck_libs, engine, v, r))


def test_cbrng_small_positions_are_block_words():
    # Position v of the stream is word v%4 of the block at counter v//4 (reading R1):
    # the first 8 positions are the two first blocks, word by word.
    r = 0x243F6A8885A308D3
    key = [r & 0xFFFFFFFF, r >> 32]
    blocks = np.concatenate([oracle.philox4x32_10([0, 0, 0, 0], key),
                             oracle.philox4x32_10([1, 0, 0, 0], key)])
    assert [oracle.cbrng(v, r) for v in range(8)] == list(blocks)


# --- threshold (Sec. 2.2, Eq. 1; reading R2) -------------------------------------

def test_threshold_closed_forms():
    assert oracle.threshold(0.0) == 0
    assert oracle.threshold(1.0) == 1 << 32
    assert oracle.threshold(0.25) == 1 << 30
    assert oracle.threshold(0.5) == 1 << 31
    assert oracle.threshold(-0.5) == 0
    assert oracle.threshold(2.0) == 1 << 32
    rng = np.random.default_rng(3)
    x = rng.integers(0, 1 << 32, 100_000, dtype=np.uint64)
    # gamma = 1/4: green <=> the top two bits are zero; gamma = 1/2: top bit zero.
    assert np.array_equal(x < oracle.threshold(0.25), (x >> np.uint64(30)) == 0)
    assert np.array_equal(x < oracle.threshold(0.5), (x >> np.uint64(31)) == 0)


@pytest.mark.parametrize("gamma", [0.1, 0.3, 1 / 3, 0.7, 1e-9, 0.999999999, 5e-324])
def test_threshold_is_exact_real_comparison(gamma):
    # x < T  <=>  x / 2^32 < gamma exactly, checked in rational arithmetic at the
    # boundary x = T - 1 (green) and x = T (not green).
    T = oracle.threshold(gamma)
    g = Fraction(gamma)
    assert Fraction(T - 1, 1 << 32) < g
    assert not (Fraction(T, 1 << 32) < g)


# --- seeds (Sec. 2.2 PRF, Sec. 2.3 Jenkins, Sec. 5.2 self-salt) ------------------

def test_context_seed_modular_product():
    rng = np.random.default_rng(11)
    for _ in range(2000):
        k = int(rng.integers(0, 1 << 64, dtype=np.uint64))
        p = int(rng.integers(0, 1 << 32, dtype=np.uint64))
        assert oracle.seed_context(k, p) == (k * p) % (1 << 64)
    k = oracle.PAPER_KEY
    assert oracle.seed_context(k, 0) == 0          # reading R3: p = 0 gives r = 0
    assert oracle.seed_context(k, 1) == k
    assert oracle.seed_context(1 << 63, 3) == 1 << 63
    assert oracle.seed_context(1 << 63, 2) == 0
    # additivity in p (mod 2^64)
    a, b = 123457, 98765431
    assert oracle.seed_context(k, a + b) == (oracle.seed_context(k, a) + oracle.seed_context(k, b)) % (1 << 64)
    # negative token ids are their 32-bit pattern (reading R8)
    assert oracle.seed_context(k, -1) == (k * 0xFFFFFFFF) % (1 << 64)


def test_jenkins_is_a_bijection_on_samples():
    # Every step of the mix is invertible, so no two inputs may collide.
    a = np.arange(1 << 20, dtype=np.uint32)
    h = oracle.jenkins32_many(a)
    assert np.unique(h).size == a.size
    rng = np.random.default_rng(5)
    b = np.unique(rng.integers(0, 1 << 32, 1 << 20, dtype=np.uint64).astype(np.uint32))
    assert np.unique(oracle.jenkins32_many(b)).size == b.size


def test_jenkins_avalanche():
    # Flipping one input bit flips about half of the 32 output bits on average.
    rng = np.random.default_rng(6)
    a = rng.integers(0, 1 << 32, 20000, dtype=np.uint64).astype(np.uint32)
    h = oracle.jenkins32_many(a)
    flips = []
    for bit in range(32):
        d = h ^ oracle.jenkins32_many(a ^ np.uint32(1 << bit))
        flips.append(np.unpackbits(d.view(np.uint8)).sum() / a.size)
    flips = np.array(flips)
    assert 15.0 < flips.mean() < 17.0
    assert flips.min() > 10.0


def test_jenkins_uniform_low_bits():
    from scipy import stats
    h = oracle.jenkins32_many(np.arange(1 << 20, dtype=np.uint32))
    counts = np.bincount(h & np.uint32(0xFFFF), minlength=1 << 16)
    _, p = stats.chisquare(counts)
    assert p > 1e-6
    counts_hi = np.bincount(h >> np.uint32(16), minlength=1 << 16)
    _, p_hi = stats.chisquare(counts_hi)
    assert p_hi > 1e-6


def test_self_salt_seed_definition():
    rng = np.random.default_rng(12)
    for _ in range(2000):
        k = int(rng.integers(0, 1 << 64, dtype=np.uint64))
        p = int(rng.integers(0, 1 << 32, dtype=np.uint64))
        v = int(rng.integers(0, 1 << 32, dtype=np.uint64))
        hp, hv = oracle.jenkins32(p), oracle.jenkins32(v)
        expect = min(k * hp * hv % (1 << 64), k * hv * hv % (1 << 64))
        assert oracle.seed_self_salt(k, p, v) == expect
    # p == v: both terms of the minimum coincide
    k = oracle.PAPER_KEY
    hv = oracle.jenkins32(77)
    assert oracle.seed_self_salt(k, 77, 77) == k * hv * hv % (1 << 64)


def test_self_salt_seed_depends_on_candidate():
    k = oracle.PAPER_KEY
    v = np.arange(50_000, dtype=np.int32)
    r = oracle.seed_many(k, np.full_like(v, 1234), v, "self_salt")
    assert np.unique(r).size > 0.99 * v.size
    rc = oracle.seed_many(k, np.full_like(v, 1234), v, "context")
    assert np.unique(rc).size == 1


# --- bias arithmetic (Sec. 2.2, Eq. 2; reading R7) -------------------------------

def test_f32_bias_matches_numpy():
    rng = np.random.default_rng(8)
    x = rng.standard_normal(200_000).astype(np.float32) * np.float32(30)
    specials = np.array([0.0, -0.0, np.inf, -np.inf, 1e-45, -1e-45, 1e-40, 3.4e38,
                         -3.4e38, 1.17549435e-38], dtype=np.float32)
    x = np.concatenate([x, specials])
    for delta in (2.0, -1.5, 1e-3, 1e-45, 0.0, -0.0, 8.0):
        with np.errstate(over="ignore"):
            expect = x + np.float32(delta)
        got = oracle.bias_f32_many(x, delta)
        assert np.array_equal(got.view(np.uint32), expect.view(np.uint32)), delta


@pytest.mark.parametrize("delta", [1.0, -1.0, 2.0, 4.0, 8.0, 0.5, 1e-3, -0.0, 3e38, 1e-40])
def test_bf16_bias_exhaustive_against_torch(delta):
    import torch
    bits = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    t = torch.from_numpy(bits.view(np.int16).copy()).view(torch.bfloat16)
    expect = (t.float() + torch.tensor(delta, dtype=torch.float32)).to(torch.bfloat16)
    expect = expect.view(torch.int16).numpy().view(np.uint16)
    got = oracle.bias_bf16_many(bits, delta)
    e_nan = np.isnan(torch.from_numpy(expect.view(np.int16).copy()).view(torch.bfloat16).float().numpy())
    g_nan = np.isnan((got.astype(np.uint32) << 16).view(np.float32))
    assert np.array_equal(e_nan, g_nan)
    assert np.array_equal(got[~g_nan], expect[~e_nan])


def test_f32_to_bf16_rounding_against_torch():
    import torch
    rng = np.random.default_rng(9)
    u = rng.integers(0, 1 << 32, 1 << 20, dtype=np.uint64).astype(np.uint32)
    # ties and near-ties, the cases round-to-nearest-even decides
    u[:4096] = (u[:4096] & np.uint32(0xFFFF0000)) | np.uint32(0x8000)
    u[4096:8192] = (u[4096:8192] & np.uint32(0xFFFF0000)) | np.uint32(0x7FFF)
    x = u.view(np.float32)
    expect = torch.from_numpy(x.copy()).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    got = oracle.f32_to_bf16_many(x)
    nan = np.isnan(x)
    assert np.array_equal(got[~nan], expect[~nan])
    assert np.all(np.isnan((got[nan].astype(np.uint32) << 16).view(np.float32)))


# --- z-score (Sec. 3) ------------------------------------------------------------

def test_z_score_is_standardised_binomial():
    from scipy import stats
    for T, gamma in [(199, 0.25), (511, 0.25), (511, 0.5), (1, 0.5), (10_000, 0.1)]:
        mean, var = stats.binom(T, gamma).stats(moments="mv")
        for g in {0, 1, T // 3, int(gamma * T), T}:
            z = oracle.z_score(g, T, gamma)
            assert z == pytest.approx((g - float(mean)) / math.sqrt(float(var)), rel=1e-12, abs=1e-12)
    assert oracle.z_score(128, 512, 0.25) == 0.0
    assert oracle.z_score(511, 511, 0.25) == pytest.approx(math.sqrt(511 * 0.75 / 0.25), rel=1e-13)
    assert math.isnan(oracle.z_score(0, 0, 0.25))


# --- whole pipeline on tiny inputs vs an independent composition ------------------

def _brute_green(libs, key, prev, V, gamma, seeding):
    """Green list built from the ATen engine, Python big-int seeds, exact rationals."""
    v = np.arange(V, dtype=np.uint32)
    if seeding == "context":
        r = np.full(V, (key * (prev & 0xFFFFFFFF)) % (1 << 64), dtype=np.uint64)
    else:
        hp = oracle.jenkins32(prev)  # Jenkins itself is pinned by properties only
        r = np.array([min(key * hp * oracle.jenkins32(x) % (1 << 64),
                          key * oracle.jenkins32(x) ** 2 % (1 << 64)) for x in range(V)],
                     dtype=np.uint64)
    words = _engine_words(libs, "aten", v, r)
    g = Fraction(gamma)
    return np.array([Fraction(int(w), 1 << 32) < g for w in words])


@pytest.mark.parametrize("seeding", ["context", "self_salt"])
@pytest.mark.parametrize("gamma", [0.25, 0.5, 0.3])
def test_watermark_and_mask_brute_force(xcheck_libs, seeding, gamma):
    rng = np.random.default_rng(21)
    B, V, delta = 4, 67, np.float32(2.0)
    key = 0x243F6A8885A308D3
    x = rng.standard_normal((B, V)).astype(np.float32)
    prev = rng.integers(0, V, B).astype(np.int32)
    got = oracle.watermark(x, prev, key, gamma, float(delta), seeding)
    mask = oracle.green_mask(B, V, prev, key, gamma, seeding)
    for b in range(B):
        green = _brute_green(xcheck_libs, key, int(prev[b]), V, gamma, seeding)
        expect = np.where(green, x[b] + delta, x[b])
        assert np.array_equal(got[b].view(np.uint32), expect.view(np.uint32))
        bits = np.array([(mask[b, v // 32] >> (v % 32)) & 1 for v in range(V)], dtype=bool)
        assert np.array_equal(bits, green)
        # bits past V stay clear
        assert mask[b, -1] >> (V % 32) == 0


@pytest.mark.parametrize("seeding", ["context", "self_salt"])
def test_detect_brute_force(xcheck_libs, seeding):
    rng = np.random.default_rng(22)
    key, gamma = oracle.PAPER_KEY, 0.25
    tok = rng.integers(0, 5000, (5, 40)).astype(np.int32)
    counts, z = oracle.detect(tok, key, gamma, seeding)
    for n in range(tok.shape[0]):
        p = tok[n, :-1].astype(np.int64)
        v = tok[n, 1:].astype(np.uint32)
        if seeding == "context":
            r = np.array([(key * (int(a) & 0xFFFFFFFF)) % (1 << 64) for a in p], dtype=np.uint64)
        else:
            r = np.array([min(key * oracle.jenkins32(int(a)) * oracle.jenkins32(int(b)) % (1 << 64),
                              key * oracle.jenkins32(int(b)) ** 2 % (1 << 64))
                          for a, b in zip(p, v)], dtype=np.uint64)
        words = _engine_words(xcheck_libs, "aten", v, r)
        g = int(sum(Fraction(int(w), 1 << 32) < Fraction(gamma) for w in words))
        assert counts[n] == g
        T = tok.shape[1] - 1
        assert z[n] == pytest.approx((g - T * gamma) / math.sqrt(T * gamma * (1 - gamma)), rel=1e-12)


def test_detect_degenerate_lengths():
    tok = np.zeros((3, 1), dtype=np.int32)
    counts, z = oracle.detect(tok, oracle.PAPER_KEY, 0.25)
    assert np.all(counts == 0) and np.all(np.isnan(z))
    counts, z = oracle.detect(np.zeros((2, 0), dtype=np.int32), oracle.PAPER_KEY, 0.25)
    assert np.all(counts == 0) and np.all(np.isnan(z))
