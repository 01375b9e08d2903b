"""Seeded synthetic inputs for the watermark and detect hot path.

This module holds none of the watermark's arithmetic: it draws logits, previous
tokens and token sequences with numpy's PCG64 and shapes them like the paper's
workloads (vocabulary ~1.5e5, decode batches 1..1024, sequences of a few hundred
tokens).  The one place that needs green-list membership, the watermarked
sequence sampler, takes it as a callback, so the tests can pass the CPU oracle
and the benchmark can pass the HIP library.

Configurations (seed = 42 + config id; 42 and the key 15485863 are the values the
paper fixes for its experiments in App. C):

  c1  context seeding, B=1,    V=32000,  fp32 N(0,1),  gamma=0.25, delta=2;
      detect on 8 x 200 uniform token ids
  c2  context seeding, B=64,   V=128256, bf16 2*N(0,1), gamma=0.5, delta=2;
      sweep gamma in {0.25, 0.5} x delta in {1, 2, 4, 8}
  c3  self-salt,       B=64,   V=128256, fp32 N(0,1),  gamma=0.25, delta=4
  c4  self-salt (and context at the same shape), B in {256, 1024}, V=152064,
      fp32 3*N(0,1) + 8*[U < 0.05], gamma=0.25, delta=2
  c5  detect, N=4096 x L=512 over V=128256: rows [0, N/2) uniform ids (null),
      rows [N/2, N) sampled from the watermarked softmax of N(0,1) logits
      (gamma=0.25, delta=2), one array per seeding scheme
"""
from __future__ import annotations

import math
from typing import Callable

import numpy as np

PAPER_KEY = 15485863          # hash key of the paper's experiments (App. C)
PAPER_SEED = 42               # random seed of the paper's experiments (App. C)
WIDE_KEY = 0x243F6A8885A308D3  # a key with both 32-bit halves non-zero

C1 = dict(name="c1", B=1, V=32000, dtype="f32", sigma=1.0, seeding="context",
          gamma=0.25, delta=2.0, detect_N=8, detect_L=200)
C2 = dict(name="c2", B=64, V=128256, dtype="bf16", sigma=2.0, seeding="context",
          gamma=0.5, delta=2.0,
          sweep=[(g, d) for g in (0.25, 0.5) for d in (1.0, 2.0, 4.0, 8.0)])
C3 = dict(name="c3", B=64, V=128256, dtype="f32", sigma=1.0, seeding="self_salt",
          gamma=0.25, delta=4.0)
C4 = dict(name="c4", B=256, B_large=1024, V=152064, dtype="f32", sigma=3.0,
          seeding="self_salt", gamma=0.25, delta=2.0, peak_frac=0.05, peak_shift=8.0)
C5 = dict(name="c5", N=4096, L=512, V=128256, gamma=0.25, delta=2.0)
CONFIGS = {c["name"]: c for c in (C1, C2, C3, C4, C5)}
CONFIG_ID = {"c1": 1, "c2": 2, "c3": 3, "c4": 4, "c5": 5}


def rng_for(config: str, salt: int = 0) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(PAPER_SEED + CONFIG_ID[config] + 1000 * salt))


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round-to-nearest-even fp32 -> bf16 of input data, via torch's CPU cast."""
    import torch
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16).copy()


def logits(B: int, V: int, sigma: float = 1.0, rng: np.random.Generator | None = None,
           peak_frac: float = 0.0, peak_shift: float = 0.0) -> np.ndarray:
    """fp32 logits sigma*N(0,1), optionally with a fraction of entries raised."""
    rng = rng or np.random.default_rng(PAPER_SEED)
    x = rng.standard_normal((B, V), dtype=np.float32)
    if sigma != 1.0:
        x *= np.float32(sigma)
    if peak_frac > 0.0:
        x += np.float32(peak_shift) * (rng.random((B, V), dtype=np.float32) < peak_frac)
    return x


def prev_tokens(B: int, V: int, rng: np.random.Generator) -> np.ndarray:
    return rng.integers(0, V, size=B, dtype=np.int64).astype(np.int32)


def context_tokens(B: int, width: int, V: int, rng: np.random.Generator) -> np.ndarray:
    """[B, width] windows of uniform token ids (the tokens before a decode step)."""
    return rng.integers(0, V, size=(B, width), dtype=np.int64).astype(np.int32)


def uniform_tokens(N: int, L: int, V: int, rng: np.random.Generator) -> np.ndarray:
    return rng.integers(0, V, size=(N, L), dtype=np.int64).astype(np.int32)


def watermark_inputs(config: str, B: int | None = None, V: int | None = None):
    """(logits, prev) for a watermark config; logits are fp32, or uint16 bf16 bits."""
    c = CONFIGS[config]
    B = B or c["B"]
    V = V or c["V"]
    rng = rng_for(config)
    x = logits(B, V, c["sigma"], rng, c.get("peak_frac", 0.0), c.get("peak_shift", 0.0))
    prev = prev_tokens(B, V, rng)
    if c["dtype"] == "bf16":
        x = f32_to_bf16_bits(x)
    return x, prev


def green_probability(gamma: float, delta: float) -> float:
    """Probability that a token drawn from softmax(l + delta*[green]) is green when
    the logits are i.i.d. and a fraction gamma of the vocabulary is green: by
    exchangeability each green token weighs e^delta against 1."""
    w = gamma * math.exp(delta)
    return w / (w + 1.0 - gamma)


Membership = Callable[[np.ndarray, np.ndarray], np.ndarray]


def sample_watermarked(N: int, L: int, V: int, gamma: float, delta: float,
                       is_green: Membership, rng: np.random.Generator,
                       candidates: int = 16, width: int = 1) -> np.ndarray:
    """Token sequences as a watermarked sampler would emit them from i.i.d. logits.

    At each step after the first `width` the colour is drawn (green with
    probability green_probability(gamma, delta)), then uniform candidates are drawn
    until one has that colour under is_green(window, cand), where window is the
    previous token ([n] ids) for width 1, or the `width` tokens before the step
    ([n, width] ids).  The first `width` tokens are uniform.  Candidates come in
    batches of ``candidates`` per row; the first match in draw order is kept, which
    is plain rejection sampling.  ``is_green`` is the caller's membership test.
    """
    q = green_probability(gamma, delta)
    tok = np.empty((N, L), dtype=np.int32)
    if L == 0:
        return tok
    head = min(width, L)
    tok[:, :head] = rng.integers(0, V, size=(N, head), dtype=np.int64).astype(np.int32)
    for i in range(head, L):
        want = rng.random(N) < q
        chosen = np.full(N, -1, dtype=np.int64)
        pending = np.arange(N)
        while pending.size:
            cand = rng.integers(0, V, size=(pending.size, candidates), dtype=np.int64)
            if width == 1:
                window = np.repeat(tok[pending, i - 1], candidates)
            else:
                window = np.repeat(tok[pending, i - width:i], candidates, axis=0)
            green = np.asarray(is_green(window.astype(np.int32),
                                        cand.reshape(-1).astype(np.int32)), dtype=bool)
            match = green.reshape(pending.size, candidates) == want[pending][:, None]
            hit = match.any(axis=1)
            first = match.argmax(axis=1)
            chosen[pending[hit]] = cand[hit, first[hit]]
            pending = pending[~hit]
        tok[:, i] = chosen.astype(np.int32)
    return tok


def detect_inputs(N: int, L: int, V: int, gamma: float, delta: float, seeding: str,
                  is_green: Membership, config: str = "c5", width: int = 1) -> np.ndarray:
    """c5-style detect batch: first half uniform (null), second half watermarked."""
    rng = rng_for(config, salt=(1 if seeding == "context" else 2) + 10 * (width - 1))
    n_null = N // 2
    null = uniform_tokens(n_null, L, V, rng)
    wm = sample_watermarked(N - n_null, L, V, gamma, delta, is_green, rng, width=width)
    return np.concatenate([null, wm], axis=0)
